"""Pins of the float64 GPT-step oracle (``oracle/gpt.py``) against things other
than itself: finite differences of its loss, library routines that compute the
same special case (torch's embedding lookup and its autograd, torch's AdamW),
and a closed form (a zero head gives the uniform distribution, loss = ln V)."""
import math

import numpy as np
import pytest
import torch

from oracle.gpt import GPTParams, adamw, embed_bwd, embed_fwd, gpt_fwd_bwd
from oracle.layer import LayerParams

B, S, D, H, F, V, L = 2, 6, 8, 2, 16, 9, 2


def tiny_model(seed=0, with_pe=True, activation="gelu"):
    r = np.random.default_rng(seed)
    n = lambda *s, sc=0.4: r.normal(0.0, sc, s)
    layers = [LayerParams(Wq=n(D, D), Wk=n(D, D), Wv=n(D, D), Wo=n(D, D), W1=n(D, F), W2=n(F, D),
                          ln1_g=1 + n(D, sc=0.2), ln1_b=n(D, sc=0.2), ln2_g=1 + n(D, sc=0.2),
                          ln2_b=n(D, sc=0.2), b1=n(F, sc=0.2), b2=n(D, sc=0.2), activation=activation)
              for _ in range(L)]
    P = GPTParams(Wte=n(V, D, sc=1.0), Wpe=n(S, D, sc=0.5) if with_pe else None, layers=layers,
                  lnf_g=1 + n(D, sc=0.2), lnf_b=n(D, sc=0.2), Wout=n(D, V, sc=0.5))
    tok = r.integers(0, V, (B, S))
    tok[0, :3] = 4                       # repeated tokens exercise the scatter-add
    tgt = r.integers(0, V, (B, S))
    return P, tok, tgt


def _entries(P: GPTParams):
    """(name, array) for every parameter array of the model."""
    out = [("Wte", P.Wte), ("Wpe", P.Wpe), ("lnf_g", P.lnf_g), ("lnf_b", P.lnf_b), ("Wout", P.Wout)]
    for l, lp in enumerate(P.layers):
        for k in ("Wq", "Wk", "Wv", "Wo", "W1", "W2", "ln1_g", "ln1_b", "ln2_g", "ln2_b", "b1", "b2"):
            out.append((f"{l}.{k}", getattr(lp, k)))
    return [(k, a) for k, a in out if a is not None]


def _grad(g, name):
    if "." in name:
        l, k = name.split(".")
        return g["layers"][int(l)]["d" + k]
    return g[name]


@pytest.mark.parametrize("activation", ["gelu", "relu"])
def test_gradients_match_finite_differences(activation):
    """Directional derivative of the loss along a random direction of every
    parameter array, by central differences."""
    P, tok, tgt = tiny_model(1, activation=activation)
    g = gpt_fwd_bwd(tok, tgt, P, H, dloss=1.0)
    r = np.random.default_rng(7)
    for name, arr in _entries(P):
        d = r.normal(size=arr.shape)
        h = 1e-6
        arr += h * d
        lp = gpt_fwd_bwd(tok, tgt, P, H, backward=False)["loss"]
        arr -= 2 * h * d
        lm = gpt_fwd_bwd(tok, tgt, P, H, backward=False)["loss"]
        arr += h * d
        fd = (lp - lm) / (2 * h)
        an = float((_grad(g, name) * d).sum())
        assert abs(fd - an) <= 1e-6 * max(1.0, abs(fd)), (name, fd, an)


def test_upstream_gradient_scales_linearly():
    P, tok, tgt = tiny_model(2)
    g1 = gpt_fwd_bwd(tok, tgt, P, H, dloss=1.0)
    g3 = gpt_fwd_bwd(tok, tgt, P, H, dloss=-3.0)
    for name, _ in _entries(P):
        np.testing.assert_allclose(_grad(g3, name), -3.0 * _grad(g1, name), rtol=1e-12, atol=1e-15)


def test_zero_head_is_uniform():
    """Wout = 0: every token sees uniform probabilities, loss = ln V exactly,
    dWout = (1/T) h^T (1/V - onehot(y)), and no gradient reaches the body."""
    P, tok, tgt = tiny_model(3)
    P.Wout[:] = 0.0
    g = gpt_fwd_bwd(tok, tgt, P, H)
    assert abs(g["loss"] - math.log(V)) < 1e-14
    hf = g["h"].reshape(B * S, D)
    onehot = np.eye(V)[tgt.reshape(-1)]
    np.testing.assert_allclose(g["Wout"], hf.T @ (1.0 / V - onehot) / (B * S), rtol=1e-12, atol=1e-15)
    for name in ("Wte", "Wpe", "0.Wq", "1.W2", "lnf_g"):
        assert np.abs(_grad(g, name)).max() == 0.0, name


def test_embedding_matches_torch():
    """Gather and scatter-add against torch's embedding lookup and its autograd
    (float64), with repeated tokens."""
    r = np.random.default_rng(4)
    Wte, Wpe = r.normal(size=(V, D)), r.normal(size=(S, D))
    tok = r.integers(0, V, (B, S))
    tok[1, 2:5] = 0
    dX = r.normal(size=(B, S, D))
    X = embed_fwd(tok, Wte, Wpe)
    tw = torch.tensor(Wte, requires_grad=True)
    tp = torch.tensor(Wpe, requires_grad=True)
    ref = torch.nn.functional.embedding(torch.tensor(tok), tw) + tp[None]
    ref.backward(torch.tensor(dX))
    np.testing.assert_array_equal(X, ref.detach().numpy())
    dWte, dWpe = embed_bwd(tok, dX, V, True)
    np.testing.assert_allclose(dWte, tw.grad.numpy(), rtol=1e-14, atol=1e-14)
    np.testing.assert_allclose(dWpe, tp.grad.numpy(), rtol=1e-14, atol=1e-14)


def test_embedding_bad_token():
    r = np.random.default_rng(5)
    Wte = r.normal(size=(V, D))
    tok = np.array([[1, V, -1, 2]])
    X = embed_fwd(tok, Wte, None)
    assert np.isnan(X[0, 1]).all() and np.isnan(X[0, 2]).all()
    np.testing.assert_array_equal(X[0, 0], Wte[1])
    dWte, dWpe = embed_bwd(tok, np.ones((1, 4, D)), V, False)
    assert dWpe is None and dWte.sum() == 2 * D


def test_adamw_matches_torch():
    """Three AdamW steps against torch.optim.AdamW (float64), weight decay 0.1."""
    r = np.random.default_rng(6)
    p0 = r.normal(size=(5, 7))
    grads = [r.normal(size=(5, 7)) for _ in range(3)]
    grads[1][0, 0] = 0.0
    tp = torch.tensor(p0, requires_grad=True)
    opt = torch.optim.AdamW([tp], lr=2e-4 * 50, betas=(0.9, 0.95), eps=1e-8, weight_decay=0.1)
    p, m, v = p0.copy(), np.zeros_like(p0), np.zeros_like(p0)
    for t, gr in enumerate(grads, start=1):
        tp.grad = torch.tensor(gr)
        opt.step()
        p, m, v = adamw(p, gr, m, v, t, lr=2e-4 * 50, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1)
        np.testing.assert_allclose(p, tp.detach().numpy(), rtol=1e-14, atol=1e-15)


def test_adamw_first_step_closed_form():
    """At step 1 the bias-corrected moments are g and g^2, so the update is
    -lr wd p - lr g / (|g| + eps)."""
    p = np.array([1.0, -2.0, 0.5, 3.0])
    g = np.array([0.3, -1e-3, 0.0, 2.0])
    lr, wd, eps = 1e-2, 0.1, 1e-8
    pn, m, v = adamw(p, g, np.zeros(4), np.zeros(4), 1, lr=lr, beta1=0.9, beta2=0.95, eps=eps, weight_decay=wd)
    np.testing.assert_allclose(pn, p - lr * wd * p - lr * g / (np.abs(g) + eps), rtol=1e-13, atol=1e-16)
    np.testing.assert_allclose(m, 0.1 * g, rtol=1e-15)
    np.testing.assert_allclose(v, 0.05 * g * g, rtol=1e-15)


# ----------------------------------------------------------------------------- bf16 rounding model of the step
def test_bf16_gpt_model_without_rounding_is_the_oracle():
    """``oracle/bf16_gpt.py`` with its rounding off is the float64 GPT step; with it on
    the loss moves by bf16-scale amounts only."""
    from oracle.bf16_gpt import bf16_gpt_fwd_bwd
    P, tok, tgt = tiny_model(5)
    ref = gpt_fwd_bwd(tok, tgt, P, H)
    m = bf16_gpt_fwd_bwd(tok, tgt, P, H, round_operands=False)
    assert abs(m["loss"] - ref["loss"]) <= 1e-12 * abs(ref["loss"])
    for name, _ in _entries(P):
        np.testing.assert_allclose(_grad(m, name), _grad(ref, name), rtol=0, atol=1e-11, err_msg=name)
    np.testing.assert_allclose(m["dX0"], ref["dX0"], rtol=0, atol=1e-11)
    mr = bf16_gpt_fwd_bwd(tok, tgt, P, H)
    assert 1e-6 < abs(mr["loss"] - ref["loss"]) / abs(ref["loss"]) < 2e-2
