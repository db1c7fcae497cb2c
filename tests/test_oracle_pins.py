"""Pins for the float64 oracle, each independent of the oracle's own code.

- golden values derived by hand / from standard tables (tests/golden/);
- brute force: pure-Python loops with math.exp / math.erf on tiny inputs;
- closed forms (uniform attention, single token, zero weights, LayerNorm moments);
- invariants (row sums, key shift, causality, batch independence, permutation
  equivariance, independence of the block sizes via Algorithm 1);
- central finite differences of the oracle's forward for every gradient;
- an independent torch autograd implementation.
"""
import json
import math
import os

import numpy as np
import pytest
import torch

import oracle
from oracle.layer import LayerParams, attention_head, layer_bwd, layer_fwd

EPS = 1e-5


def rand_params(rng, D, F, affine=True, biases=True, scale=None):
    s = scale if scale is not None else D ** -0.5
    p = LayerParams(Wq=rng.normal(0, s, (D, D)), Wk=rng.normal(0, s, (D, D)),
                    Wv=rng.normal(0, s, (D, D)), Wo=rng.normal(0, s, (D, D)),
                    W1=rng.normal(0, s, (D, F)), W2=rng.normal(0, s, (F, D)))
    if affine:
        p.ln1_g, p.ln1_b = 1 + 0.1 * rng.normal(size=D), 0.1 * rng.normal(size=D)
        p.ln2_g, p.ln2_b = 1 + 0.1 * rng.normal(size=D), 0.1 * rng.normal(size=D)
    if biases:
        p.b1, p.b2 = 0.1 * rng.normal(size=F), 0.1 * rng.normal(size=D)
    return p


# ----------------------------------------------------------------------------- golden
def test_attention_golden(golden_dir):
    g = json.load(open(os.path.join(golden_dir, "attention_closed_form.json")))
    Q, K, V = (np.array(g[k], dtype=np.float64) for k in ("Q", "K", "V"))
    for mode, causal in (("noncausal", False), ("causal", True)):
        O, P, lse = attention_head(Q, K, V, causal)
        np.testing.assert_allclose(O, g[mode]["O"], rtol=0, atol=1e-14)
        np.testing.assert_allclose(P, g[mode]["P"], rtol=0, atol=1e-15)
        np.testing.assert_allclose(lse, g[mode]["lse"], rtol=0, atol=1e-15)
        Ob, lseb = oracle.blockwise_attention_head(Q, K, V, causal, 1, 1)
        np.testing.assert_allclose(Ob, g[mode]["O"], rtol=0, atol=1e-14)
        np.testing.assert_allclose(lseb, g[mode]["lse"], rtol=0, atol=1e-15)


def test_gelu_golden(golden_dir):
    g = json.load(open(os.path.join(golden_dir, "normal_cdf.json")))
    x = np.array(g["x"])
    phi_cdf = np.array(g["Phi"])
    # GELU(x) = x Phi(x); GELU(-x) = -x (1 - Phi(x))
    np.testing.assert_allclose(oracle.gelu(x), x * phi_cdf, rtol=1e-15, atol=1e-16)
    np.testing.assert_allclose(oracle.gelu(-x), -x * (1 - phi_cdf), rtol=1e-13, atol=1e-16)
    dens = np.exp(-x * x / 2) / math.sqrt(2 * math.pi)
    np.testing.assert_allclose(oracle.gelu_grad(x), phi_cdf + x * dens, rtol=1e-15)
    np.testing.assert_allclose(oracle.gelu_grad(-x), 1 - phi_cdf - x * dens, rtol=1e-13, atol=1e-16)


def test_gelu_identities():
    z = np.linspace(-6, 6, 1001)
    np.testing.assert_allclose(oracle.gelu(z) - oracle.gelu(-z), z, atol=1e-14)
    h = 1e-6
    fd = (oracle.gelu(z + h) - oracle.gelu(z - h)) / (2 * h)
    np.testing.assert_allclose(oracle.gelu_grad(z), fd, atol=1e-8)


# ----------------------------------------------------------------------------- brute force
def brute_attention(Q, K, V, causal):
    S, dh = len(Q), len(Q[0])
    O, lse = [], []
    for q in range(S):
        keys = [k for k in range(len(K)) if (k <= q or not causal)]
        sc = [sum(Q[q][d] * K[k][d] for d in range(dh)) / math.sqrt(dh) for k in keys]
        m = max(sc)
        e = [math.exp(s - m) for s in sc]
        tot = sum(e)
        O.append([sum(e[i] * V[k][d] for i, k in enumerate(keys)) / tot for d in range(dh)])
        lse.append(m + math.log(tot))
    return O, lse


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("S,dh", [(1, 1), (3, 2), (4, 4)])
def test_attention_bruteforce(causal, S, dh):
    rng = np.random.default_rng(S * 10 + dh)
    Q, K, V = (rng.normal(size=(S, dh)) for _ in range(3))
    O, P, lse = attention_head(Q, K, V, causal)
    Ob, lseb = brute_attention(Q.tolist(), K.tolist(), V.tolist(), causal)
    np.testing.assert_allclose(O, Ob, rtol=0, atol=1e-14)
    np.testing.assert_allclose(lse, lseb, rtol=0, atol=1e-14)


def brute_layer(X, p, H, causal, eps):
    """The whole layer with Python floats and loops only."""
    B, S, D = len(X), len(X[0]), len(X[0][0])
    F = len(p["W1"][0])
    dh = D // H

    def ln(row, g, b):
        mu = sum(row) / D
        var = sum((v - mu) ** 2 for v in row) / D
        r = 1.0 / math.sqrt(var + eps)
        return [(row[i] - mu) * r * (g[i] if g else 1.0) + (b[i] if b else 0.0) for i in range(D)]

    def mat(row, W):
        return [sum(row[i] * W[i][j] for i in range(len(row))) for j in range(len(W[0]))]

    Y = []
    for b in range(B):
        U = [ln(X[b][t], p["ln1_g"], p["ln1_b"]) for t in range(S)]
        Qm, Km, Vm = ([mat(u, p[w]) for u in U] for w in ("Wq", "Wk", "Wv"))
        O = [[0.0] * D for _ in range(S)]
        for h in range(H):
            cs = range(h * dh, (h + 1) * dh)
            Oh, _ = brute_attention([[r[c] for c in cs] for r in Qm], [[r[c] for c in cs] for r in Km],
                                    [[r[c] for c in cs] for r in Vm], causal)
            for t in range(S):
                for i, c in enumerate(cs):
                    O[t][c] = Oh[t][i]
        Yb = []
        for t in range(S):
            hd = [X[b][t][j] + v for j, v in enumerate(mat(O[t], p["Wo"]))]
            vn = ln(hd, p["ln2_g"], p["ln2_b"])
            z = [v + (p["b1"][j] if p["b1"] else 0.0) for j, v in enumerate(mat(vn, p["W1"]))]
            g = [v * 0.5 * (1 + math.erf(v / math.sqrt(2))) for v in z]
            Yb.append([hd[j] + v + (p["b2"][j] if p["b2"] else 0.0) for j, v in enumerate(mat(g, p["W2"]))])
        Y.append(Yb)
    return Y


@pytest.mark.parametrize("causal", [False, True])
def test_layer_bruteforce(causal):
    rng = np.random.default_rng(7)
    B, S, D, H, F = 2, 3, 4, 2, 6
    p = rand_params(rng, D, F)
    X = rng.normal(size=(B, S, D))
    Y, _ = layer_fwd(X, p, H, causal, EPS)
    pl = {k: (None if v is None else v.tolist()) for k, v in vars(p).items()
          if k not in ("activation", "dropout", "dropout_seed")}
    Yb = brute_layer(X.tolist(), pl, H, causal, EPS)
    np.testing.assert_allclose(Y, Yb, rtol=0, atol=1e-13)


# ----------------------------------------------------------------------------- closed forms
def test_uniform_attention_is_prefix_mean():
    rng = np.random.default_rng(1)
    S, dh = 9, 8
    Q, V = rng.normal(size=(S, dh)), rng.normal(size=(S, dh))
    K = np.zeros((S, dh))                       # all scores 0 -> uniform weights
    O, _, lse = attention_head(Q, K, V, causal=True)
    np.testing.assert_allclose(O, np.cumsum(V, 0) / np.arange(1, S + 1)[:, None], atol=1e-14)
    np.testing.assert_allclose(lse, np.log(np.arange(1, S + 1)), atol=1e-14)
    O, _, lse = attention_head(Q, K, V, causal=False)
    np.testing.assert_allclose(O, np.broadcast_to(V.mean(0), O.shape), atol=1e-14)


def test_single_token_attention_returns_value():
    rng = np.random.default_rng(2)
    Q, K, V = (rng.normal(size=(1, 16)) for _ in range(3))
    O, P, lse = attention_head(Q, K, V, causal=False)
    np.testing.assert_array_equal(O, V)
    np.testing.assert_allclose(lse, (Q @ K.T)[0] / 4.0, atol=1e-15)


def test_dominant_score_selects_value():
    S, dh = 5, 4
    Q = np.zeros((S, dh)); K = np.zeros((S, dh)); V = np.arange(S * dh, dtype=float).reshape(S, dh)
    Q[:, 0] = 200.0
    K[3, 0] = 1.0                               # key 3 wins by exp(100) for every query
    O, _, _ = attention_head(Q, K, V, causal=False)
    np.testing.assert_allclose(O, np.broadcast_to(V[3], O.shape), atol=1e-12)


def test_layer_norm_moments():
    x = np.array([[1.0, 2.0, 3.0, 4.0]])
    out, xhat, rstd = oracle.layer_norm_fwd(x, None, None, EPS)
    np.testing.assert_allclose(out, (x - 2.5) / math.sqrt(1.25 + EPS), atol=1e-15)
    rng = np.random.default_rng(3)
    z = rng.normal(3.0, 2.0, size=(6, 64))
    out, _, _ = oracle.layer_norm_fwd(z, None, None, EPS)
    var = z.var(axis=1)
    np.testing.assert_allclose(out.mean(1), 0, atol=1e-14)
    np.testing.assert_allclose(out.var(1), var / (var + EPS), rtol=1e-13)


def test_zero_weights_short_circuit():
    rng = np.random.default_rng(4)
    B, S, D, H, F = 1, 6, 8, 2, 16
    X = rng.normal(size=(B, S, D))
    p = rand_params(rng, D, F, affine=True, biases=False)
    p.Wo = np.zeros((D, D))
    Y, c = layer_fwd(X, p, H, True, EPS)
    np.testing.assert_array_equal(c["Hd"], X)              # Wo = 0: residual 1 passes X
    p.W1 = np.zeros((D, F))
    Y, c = layer_fwd(X, p, H, True, EPS)
    np.testing.assert_array_equal(c["G"], 0.0)             # GELU(0) = 0
    np.testing.assert_array_equal(Y, X)                    # FFN adds nothing


# ----------------------------------------------------------------------------- invariants
def test_probability_rows_and_key_shift():
    rng = np.random.default_rng(5)
    S, dh = 33, 16
    Q, K, V = (rng.normal(size=(S, dh)) for _ in range(3))
    for causal in (False, True):
        O, P, lse = attention_head(Q, K, V, causal)
        np.testing.assert_allclose(P.sum(1), 1.0, atol=1e-14)
        if causal:
            assert np.all(np.triu(P, 1) == 0.0)
        u = rng.normal(size=dh)                 # same shift on every key: scores += q.u/sqrt(dh)
        O2, _, lse2 = attention_head(Q, K + u, V, causal)
        np.testing.assert_allclose(O2, O, atol=1e-12)
        np.testing.assert_allclose(lse2, lse + Q @ u / 4.0, atol=1e-12)


def test_causality_and_batch_independence():
    rng = np.random.default_rng(6)
    B, S, D, H, F = 2, 17, 16, 2, 32
    p = rand_params(rng, D, F)
    X = rng.normal(size=(B, S, D))
    Y, _ = layer_fwd(X, p, H, True, EPS)
    for t in (0, 5, 16):
        X2 = X.copy()
        X2[:, t:] += rng.normal(size=X2[:, t:].shape)
        Y2, _ = layer_fwd(X2, p, H, True, EPS)
        np.testing.assert_array_equal(Y2[:, :t], Y[:, :t])
        assert not np.allclose(Y2[:, t:], Y[:, t:])
    X3 = X.copy()
    X3[1] += 1.0 + rng.normal(size=X3[1].shape)
    Y3, _ = layer_fwd(X3, p, H, False, EPS)
    Y0, _ = layer_fwd(X, p, H, False, EPS)
    np.testing.assert_array_equal(Y3[0], Y0[0])


def test_noncausal_permutation_equivariance():
    rng = np.random.default_rng(8)
    B, S, D, H, F = 1, 11, 16, 4, 24
    p = rand_params(rng, D, F)
    X = rng.normal(size=(B, S, D))
    perm = rng.permutation(S)
    Y, _ = layer_fwd(X, p, H, False, EPS)
    Yp, _ = layer_fwd(X[:, perm], p, H, False, EPS)
    np.testing.assert_allclose(Yp, Y[:, perm], atol=1e-12)


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("S,blocks", [
    (1, [(1, 1)]),
    (7, [(1, 1), (3, 2), (7, 7), (6, 1), (2, 5)]),
    (64, [(1, 3), (16, 16), (63, 64), (64, 1)]),
    (250, [(16, 128), (128, 16), (129, 3), (249, 250), (250, 250)]),
    (512, [(128, 128), (129, 511), (512, 64)]),
])
def test_blockwise_equals_unblocked(causal, S, blocks):
    rng = np.random.default_rng(S)
    B, D, H, F = (2, 16, 2, 32) if S < 250 else (1, 32, 2, 32)
    p = rand_params(rng, D, F)
    X = rng.normal(size=(B, S, D))
    Y, c = layer_fwd(X, p, H, causal, EPS)
    for Bq, Bkv in blocks:
        Yb, Ob, lseb = oracle.blockwise_layer_fwd(X, p, H, causal, Bq, Bkv, EPS)
        np.testing.assert_allclose(Ob, c["O"], rtol=0, atol=1e-12 * np.abs(c["O"]).max())
        np.testing.assert_allclose(lseb, c["lse"], rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(Yb, Y, rtol=0, atol=1e-12 * np.abs(Y).max())


# ----------------------------------------------------------------------------- gradients
GRAD_OF = {"dX": "X", "dWq": "Wq", "dWk": "Wk", "dWv": "Wv", "dWo": "Wo", "dW1": "W1", "dW2": "W2",
           "db1": "b1", "db2": "b2", "dln1_g": "ln1_g", "dln1_b": "ln1_b", "dln2_g": "ln2_g",
           "dln2_b": "ln2_b"}


@pytest.mark.parametrize("causal,activation", [(False, "gelu"), (True, "gelu"), (True, "relu")])
def test_finite_differences(causal, activation):
    rng = np.random.default_rng(11 + causal)
    B, S, D, H, F = 2, 7, 8, 2, 16
    p = rand_params(rng, D, F, scale=0.5)
    p.activation = activation
    X = rng.normal(size=(B, S, D))
    dY = rng.normal(size=(B, S, D))
    Y, cache = layer_fwd(X, p, H, causal, EPS)
    grads = layer_bwd(cache, p, dY)

    def loss(Xv, pv):
        return float((layer_fwd(Xv, pv, H, causal, EPS)[0] * dY).sum())

    for gname, pname in GRAD_OF.items():
        base = X if pname == "X" else getattr(p, pname)
        fd = np.empty_like(base)
        for idx in np.ndindex(base.shape):
            orig = base[idx]
            h = 1e-6 * max(1.0, abs(orig))
            base[idx] = orig + h
            lp = loss(X, p)
            base[idx] = orig - h
            lm = loss(X, p)
            base[idx] = orig
            fd[idx] = (lp - lm) / (2 * h)
        an = grads[gname]
        err = np.abs(fd - an).max() / max(np.abs(an).max(), 1e-3)
        assert err < 1e-6, (gname, err)


def test_gradient_invariants():
    rng = np.random.default_rng(12)
    B, S, D, H, F = 2, 9, 16, 2, 24
    p = rand_params(rng, D, F)
    X, dY = rng.normal(size=(B, S, D)), rng.normal(size=(B, S, D))
    _, cache = layer_fwd(X, p, H, True, EPS)
    g = layer_bwd(cache, p, dY)
    # the gradient that flows into a LayerNorm input sums to zero per token
    np.testing.assert_allclose((g["dX"] - g["dHd"]).sum(-1), 0, atol=1e-12)
    np.testing.assert_allclose(g["db2"], dY.sum((0, 1)), atol=1e-13)
    # causal: the last token's key/value receive gradient only from the last query
    dY2 = np.zeros_like(dY)
    dY2[:, :-1] = dY[:, :-1]
    g2 = layer_bwd(cache, p, dY2)
    np.testing.assert_allclose(g2["dK"][:, -1], 0, atol=1e-15)
    np.testing.assert_allclose(g2["dV"][:, -1], 0, atol=1e-15)


def torch_layer(X, p, H, causal, eps):
    """An independent float64 implementation with torch ops + autograd."""
    import torch.nn.functional as Fn
    B, S, D = X.shape
    dh = D // H
    t = {k: (None if v is None else torch.tensor(v, requires_grad=True)) for k, v in vars(p).items()
         if k not in ("activation", "dropout", "dropout_seed")}
    Xt = torch.tensor(X, requires_grad=True)
    U = Fn.layer_norm(Xt, (D,), t["ln1_g"], t["ln1_b"], eps)
    q = (U @ t["Wq"]).view(B, S, H, dh).transpose(1, 2)
    k = (U @ t["Wk"]).view(B, S, H, dh).transpose(1, 2)
    v = (U @ t["Wv"]).view(B, S, H, dh).transpose(1, 2)
    sc = q @ k.transpose(-1, -2) / math.sqrt(dh)
    if causal:
        sc = sc.masked_fill(~torch.ones(S, S, dtype=torch.bool).tril(), float("-inf"))
    o = (torch.softmax(sc, -1) @ v).transpose(1, 2).reshape(B, S, D)
    hd = Xt + o @ t["Wo"]
    z = Fn.layer_norm(hd, (D,), t["ln2_g"], t["ln2_b"], eps) @ t["W1"]
    if t["b1"] is not None:
        z = z + t["b1"]
    y = hd + (Fn.relu(z) if p.activation == "relu" else Fn.gelu(z)) @ t["W2"]
    if t["b2"] is not None:
        y = y + t["b2"]
    return y, Xt, t


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("affine,biases", [(True, True), (False, False)])
@pytest.mark.parametrize("activation", ["gelu", "relu"])
def test_torch_autograd_crosscheck(causal, affine, biases, activation):
    rng = np.random.default_rng(13)
    B, S, D, H, F = 2, 37, 32, 4, 64
    p = rand_params(rng, D, F, affine=affine, biases=biases)
    p.activation = activation
    X, dY = rng.normal(size=(B, S, D)), rng.normal(size=(B, S, D))
    Y, cache = layer_fwd(X, p, H, causal, EPS)
    g = layer_bwd(cache, p, dY)
    yt, Xt, t = torch_layer(X, p, H, causal, EPS)
    yt.backward(torch.tensor(dY))
    np.testing.assert_allclose(Y, yt.detach().numpy(), rtol=0, atol=1e-12)
    for gname, pname in GRAD_OF.items():
        ref = Xt.grad if pname == "X" else (t[pname].grad if t[pname] is not None else None)
        if ref is None:
            assert g[gname] is None
            continue
        ref = ref.numpy()
        np.testing.assert_allclose(g[gname], ref, rtol=0, atol=1e-11 * max(1.0, np.abs(ref).max()),
                                   err_msg=gname)


# ----------------------------------------------------------------------------- rows oracle
@pytest.mark.parametrize("causal", [False, True])
def test_rows_oracle_matches_full(causal):
    rng = np.random.default_rng(14)
    B, S, D, H, F = 2, 40, 16, 2, 32
    p = rand_params(rng, D, F)
    X, dY = rng.normal(size=(B, S, D)), rng.normal(size=(B, S, D))
    rows = np.array([0, 3, 17, 18, 31])
    dYm = np.zeros_like(dY)
    dYm[:, rows] = dY[:, rows]
    Y, cache = layer_fwd(X, p, H, causal, EPS)
    g = layer_bwd(cache, p, dYm)
    Yr, gr = oracle.rows_layer_fwd_bwd(X, p, H, causal, rows, dY[:, rows], EPS)
    np.testing.assert_allclose(Yr, Y[:, rows], rtol=0, atol=1e-13)
    for k in GRAD_OF:
        np.testing.assert_allclose(gr[k], g[k], rtol=0, atol=1e-12, err_msg=k)
    Yr2, none = oracle.rows_layer_fwd_bwd(X, p, H, causal, rows, None, EPS)
    assert none is None
    np.testing.assert_array_equal(Yr2, Yr)


# ----------------------------------------------------------------------------- bf16 rounding model
def test_bf16_rounding_matches_torch():
    from oracle.bf16_model import to_bf16
    rng = np.random.default_rng(15)
    x = np.concatenate([rng.normal(size=4000) * 10 ** rng.uniform(-6, 6, 4000),
                        np.array([0.0, -0.0, 1.0, 1.00390625, 1.01171875, -3.0e38, 1e-40])])
    x32 = x.astype(np.float32)
    ref = torch.from_numpy(x32).to(torch.bfloat16).double().numpy()
    np.testing.assert_array_equal(to_bf16(x32.astype(np.float64)), ref)
    # ties go to even: 1 + 2^-8 lies halfway between 1 and 1 + 2^-7
    assert to_bf16(np.array([1.0 + 2 ** -8]))[0] == 1.0
    assert to_bf16(np.array([1.0 + 3 * 2 ** -8]))[0] == 1.0 + 2 ** -6


@pytest.mark.parametrize("causal", [False, True])
def test_bf16_model_without_rounding_is_the_oracle(causal):
    from oracle.bf16_model import bf16_layer_fwd_bwd
    rng = np.random.default_rng(16)
    B, S, D, H, F = 2, 21, 16, 2, 32
    p = rand_params(rng, D, F)
    X, dY = rng.normal(size=(B, S, D)), rng.normal(size=(B, S, D))
    Y, cache = layer_fwd(X, p, H, causal, EPS)
    g = layer_bwd(cache, p, dY)
    m = bf16_layer_fwd_bwd(X, p, H, causal, dY, EPS, round_operands=False)
    np.testing.assert_allclose(m["Y"], Y, atol=1e-12)
    np.testing.assert_allclose(m["O"], cache["O"], atol=1e-12)
    for k in GRAD_OF:
        np.testing.assert_allclose(m[k], g[k], atol=1e-11, err_msg=k)
    mr = bf16_layer_fwd_bwd(X, p, H, causal, dY, EPS)     # rounding on: close, not equal
    rel = np.abs(mr["Y"] - Y).max() / np.abs(Y).max()
    assert 1e-5 < rel < 5e-2


# ----------------------------------------------------------------------------- bf16 rounding model on rows
@pytest.mark.parametrize("causal", [False, True])
def test_bf16_rows_model_matches_full_model(causal):
    """With dY zero outside the selected rows, the rows-restricted rounding model returns the
    full rounding model's Y rows and every gradient (rounding included)."""
    from oracle.bf16_model import bf16_layer_fwd_bwd, to_bf16
    from oracle.bf16_rows import bf16_rows_fwd_bwd
    rng = np.random.default_rng(17)
    B, S, D, H, F = 2, 37, 16, 2, 32
    p = rand_params(rng, D, F)
    X, dY = rng.normal(size=(B, S, D)), to_bf16(rng.normal(size=(B, S, D)))
    rows = np.array([0, 5, 18, 19, 36])
    dYm = np.zeros_like(dY)
    dYm[:, rows] = dY[:, rows]
    full = bf16_layer_fwd_bwd(X, p, H, causal, dYm, EPS)
    part = bf16_rows_fwd_bwd(X, p, H, causal, rows, dY[:, rows], EPS)
    np.testing.assert_allclose(part["Y"], full["Y"][:, rows], rtol=0, atol=1e-12)
    for k in list(GRAD_OF) + ["db1", "db2", "dln1_g", "dln1_b", "dln2_g", "dln2_b"]:
        np.testing.assert_allclose(part[k], full[k], rtol=0, atol=1e-11, err_msg=k)


@pytest.mark.parametrize("causal", [False, True])
def test_bf16_rows_model_without_rounding_is_the_rows_oracle(causal):
    from oracle.bf16_rows import bf16_rows_fwd_bwd
    rng = np.random.default_rng(18)
    B, S, D, H, F = 1, 29, 16, 2, 32
    p = rand_params(rng, D, F)
    X, dY = rng.normal(size=(B, S, D)), rng.normal(size=(B, S, D))
    rows = np.array([2, 11, 28])
    Yr, gr = oracle.rows_layer_fwd_bwd(X, p, H, causal, rows, dY[:, rows], EPS)
    m = bf16_rows_fwd_bwd(X, p, H, causal, rows, dY[:, rows], EPS, round_operands=False)
    np.testing.assert_allclose(m["Y"], Yr, rtol=0, atol=1e-12)
    for k in GRAD_OF:
        np.testing.assert_allclose(m[k], gr[k], rtol=0, atol=1e-11, err_msg=k)


def test_relu_ffn_closed_form():
    """With every FFN pre-activation positive (b1 large) eq. (2)'s ReLU FFN is the plain
    affine map (Vn W1 + b1) W2 + b2; with every one negative it is b2 alone."""
    rng = np.random.default_rng(17)
    B, S, D, H, F = 1, 6, 8, 2, 12
    X = rng.normal(size=(B, S, D))
    for sign in (1.0, -1.0):
        p = rand_params(rng, D, F)
        p.activation = "relu"
        p.b1 = sign * 1e3 * np.ones(F)
        Y, c = layer_fwd(X, p, H, True, EPS)
        lin = (c["Vn"] @ p.W1 + p.b1) @ p.W2 if sign > 0 else 0.0
        np.testing.assert_allclose(Y, c["Hd"] + lin + p.b2, rtol=0, atol=1e-9)
