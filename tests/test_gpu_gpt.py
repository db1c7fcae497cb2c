"""GPU parity of the GPT training step (embedding, L BPT layers, final LayerNorm,
LM-head cross-entropy, AdamW) and of its new entry points, through the C ABI,
against the float64 oracle (``oracle/gpt.py``) on the same seeded inputs."""
import numpy as np
import pytest
import torch

from bpt_inputs import make_gpt_inputs
from oracle.gpt import GPTParams, adamw, embed_bwd, embed_fwd, gpt_fwd_bwd
from oracle.layer import LayerParams, layer_norm_bwd, layer_norm_fwd
from paper_2305_19370_amd import bpt
from paper_2305_19370_amd.gpt import GPT, GPTShape, LAYER_MATS, LAYER_VECS
from tests.gpu_util import say, stats

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def f64(t):
    return t.detach().to("cpu").double().numpy()


def oracle_params(inp, s: GPTShape) -> GPTParams:
    layers = []
    for l in range(s.L):
        kw = {k: f64(inp[f"{l}.{k}"]) for k in LAYER_MATS}
        kw.update({k: (f64(inp[f"{l}.{k}"]) if f"{l}.{k}" in inp else None) for k in LAYER_VECS})
        layers.append(LayerParams(**kw, activation=s.activation))
    return GPTParams(Wte=f64(inp["Wte"]), Wpe=f64(inp["Wpe"]) if "Wpe" in inp else None, layers=layers,
                     lnf_g=f64(inp["lnf_g"]), lnf_b=f64(inp["lnf_b"]), Wout=f64(inp["Wout"])[:, :s.V])


def build(s: GPTShape, seed: int):
    inp = make_gpt_inputs(s.L, s.B, s.S, s.D, s.F, s.V, s.ldw, dtype=s.dtype, seed=seed, pos_table=s.pos_table,
                          biases=s.biases)
    m = GPT(s, device=DEV, init=False)
    for name in m.names():
        m.master(name).copy_(inp[name].float())
    m.sync_lowp()
    return m, inp


def grad_pairs(m: GPT, ref, s: GPTShape):
    """(name, gpu, oracle) for every parameter gradient."""
    out = [("Wte", m.grad("Wte"), ref["Wte"]), ("lnf_g", m.grad("lnf_g"), ref["lnf_g"]),
           ("lnf_b", m.grad("lnf_b"), ref["lnf_b"]), ("Wout", m.grad("Wout")[:, :s.V], ref["Wout"])]
    if s.pos_table:
        out.append(("Wpe", m.grad("Wpe"), ref["Wpe"]))
    for l in range(s.L):
        for k in LAYER_MATS + LAYER_VECS:
            if f"{l}.{k}" in m.names():
                out.append((f"{l}.{k}", m.grad(f"{l}.{k}"), ref["layers"][l]["d" + k]))
    return out


def run_step(s: GPTShape, seed: int):
    say(f"[gpt] {s}")
    m, inp = build(s, seed)
    tok, tgt = inp["tokens"].to(DEV), inp["targets"].to(DEV)
    loss = m.forward(tok, tgt)
    m.backward(tok, tgt)
    torch.cuda.synchronize()
    ref = gpt_fwd_bwd(inp["tokens"].numpy().reshape(s.B, s.S), inp["targets"].numpy().reshape(s.B, s.S),
                      oracle_params(inp, s), s.H, s.causal, s.ln_eps)
    return m, inp, float(loss.item()), ref


@pytest.mark.parametrize("kw", [
    dict(L=2, B=2, S=320, D=256, H=4, F=1024, V=1000, Bq=128, Bkv=128),
    dict(L=1, B=1, S=200, D=256, H=2, F=512, V=777, Bq=64, Bkv=128, activation="relu", biases=False,
         pos_table=False),
], ids=["gelu_L2_ragged", "relu_L1_nopos"])
def test_gpt_step_f32(kw):
    """fp32 path: loss, dX of the embedding output and every gradient within
    max|diff| <= 1e-4 rms(ref) (the layer's fp32 bound); padding columns of dWout zero."""
    s = GPTShape(dtype="f32", **kw)
    m, inp, loss, ref = run_step(s, 1)
    assert abs(loss - ref["loss"]) <= 1e-5 * abs(ref["loss"]), (loss, ref["loss"])
    st = stats(f64(m.dX0).reshape(s.B, s.S, s.D), ref["dX0"])
    assert st["e_max"] <= 1e-4, st
    for name, g, r in grad_pairs(m, ref, s):
        st = stats(f64(g), r)
        assert st["e_max"] <= 1e-4, (name, st)
    assert float(m.grad("Wout")[:, s.V:].abs().max()) == 0.0


def test_gpt_step_bf16():
    """bf16 path (bf16 weights and activations, fp32 accumulation, fp32 masters): every
    gradient and the loss gated like one layer's bf16 outputs, over the rounding model
    of the whole step (oracle/bf16_gpt.py: each layer's bf16 rounding model, bf16 layer
    outputs and head operands): e_max <= max(2e-2, F_max x the model's), e_mean <=
    max(2e-3, F_mean x the model's), and |loss - ref| <= F_max x the model's."""
    from oracle.bf16_gpt import bf16_gpt_fwd_bwd
    from tests.gpu_util import bf16_limits
    s = GPTShape(L=2, B=1, S=512, D=256, H=2, F=1024, V=2000, Bq=128, Bkv=128, dtype="bf16")
    m, inp, loss, ref = run_step(s, 2)
    P = oracle_params(inp, s)
    model = bf16_gpt_fwd_bwd(inp["tokens"].numpy().reshape(s.B, s.S), inp["targets"].numpy().reshape(s.B, s.S),
                             P, s.H, s.causal, s.ln_eps)
    lim_loss = bf16_limits({"e_max": abs(model["loss"] - ref["loss"]), "e_mean": 0.0})[0]
    say(f"[gpt] bf16 loss {loss:.6f} ref {ref['loss']:.6f} model {model['loss']:.6f} (limit {lim_loss:.3e})")
    assert abs(loss - ref["loss"]) <= lim_loss, (loss, ref["loss"], model["loss"])
    bad, rows = [], []
    mpairs = {n: r for n, _, r in grad_pairs(m, model, s)}
    for name, g, r in grad_pairs(m, ref, s):
        st = stats(f64(g), r)
        lim_max, lim_mean = bf16_limits(stats(mpairs[name], r))
        rows.append(f"{name:10s} e_max {st['e_max']:.2e} (<= {lim_max:.2e})  e_mean {st['e_mean']:.2e} "
                    f"(<= {lim_mean:.2e})")
        if not (st["e_max"] <= lim_max and st["e_mean"] <= lim_mean):
            bad.append(name)
    say("[gpt] bf16\n" + "\n".join(rows))
    assert not bad, bad


def test_gpt_train_steps_update_masters_and_copies():
    """Three steps of forward, backward and AdamW: the fp32 masters follow the oracle's
    AdamW of the GPU's own gradients, the bf16 copies are the masters rounded to nearest
    even, and the loss decreases on a repeated batch."""
    s = GPTShape(L=1, B=1, S=256, D=256, H=2, F=512, V=500, Bq=128, Bkv=128, dtype="bf16")
    say(f"[gpt] train steps {s}")
    m, inp = build(s, 3)
    tok, tgt = inp["tokens"].to(DEV), inp["targets"].to(DEV)
    losses = []
    mom = {n: (np.zeros(m.master(n).shape), np.zeros(m.master(n).shape)) for n in m.names()}
    for step in range(1, 4):
        before = {n: f64(m.master(n)) for n in m.names()}
        losses.append(float(m.forward(tok, tgt).item()))
        m.backward(tok, tgt)
        grads = {n: f64(m.grad(n)) for n in m.names()}
        m.optimizer_step(lr=3e-3, weight_decay=0.1)
        torch.cuda.synchronize()
        for n in m.names():
            wd = 0.1 if n in m.decay.index else 0.0
            p, mm, vv = adamw(before[n], grads[n], *mom[n], step, lr=3e-3, weight_decay=wd)
            mom[n] = (mm, vv)
            got = f64(m.master(n))
            assert np.abs(got - p).max() <= 1e-6 * (np.abs(p).max() + 3e-3), (step, n)
            if n in m.decay.index:
                assert torch.equal(m.weight(n), m.master(n).to(torch.bfloat16)), (step, n)
    say(f"[gpt] losses {losses}")
    assert losses[2] < losses[0]


@pytest.mark.parametrize("n,lowp", [(9_000_003, "bf16"), (5, "f32"), (4096, None)])
def test_adamw_kernel(n, lowp):
    """Two AdamW steps against the oracle on random state (grid-stride and tail cases)."""
    say(f"[adamw] n={n} lowp={lowp}")
    g = torch.Generator(device="cpu").manual_seed(n)
    p0 = torch.randn(n, generator=g)
    m0 = torch.randn(n, generator=g) * 0.1
    v0 = torch.rand(n, generator=g) * 0.01
    grads = [torch.randn(n, generator=g) for _ in range(2)]
    p, m, v = p0.to(DEV), m0.to(DEV), v0.to(DEV)
    low = None if lowp is None else torch.empty(n, dtype=torch.bfloat16 if lowp == "bf16" else torch.float32,
                                                device=DEV)
    rp, rm, rv = p0.double().numpy(), m0.double().numpy(), v0.double().numpy()
    for step in (5, 6):
        bpt.adamw_step(p, grads[step - 5].to(DEV), m, v, step, lr=1e-2, weight_decay=0.1, p_lowp=low)
        rp, rm, rv = adamw(rp, grads[step - 5].double().numpy(), rm, rv, step, lr=1e-2, weight_decay=0.1)
    torch.cuda.synchronize()
    assert np.abs(f64(p) - rp).max() <= 1e-6 * (np.abs(rp).max() + 1e-2)
    assert np.abs(f64(m) - rm).max() <= 1e-6 * np.abs(rm).max()
    assert np.abs(f64(v) - rv).max() <= 1e-6 * np.abs(rv).max()
    if low is not None:
        assert torch.equal(low, p.to(low.dtype))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_embedding(dtype):
    """Gather (NaN row for an out-of-range token) and both gradients; a small vocabulary
    so that tokens repeat many times in dWte's atomic sums."""
    B, S, D, V = 2, 300, 264, 50
    say(f"[embed] {dtype} B={B} S={S} D={D} V={V}")
    inp = make_gpt_inputs(0, B, S, D, 8, V, 64, dtype=dtype, seed=4)
    tok = inp["tokens"].clone()
    tok[3], tok[S + 7] = V, -1
    dt = torch.float32 if dtype == "f32" else torch.bfloat16
    dX = (torch.randn((B * S, D), generator=torch.Generator().manual_seed(9))).to(dt)
    cfg = bpt.make_embed_config(B, S, D, V, dtype=dtype)
    X = torch.empty((B * S, D), dtype=dt, device=DEV)
    dWte = torch.full((V, D), 7.0, device=DEV)
    dWpe = torch.full((S, D), 7.0, device=DEV)
    bpt.embed_fwd(cfg, tok.to(DEV), inp["Wte"].to(DEV), inp["Wpe"].to(DEV), X)
    bpt.embed_bwd(cfg, tok.to(DEV), dX.to(DEV), dWte, dWpe)
    torch.cuda.synchronize()
    tok2 = tok.numpy().reshape(B, S)
    rX = embed_fwd(tok2, f64(inp["Wte"]), f64(inp["Wpe"])).reshape(B * S, D)
    gX = f64(X)
    bad = np.isnan(rX[:, 0])
    assert bad.sum() == 2 and np.isnan(gX[bad]).all() and np.isfinite(gX[~bad]).all()
    if dtype == "f32":
        assert np.array_equal(gX[~bad], rX[~bad].astype(np.float32).astype(np.float64))
    else:
        assert (np.abs(gX[~bad] - rX[~bad]) <= 2.0 ** -8 * np.abs(rX[~bad])).all()
    rWte, rWpe = embed_bwd(tok2, f64(dX).reshape(B, S, D), V, True)
    assert stats(f64(dWte), rWte)["e_max"] <= 1e-5
    assert stats(f64(dWpe), rWpe)["e_max"] <= 1e-6


@pytest.mark.parametrize("rows,D,dtype", [(100, 4096, "f32"), (77, 264, "f32"), (130, 2048, "bf16")])
def test_final_layernorm(rows, D, dtype):
    say(f"[ln] rows={rows} D={D} {dtype}")
    gen = torch.Generator().manual_seed(rows)
    dt = torch.float32 if dtype == "f32" else torch.bfloat16
    X = (torch.randn((rows, D), generator=gen) * 2 + 0.5).to(dt)
    g = torch.randn(D, generator=gen) * 0.1 + 1
    b = torch.randn(D, generator=gen) * 0.1
    dY = torch.randn((rows, D), generator=gen).to(dt)
    cfg = bpt.make_ln_config(rows, D, 1e-5, in_dtype=dtype)
    Y = torch.empty((rows, D), dtype=dt, device=DEV)
    dX = torch.empty((rows, D), dtype=dt, device=DEV)
    mean = torch.empty(rows, device=DEV)
    rstd = torch.empty(rows, device=DEV)
    dg = torch.empty(D, device=DEV)
    db = torch.empty(D, device=DEV)
    ws = torch.empty(bpt.ln_workspace_bytes(cfg), dtype=torch.uint8, device=DEV)
    Xd, gd, bd = X.to(DEV), g.to(DEV), b.to(DEV)
    bpt.ln_fwd(cfg, Xd, gd, bd, Y, mean, rstd)
    bpt.ln_bwd(cfg, Xd, gd, mean, rstd, dY.to(DEV), dX, dg, db, ws)
    torch.cuda.synchronize()
    rY, xhat, rr = layer_norm_fwd(f64(X), f64(g), f64(b), 1e-5)
    rdX, rdg, rdb = layer_norm_bwd(f64(dY), xhat, rr, f64(g))
    for name, got, r in (("Y", Y, rY), ("dX", dX, rdX)):
        if dtype == "f32":
            assert stats(f64(got), r)["e_max"] <= 1e-5, name
        else:   # one rounding to bf16 (half an ulp, 2^-9 relative) of an fp32 result
            d = np.abs(f64(got) - r)
            assert (d <= 2.0 ** -8 * np.abs(r) + 1e-4 * np.sqrt(np.mean(r * r))).all(), name
    for name, got, r in (("dg", dg, rdg), ("db", db, rdb)):      # fp32 outputs
        assert stats(f64(got), r)["e_max"] <= 1e-5, (name, stats(f64(got), r))


def test_gpt_step_f32_with_dropout():
    """fp32 step with residual dropout 0.1 in every layer: layer l of step 0 uses key
    dropout_seed + l, and the oracle given the same keys matches at the fp32 bound."""
    s = GPTShape(L=2, B=2, S=128, D=256, H=4, F=512, V=300, Bq=64, Bkv=64, dtype="f32", dropout=0.1,
                 dropout_seed=0xABCDEF0123)
    say(f"[gpt] dropout {s}")
    m, inp = build(s, 5)
    tok, tgt = inp["tokens"].to(DEV), inp["targets"].to(DEV)
    loss = float(m.forward(tok, tgt).item())
    m.backward(tok, tgt)
    torch.cuda.synchronize()
    P = oracle_params(inp, s)
    for l, lp in enumerate(P.layers):
        lp.dropout, lp.dropout_seed = s.dropout, s.dropout_seed + l
    ref = gpt_fwd_bwd(inp["tokens"].numpy().reshape(s.B, s.S), inp["targets"].numpy().reshape(s.B, s.S), P, s.H)
    assert abs(loss - ref["loss"]) <= 1e-5 * abs(ref["loss"]), (loss, ref["loss"])
    for name, g, r in grad_pairs(m, ref, s):
        st = stats(f64(g), r)
        assert st["e_max"] <= 1e-4, (name, st)
    P0 = oracle_params(inp, s)           # without dropout the loss differs: the masks are live
    assert abs(gpt_fwd_bwd(inp["tokens"].numpy().reshape(s.B, s.S), inp["targets"].numpy().reshape(s.B, s.S),
                           P0, s.H, backward=False)["loss"] - loss) > 1e-4
