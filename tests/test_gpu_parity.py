"""GPU parity: libbpt (through the C ABI) against the float64 oracle on the same
seeded inputs. Shapes span several tiles with ragged tails; both causal and
non-causal; fp32 and bf16 paths; LayerNorm affine parameters and FFN biases on.

Gates (written in tests/gpu_util.py; e_max = max|diff| / rms(ref), e_mean =
mean|diff| / rms(ref), with ref the float64 oracle):
  fp32: e_max <= 1e-4 for every output and gradient (max|diff| <= 1e-4 rms(ref), which
        also bounds the normwise relative error max|diff| / max|ref|), and the
        elementwise relative error |diff| / |ref| <= 1e-4 on every element with
        |ref| >= tau rms(ref);
  bf16: e_max <= max(2e-2, F_max x e_max of the bf16 rounding model) and
        e_mean <= max(2e-3, F_mean x e_mean of the rounding model), per tensor.
        The rounding model (oracle/bf16_model.py) is the same definition with every
        matrix-multiply operand rounded to bf16: what any bf16-operand implementation
        lands at on this input. For most tensors the first term decides; the weight
        gradients and, with the causal mask, dX carry a bf16 floor above 2e-2 / 2e-3.
tau, F_max and F_mean come from tests/expected/model_factors.json, derived on the CPU
from rounding models only (tests/expected/derive_model_factors.py): F covers the
spread between bf16-operand implementations that accumulate in float32 in different
orders, tau is where float32 implementations meet the elementwise bound.
"""
import math

import numpy as np
import pytest
import torch

from bpt_inputs import WORKLOADS, make_inputs, small_workload
from gpu_util import (GRAD_NAMES, bf16_limits, bf16_model, fp32_ok, fp32_stats, run_gpu, run_oracle, say, stats,
                      table)
import oracle

pytestmark = pytest.mark.gpu

QKV_GRADS = ("dQ", "dK", "dV")


def compare_all(w, inp, gpu, Yr, g, tol_kind, label, activation="gelu", dropout=0.0, dropout_seed=0):
    rows, bad = [], []
    names = ["Y", "dX"] + [n for n in GRAD_NAMES + QKV_GRADS if n in gpu]
    model = bf16_model(w, inp, activation, dropout, dropout_seed) if tol_kind == "bf16" else None
    for n in names:
        ref = Yr if n == "Y" else g[n]
        if tol_kind == "fp32":
            s = fp32_stats(gpu[n].numpy(), ref)
            ok = fp32_ok(s)
        else:
            s = stats(gpu[n].numpy(), ref)
            ms = stats(model[n], ref)
            lim_max, lim_mean = bf16_limits(ms)
            s["lim_max"], s["lim_mean"] = lim_max, lim_mean
            ok = s["e_max"] <= lim_max and s["e_mean"] <= lim_mean
        rows.append((n, s))
        if not ok:
            bad.append(n)
    say(f"\n[{label}]\n" + table(rows))
    assert not bad, f"{label}: out of tolerance: {bad}"


@pytest.mark.parametrize("causal", [True, False])
@pytest.mark.parametrize("H", [4, 2])          # head dim 64 and 128
def test_fp32_small_ragged(causal, H):
    w = small_workload("f32", B=2, S=250, D=256, H=H, F=512, causal=causal, Bq=64, Bkv=64)
    inp = make_inputs(w, seed=1, affine=True, biases=True)
    say(f"case fp32 small {w.name}")
    gpu = run_gpu(w, inp, group_blocks=2, qkv_grads=True)
    Yr, _, g = run_oracle(w, inp)
    compare_all(w, inp, gpu, Yr, g, "fp32", w.name)


def test_fp32_workload_s512():
    w = WORKLOADS["fp32_s512_d256"]
    inp = make_inputs(w, seed=0)
    say(f"case {w.name}")
    gpu = run_gpu(w, inp)
    Yr, _, g = run_oracle(w, inp)
    compare_all(w, inp, gpu, Yr, g, "fp32", w.name)


@pytest.mark.parametrize("causal", [True, False])
@pytest.mark.parametrize("S,H", [(250, 2), (700, 4)])
def test_bf16_small_ragged(causal, S, H):
    """Every output and gradient, and the attention backward's own outputs dQ, dK, dV
    (kernel-level parity of the backward of Section 3: P rebuilt from the log-sum-exp)."""
    w = small_workload("bf16", B=2, S=S, D=256, H=H, F=512, causal=causal, Bq=128, Bkv=128)
    inp = make_inputs(w, seed=2, affine=True, biases=True)
    say(f"case bf16 small {w.name}")
    gpu = run_gpu(w, inp, group_blocks=2, qkv_grads=True)
    Yr, _, g = run_oracle(w, inp)
    compare_all(w, inp, gpu, Yr, g, "bf16", w.name)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_relu_ffn_with_biases(dtype):
    """Eq. (2)'s FFN as printed: ReLU with both biases (the GELU of GPT models is the
    default activation)."""
    w = small_workload(dtype, B=2, S=250, D=256, H=2, F=512, causal=True, Bq=64, Bkv=64)
    inp = make_inputs(w, seed=8, affine=True, biases=True)
    say(f"case relu {w.name}")
    gpu = run_gpu(w, inp, group_blocks=2, activation="relu")
    Yr, _, g = run_oracle(w, inp, activation="relu")
    compare_all(w, inp, gpu, Yr, g, "fp32" if dtype == "f32" else "bf16", w.name + "_relu", activation="relu")


@pytest.mark.parametrize("causal", [True, False])
def test_bf16_large_scores(causal):
    """Scores far above the first key tile's maximum. Wq scaled by 16 (exact in bf16)
    puts the scores' spread at ~23 octaves: the softmax is nearly one-hot and later key
    tiles raise a row's maximum by more than 11 octaves hundreds of times (counted on
    the oracle's Q, K), so the forward leaves its fast path and rescales."""
    w = small_workload("bf16", B=1, S=700, D=256, H=2, F=512, causal=causal, Bq=128, Bkv=128)
    inp = make_inputs(w, seed=7)
    inp["Wq"] = (inp["Wq"].float() * 16).to(inp["Wq"].dtype)
    say(f"case bf16 large scores {w.name}")
    gpu = run_gpu(w, inp, qkv_grads=True)
    Yr, _, g = run_oracle(w, inp)
    compare_all(w, inp, gpu, Yr, g, "bf16", w.name + "_x16")


def test_bf16_saved_intermediates():
    """Kernel-level parity on what the forward saves: Q, K, V (projection GEMM),
    O and log-sum-exp (attention), h (output projection + residual), LN statistics."""
    w = small_workload("bf16", B=2, S=333, D=512, H=4, F=1024, causal=True, Bq=100, Bkv=100)
    inp = make_inputs(w, seed=3, affine=True, biases=True)
    say(f"case saved {w.name}")
    gpu = run_gpu(w, inp, backward=False, saved_views=True, group_blocks=1)
    Yr, c, _ = run_oracle(w, inp, backward=False)
    sv = gpu["saved"]
    B, S, D, H = w.B, w.S, w.D, w.H
    qkv = sv["qkv"]
    # the bf16 path stores Q multiplied by log2(e)/sqrt(dh) (the scores' base-2 scale)
    qscale = math.log2(math.e) / math.sqrt(D // H)
    checks = {
        "Q": (qkv[:, :D].reshape(B, S, D) / qscale, c["Q"]),
        "K": (qkv[:, D:2 * D].reshape(B, S, D), c["K"]),
        "V": (qkv[:, 2 * D:].reshape(B, S, D), c["V"]),
        "O": (sv["o"].reshape(B, S, D), c["O"]),
        "lse": (sv["lse"][:, :, :S], c["lse"]),
        "h": (sv["h"].reshape(B, S, D), c["Hd"]),
        "mu1": (sv["mu1"].reshape(B, S), c["X"].mean(-1)),
        "rstd1": (sv["rstd1"].reshape(B, S), c["rstd1"][..., 0]),
        "rstd2": (sv["rstd2"].reshape(B, S), c["rstd2"][..., 0]),
        "Y": (gpu["Y"], Yr),
    }
    model = bf16_model(w, inp)
    model_of = {"O": model["O"], "lse": model["lse"], "h": model["Hd"], "Y": model["Y"]}
    rows, bad = [], []
    for n, (got, ref) in checks.items():
        s = stats(got.numpy(), ref)
        lim_max, lim_mean = 2e-2, 2e-3
        if n in model_of:
            lim_max, lim_mean = bf16_limits(stats(model_of[n], ref))
        s["lim_max"], s["lim_mean"] = lim_max, lim_mean
        rows.append((n, s))
        if not (s["e_max"] <= lim_max and s["e_mean"] <= lim_mean):
            bad.append(n)
    say("\n" + table(rows))
    assert not bad, bad


@pytest.mark.parametrize("Bq,Bkv,groups", [(128, 128, 1), (64, 32, 3), (333, 333, 1), (1000, 7, 1)])
def test_bf16_block_sizes(Bq, Bkv, groups):
    """Bq / Bkv / FFN grouping change the result only through rounding."""
    w = small_workload("bf16", B=1, S=1000, D=256, H=2, F=512, causal=True, Bq=Bq, Bkv=Bkv)
    inp = make_inputs(w, seed=4)
    say(f"case blocks Bq={Bq} Bkv={Bkv} groups={groups}")
    gpu = run_gpu(w, inp, group_blocks=groups)
    Yr, _, g = run_oracle(w, inp)
    compare_all(w, inp, gpu, Yr, g, "bf16", f"Bq={Bq},Bkv={Bkv},g={groups}")


def test_bf16_output_is_rounded_fp32_output():
    """A bf16 Y / dX is the fp32 result rounded to nearest even (same kernels, other store)."""
    w = small_workload("bf16", B=2, S=300, D=256, H=2, F=512, causal=True)
    inp = make_inputs(w, seed=5)
    a = run_gpu(w, inp, out_dtype="f32")
    b = run_gpu(w, inp, out_dtype="bf16")
    for n in ("Y", "dX"):
        assert torch.equal(a[n].to(torch.bfloat16).float(), b[n]), n
    for n in ("dWq", "dW1", "dW2"):
        assert torch.equal(a[n], b[n]), n


def test_causality_and_determinism():
    w = small_workload("bf16", B=1, S=512, D=256, H=2, F=512, causal=True)
    inp = make_inputs(w, seed=6)
    a = run_gpu(w, inp, backward=False)
    a2 = run_gpu(w, inp, backward=False)
    assert torch.equal(a["Y"], a2["Y"]), "forward is not bitwise repeatable"
    t = 300
    inp2 = dict(inp)
    X2 = inp["X"].clone()
    X2[:, t:] = torch.randn(X2[:, t:].shape, generator=torch.Generator().manual_seed(9)).to(X2.dtype)
    inp2["X"] = X2
    b = run_gpu(w, inp2, backward=False)
    assert torch.equal(a["Y"][:, :t], b["Y"][:, :t]), "future tokens changed past outputs"
    assert not torch.equal(a["Y"][:, t:], b["Y"][:, t:])


def test_backward_repeatable():
    """Two backward passes on the same inputs give bitwise identical outputs (every
    kernel of the backward is deterministic: no atomics, fixed reduction orders)."""
    w = small_workload("bf16", B=2, S=700, D=256, H=4, F=512, causal=True, Bq=128, Bkv=128)
    inp = make_inputs(w, seed=10, affine=True, biases=True)
    say(f"case repeat {w.name}")
    a = run_gpu(w, inp, group_blocks=2, qkv_grads=True)
    b = run_gpu(w, inp, group_blocks=2, qkv_grads=True)
    diff = [n for n in a if not torch.equal(a[n], b[n])]
    assert not diff, f"not bitwise repeatable: {diff}"


@pytest.mark.parametrize("dtype,S", [("bf16", 1), ("bf16", 7), ("bf16", 63), ("f32", 1), ("f32", 7), ("f32", 63)])
def test_short_sequences(dtype, S):
    """S below one 64-row tile (a single partial tile; S = 1 makes attention O = V): the
    ragged paths of every kernel, with two sequences so the batch offset is exercised."""
    w = small_workload(dtype, B=2, S=S, D=256, H=2, F=512, causal=True, Bq=S, Bkv=S)
    inp = make_inputs(w, seed=20 + S, affine=True, biases=True)
    say(f"case short {w.name}")
    gpu = run_gpu(w, inp, qkv_grads=True)
    Yr, _, g = run_oracle(w, inp)
    compare_all(w, inp, gpu, Yr, g, "fp32" if dtype == "f32" else "bf16", w.name)


def test_bf16_query_block_of_one():
    """Bq = 1 with one query block per FFN group: every group is a single token."""
    w = small_workload("bf16", B=1, S=70, D=256, H=2, F=512, causal=True, Bq=1, Bkv=1)
    inp = make_inputs(w, seed=13, affine=True, biases=True)
    say(f"case Bq=1 {w.name}")
    gpu = run_gpu(w, inp, group_blocks=1)
    Yr, _, g = run_oracle(w, inp)
    compare_all(w, inp, gpu, Yr, g, "bf16", w.name + "_bq1")


def test_bf16_heads_not_multiple_of_8_dh64():
    """B = 3, H = 4 (dh = 64): B*H = 12 heads are not a multiple of the 8 XCDs, so the
    attention kernels take their plain workgroup order."""
    w = small_workload("bf16", B=3, S=190, D=256, H=4, F=512, causal=True, Bq=64, Bkv=64)
    inp = make_inputs(w, seed=11, affine=True, biases=True)
    say(f"case B3 dh64 {w.name}")
    gpu = run_gpu(w, inp, qkv_grads=True)
    Yr, _, g = run_oracle(w, inp)
    compare_all(w, inp, gpu, Yr, g, "bf16", w.name)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("S", [96, 160])
def test_sequence_of_32_mod_64(dtype, S):
    """S % 64 == 32: the output-projection weight gradient takes its per-sequence form
    (O and dh both read token-major, contraction over exactly S tokens)."""
    w = small_workload(dtype, B=2, S=S, D=256, H=2, F=512, causal=True, Bq=32, Bkv=32)
    inp = make_inputs(w, seed=12, affine=False, biases=False)
    say(f"case S%64==32 {w.name}")
    gpu = run_gpu(w, inp)
    Yr, _, g = run_oracle(w, inp)
    compare_all(w, inp, gpu, Yr, g, "fp32" if dtype == "f32" else "bf16", w.name)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("groups", [0, 2])
def test_weight_gradients_split_along_tokens(dtype, groups):
    """D = 256, F = 1024, S = 512: the weight-gradient tile grids are small, so the
    contractions over tokens run in slices summed in a fixed order. The D x D gradients
    take 16 slices of 64 tokens over the whole batch; dW1 and dW2 take 16 slices of the
    group's rows with automatic grouping (one group) and 4 slices per group of two
    128-row query blocks, each group's sum added to the previous groups'."""
    w = small_workload(dtype, B=2, S=512, D=256, H=2, F=1024, causal=True, Bq=128, Bkv=128)
    inp = make_inputs(w, seed=14, affine=True, biases=True)
    say(f"case token-split weight gradients {w.name} groups={groups}")
    gpu = run_gpu(w, inp, group_blocks=groups)
    Yr, _, g = run_oracle(w, inp)
    compare_all(w, inp, gpu, Yr, g, "fp32" if dtype == "f32" else "bf16", f"{w.name} groups={groups}")


def test_bf16_workload_1b_s4096():
    """The full 1B-shaped workload (B=2, S=4096, D=2048, H=16, F=8192), every output
    and gradient, and dQ, dK, dV, against the unblocked fp64 oracle."""
    w = WORKLOADS["bf16_1b_s4096"]
    inp = make_inputs(w, seed=0)
    say(f"case {w.name}")
    gpu = run_gpu(w, inp, qkv_grads=True)
    Yr, _, g = run_oracle(w, inp)
    compare_all(w, inp, gpu, Yr, g, "bf16", w.name)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_residual_dropout(dtype):
    """Dropout (rate 0.1) on both residual branches: the GPU regenerates the oracle's
    Philox masks exactly (a wrong mask shows as O(1) errors), ragged groups over two
    sequences so the token index crosses group and sequence boundaries. Gated like every
    other case: the fp32 gate, or the bf16 gate over the rounding model run with the
    same dropout masks."""
    w = small_workload(dtype, B=2, S=250, D=256, H=2, F=512, causal=True, Bq=64, Bkv=64)
    inp = make_inputs(w, seed=9, affine=True, biases=True)
    p, seed = 0.1, 0x0123456789ABCDEF
    say(f"case dropout {w.name} p={p}")
    gpu = run_gpu(w, inp, group_blocks=2, dropout=p, dropout_seed=seed)
    prm = oracle.params_from_inputs(inp)
    prm.dropout, prm.dropout_seed = p, seed
    Yr, cache = oracle.layer_fwd(inp["X"].double().numpy(), prm, w.H, w.causal)
    g = oracle.layer_bwd(cache, prm, inp["dY"].double().numpy())
    compare_all(w, inp, gpu, Yr, g, "fp32" if dtype == "f32" else "bf16", w.name + "_dropout",
                dropout=p, dropout_seed=seed)
