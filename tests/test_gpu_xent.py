"""GPU parity of the LM-head cross-entropy (bpt_xent_fwd / bpt_xent_bwd, through the
C ABI) against the float64 oracle (oracle/xent.py) on the same seeded inputs.

Gates (e_max = max|diff| / rms(ref), e_mean = mean|diff| / rms(ref)):
  loss: |diff| <= 1e-5 * |loss| (fp32 accumulation of exact products, fp32 softmax);
  lse:  e_max <= 1e-5;
  fp32 dh, dW: e_max <= 1e-4;
  bf16 dh, dW: e_max <= max(2e-2, F_max x the rounding model's), e_mean <= max(2e-3, F_mean x),
        the model being the oracle with G = (softmax - onehot) / T rounded to bf16 (the
        one matrix-multiply operand the library rounds; h and W are bf16 already); F_max,
        F_mean as for the layer (tests/expected/model_factors.json, derived on the CPU).
"""
import math

import numpy as np
import pytest
import torch

from bpt_inputs import make_xent_inputs
from gpu_util import bf16_limits, say, stats, table
from oracle.bf16_model import to_bf16
from oracle.xent import xent_bwd, xent_fwd
from paper_2305_19370_amd import bpt

pytestmark = pytest.mark.gpu


def run_case(T, D, V, dtype, block_rows, seed, dloss=1.0, bad_target=None):
    ldw = (V + 63) // 64 * 64
    inp = make_xent_inputs(T, D, V, ldw, dtype, seed)
    if bad_target is not None:
        inp["targets"][bad_target] = V
    cfg = bpt.make_xent_config(T, D, V, ldw, block_rows, dtype)
    head = bpt.LMHeadLoss(cfg)
    h, W, y = inp["h"].cuda(), inp["W"].cuda(), inp["targets"].cuda()
    loss, lse = head.forward(h, W, y)
    dh, dW = head.backward(h, W, y, lse, dloss)
    torch.cuda.synchronize()
    gpu = dict(loss=loss.cpu().double().numpy()[0], lse=lse.cpu().double().numpy(),
               dh=dh.float().cpu().double().numpy(), dW=dW.cpu().double().numpy())
    h64, W64, y64 = inp["h"].double().numpy(), inp["W"].double().numpy(), inp["targets"].numpy()
    ref = xent_fwd(h64, W64, y64, V)
    ref.update(xent_bwd(h64, W64, y64, V, g=dloss))
    model = xent_bwd(h64, W64, y64, V, g=dloss, round_g=to_bf16) if dtype == "bf16" else None
    return gpu, ref, model, ldw


def check(gpu, ref, model, dtype, V, label):
    rows, bad = [], []
    if math.isfinite(ref["loss"]):
        err = abs(gpu["loss"] - ref["loss"])
        say(f"[{label}] loss gpu {gpu['loss']:.9f} oracle {ref['loss']:.9f} |diff| {err:.2e}")
        if not err <= 1e-5 * abs(ref["loss"]):
            bad.append("loss")
    s = stats(gpu["lse"], ref["lse"])
    rows.append(("lse", s))
    if not s["e_max"] <= 1e-5:
        bad.append("lse")
    for n in ("dh", "dW"):
        got = gpu[n] if n == "dh" else gpu[n][:, :V]
        s = stats(got, ref[n])
        if dtype == "f32":
            ok = s["e_max"] <= 1e-4
        else:
            ms = stats(model[n], ref[n])
            s["lim_max"], s["lim_mean"] = bf16_limits(ms)
            ok = s["e_max"] <= s["lim_max"] and s["e_mean"] <= s["lim_mean"]
        rows.append((n, s))
        if not ok:
            bad.append(n)
    if "dW" in gpu:
        pad = np.abs(gpu["dW"][:, V:]).max() if gpu["dW"].shape[1] > V else 0.0
        if pad != 0.0:
            bad.append("dW padding columns")
    say(f"[{label}]\n" + table(rows))
    assert not bad, f"{label}: out of tolerance: {bad}"


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_xent_small_ragged(dtype):
    """T not a multiple of the block rows (three blocks, the last of 44 rows), V not a
    multiple of 64 (24 padding columns of W)."""
    T, D, V = 300, 256, 1000
    gpu, ref, model, _ = run_case(T, D, V, dtype, block_rows=128, seed=0, dloss=0.7)
    check(gpu, ref, model, dtype, V, f"xent {dtype} T={T} D={D} V={V} rows=128")


def test_xent_bf16_medium():
    T, D, V = 2048, 1024, 8000
    gpu, ref, model, _ = run_case(T, D, V, "bf16", block_rows=0, seed=1)
    check(gpu, ref, model, "bf16", V, f"xent bf16 T={T} D={D} V={V}")


def test_xent_block_rows_do_not_change_per_token_results():
    """Blocking over tokens changes nothing per token: lse and dh are bitwise equal for
    any block size; dW only by the order in which blocks are summed."""
    T, D, V = 520, 256, 700
    a, ref, model, _ = run_case(T, D, V, "bf16", block_rows=0, seed=2)
    b, _, _, _ = run_case(T, D, V, "bf16", block_rows=96, seed=2)
    assert np.array_equal(a["lse"], b["lse"]) and np.array_equal(a["dh"], b["dh"])
    assert a["loss"] == b["loss"]
    check(b, ref, model, "bf16", V, "xent bf16 rows=96")


def test_xent_target_outside_vocabulary():
    """A target outside [0, V) makes the loss NaN; every per-token lse stays exact, and
    that token's gradient row is the softmax alone (no one-hot term)."""
    T, D, V = 130, 128, 300
    gpu, ref, model, _ = run_case(T, D, V, "f32", block_rows=64, seed=3, bad_target=77)
    assert math.isnan(gpu["loss"]) and math.isnan(ref["loss"])
    check(gpu, ref, model, "f32", V, "xent f32 bad target")
