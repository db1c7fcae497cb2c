"""Helpers shared by the GPU parity tests: run libbpt through the C ABI and the
oracle on the same seeded inputs, and compare tensors."""
from __future__ import annotations

import json
import os
import sys
from typing import Dict

import numpy as np
import torch

import oracle
from bpt_inputs import Workload
from paper_2305_19370_amd import bpt

GRAD_NAMES = ("dWq", "dWk", "dWv", "dWo", "dW1", "dW2", "db1", "db2", "dln1_g", "dln1_b", "dln2_g", "dln2_b")


def say(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def gpu_config(w: Workload, out_dtype: str = "f32", group_blocks: int = 0, **over) -> bpt.Config:
    kw = dict(B=w.B, S=w.S, D=w.D, H=w.H, F=w.F, Bq=w.Bq, Bkv=w.Bkv, causal=w.causal, dtype=w.dtype,
              out_dtype=out_dtype, group_blocks=group_blocks)
    kw.update(over)
    return bpt.make_config(**kw)


def run_gpu(w: Workload, inp: Dict, out_dtype: str = "f32", group_blocks: int = 0, backward: bool = True,
            saved_views: bool = False, qkv_grads: bool = False, **over) -> Dict:
    cfg = gpu_config(w, out_dtype, group_blocks, **over)
    layer = bpt.Layer(cfg)
    dev = {k: (v.cuda() if v is not None else None) for k, v in inp.items()}
    Y, saved = layer.forward(dev["X"], dev)
    out = {"Y": Y}
    if backward:
        dX, grads = layer.backward(dev["X"], dev, saved, dev["dY"], qkv_grads=qkv_grads)
        out["dX"] = dX
        out.update(grads)
    if saved_views:
        out["saved"] = layer.saved_views(saved)
    torch.cuda.synchronize()
    res = {}
    for k, v in out.items():
        if k == "saved":
            res[k] = {n: t.float().cpu() for n, t in v.items()}
        else:
            res[k] = v.float().cpu()
    return res


def run_oracle(w: Workload, inp: Dict, backward: bool = True, activation: str = "gelu"):
    p = oracle.params_from_inputs(inp, activation)
    X = inp["X"].double().numpy()
    Y, cache = oracle.layer_fwd(X, p, w.H, w.causal)
    g = oracle.layer_bwd(cache, p, inp["dY"].double().numpy()) if backward else None
    return Y, cache, g


def bf16_model(w: Workload, inp: Dict, activation: str = "gelu", dropout: float = 0.0,
               dropout_seed: int = 0) -> Dict:
    """The bf16-operand rounding model (oracle/bf16_model.py) on the same inputs."""
    from oracle.bf16_model import bf16_layer_fwd_bwd
    p = oracle.params_from_inputs(inp, activation)
    p.dropout, p.dropout_seed = dropout, dropout_seed
    return bf16_layer_fwd_bwd(inp["X"].double().numpy(), p, w.H, w.causal, inp["dY"].double().numpy())


# ------------------------------------------------------------------ gates (reading R14)
FP32_BOUND = 1e-4                        # stated fp32 bound (max relative error)
BF16_E_MAX, BF16_E_MEAN = 2e-2, 2e-3     # stated bf16 bounds, on errors normalised by rms(ref)
_FACTORS = os.path.join(os.path.dirname(os.path.abspath(__file__)), "expected", "model_factors.json")


def gate_factors() -> Dict[str, float]:
    """F_max, F_mean (bf16: allowed excess over the rounding model's error) and tau (fp32:
    elementwise check over |ref| >= tau rms(ref)), derived on the CPU from rounding models
    only by tests/expected/derive_model_factors.py."""
    with open(_FACTORS) as fh:
        d = json.load(fh)
    return {"F_max": float(d["F_max"]), "F_mean": float(d["F_mean"]), "tau": float(d["fp32"]["tau"])}


def bf16_limits(model_stats: Dict[str, float]):
    f = gate_factors()
    return (max(BF16_E_MAX, f["F_max"] * model_stats["e_max"]),
            max(BF16_E_MEAN, f["F_mean"] * model_stats["e_mean"]))


def fp32_stats(got, ref) -> Dict[str, float]:
    """stats() plus the elementwise relative error over |ref| >= tau rms(ref)."""
    s = stats(got, ref)
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    tau = gate_factors()["tau"]
    big = np.abs(ref) >= tau * s["rms"]
    s["rel_max"] = float((np.abs(got - ref)[big] / np.abs(ref)[big]).max()) if big.any() else 0.0
    s["lim_max"], s["lim_mean"] = FP32_BOUND, float("nan")
    return s


def fp32_ok(s: Dict[str, float]) -> bool:
    """normwise max|diff| <= 1e-4 rms(ref) (which bounds max|diff| / max|ref|) and the
    elementwise relative error <= 1e-4 over |ref| >= tau rms(ref)."""
    return s["e_max"] <= FP32_BOUND and s["rel_max"] <= FP32_BOUND


def stats(got, ref) -> Dict[str, float]:
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    assert np.isfinite(got).all(), "non-finite values in GPU result"
    d = np.abs(got - ref)
    rms = float(np.sqrt(np.mean(ref * ref))) or 1.0
    amax = float(np.abs(ref).max()) or 1.0
    return dict(max_abs=float(d.max()), mean_abs=float(d.mean()), rms=rms, e_max=float(d.max()) / rms,
                e_mean=float(d.mean()) / rms, norm_max=float(d.max()) / amax)


def table(rows) -> str:
    out = [f"{'tensor':10s} {'max_abs':>10s} {'mean_abs':>10s} {'rms':>10s} {'e_max':>9s} {'e_mean':>9s}"
           f" {'lim_max':>9s} {'lim_mean':>9s} {'rel_max':>9s}"]
    for name, s in rows:
        lm = f" {s['lim_max']:9.2e} {s['lim_mean']:9.2e}" if "lim_max" in s else ""
        rel = f" {s['rel_max']:9.2e}" if "rel_max" in s else ""
        out.append(f"{name:10s} {s['max_abs']:10.3e} {s['mean_abs']:10.3e} {s['rms']:10.3e} "
                   f"{s['e_max']:9.2e} {s['e_mean']:9.2e}{lm}{rel}")
    return "\n".join(out)
