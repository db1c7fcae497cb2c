"""Helpers shared by the GPU parity tests: run libbpt through the C ABI and the
oracle on the same seeded inputs, and compare tensors."""
from __future__ import annotations

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
            saved_views: bool = False, **over) -> Dict:
    cfg = gpu_config(w, out_dtype, group_blocks, **over)
    layer = bpt.Layer(cfg)
    dev = {k: (v.cuda() if v is not None else None) for k, v in inp.items()}
    Y, saved = layer.forward(dev["X"], dev)
    out = {"Y": Y}
    if backward:
        dX, grads = layer.backward(dev["X"], dev, saved, dev["dY"])
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


def bf16_model(w: Workload, inp: Dict, activation: str = "gelu") -> Dict:
    """The bf16-operand rounding model (oracle/bf16_model.py) on the same inputs."""
    from oracle.bf16_model import bf16_layer_fwd_bwd
    p = oracle.params_from_inputs(inp, activation)
    return bf16_layer_fwd_bwd(inp["X"].double().numpy(), p, w.H, w.causal, inp["dY"].double().numpy())


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
           f" {'lim_max':>9s} {'lim_mean':>9s}"]
    for name, s in rows:
        lm = f" {s['lim_max']:9.2e} {s['lim_mean']:9.2e}" if "lim_max" in s else ""
        out.append(f"{name:10s} {s['max_abs']:10.3e} {s['mean_abs']:10.3e} {s['rms']:10.3e} "
                   f"{s['e_max']:9.2e} {s['e_mean']:9.2e}{lm}")
    return "\n".join(out)
