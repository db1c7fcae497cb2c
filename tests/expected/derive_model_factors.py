"""Derives the factors of the bf16 parity gates from CPU-only evidence — run on the CPU.

A bf16 gate allows a GPU tensor an error of at most a factor F times what the bf16
rounding model (``oracle/bf16_model.py``: the exact definition with every
matrix-multiply operand rounded to bf16, float64 accumulation) lands at on the same
input. F must cover the difference between two valid bf16-operand implementations
that round at the same operands but accumulate in float32 in different orders. It is
measured here, without the GPU: ``oracle/bf16_tiled.py`` is such an implementation,
blockwise over key tiles in float32, in several variants (tile length, chunked
contractions, lazily moving row maximum, base-2 scores, reversed tile order). For
every input set of the GPU parity tests and every compared tensor, the ratio

    r = e(variant) / e(bf16_model),   e = max|x - ref| / rms(ref)  (and the mean analogue)

is recorded, ref being the float64 oracle. The factor is the larger of the largest
ratio seen and exp(mu + 4 sigma) of the log-ratios (mu, sigma over the whole ensemble):
a four-standard-deviation bound on a further implementation's ratio, so that across the
few hundred tensor checks of the GPU suite a valid implementation fails one with a
probability of about one percent. Results go to ``model_factors.json`` beside this file.

    python tests/expected/derive_model_factors.py [--quick]

Only ``oracle/`` and the input generator are used; nothing comes from the HIP path.
"""
from __future__ import annotations

import json
import math
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

OUT = os.path.join(HERE, "model_factors.json")
TENSORS = ("Y", "O", "lse", "Hd", "dX", "dQ", "dK", "dV", "dWq", "dWk", "dWv", "dWo", "dW1", "dW2", "db1",
           "db2", "dln1_g", "dln1_b", "dln2_g", "dln2_b")
VARIANTS = {
    "t64": dict(kv_tile=64),
    "t128_c512_lazy_b2_rev": dict(kv_tile=128, k_chunk=512, lazy=True, base2=True, reverse=True),
    "t32_c256_b2": dict(kv_tile=32, k_chunk=256, base2=True),
    "t256_c64_lazy_rev": dict(kv_tile=256, k_chunk=64, lazy=True, reverse=True),
}
# the input sets of the bf16 GPU parity tests: (name, workload kwargs, make_inputs kwargs, extras)
CASES = [
    ("ragged_s250_h2_c", dict(B=2, S=250, D=256, H=2, F=512, causal=True), dict(seed=2, affine=True, biases=True), {}),
    ("ragged_s250_h2_nc", dict(B=2, S=250, D=256, H=2, F=512, causal=False), dict(seed=2, affine=True, biases=True), {}),
    ("ragged_s700_h4_c", dict(B=2, S=700, D=256, H=4, F=512, causal=True), dict(seed=2, affine=True, biases=True), {}),
    ("ragged_s700_h4_nc", dict(B=2, S=700, D=256, H=4, F=512, causal=False), dict(seed=2, affine=True, biases=True), {}),
    ("relu_s250", dict(B=2, S=250, D=256, H=2, F=512, causal=True), dict(seed=8, affine=True, biases=True),
     {"activation": "relu"}),
    ("large_scores_c", dict(B=1, S=700, D=256, H=2, F=512, causal=True), dict(seed=7), {"wq_scale": 16}),
    ("large_scores_nc", dict(B=1, S=700, D=256, H=2, F=512, causal=False), dict(seed=7), {"wq_scale": 16}),
    ("saved_s333", dict(B=2, S=333, D=512, H=4, F=1024, causal=True), dict(seed=3, affine=True, biases=True), {}),
    ("blocks_s1000", dict(B=1, S=1000, D=256, H=2, F=512, causal=True), dict(seed=4), {}),
    ("dropout_s250", dict(B=2, S=250, D=256, H=2, F=512, causal=True), dict(seed=9, affine=True, biases=True),
     {"dropout": 0.1}),
    ("short_s1", dict(B=2, S=1, D=256, H=2, F=512, causal=True), dict(seed=21, affine=True, biases=True), {}),
    ("short_s7", dict(B=2, S=7, D=256, H=2, F=512, causal=True), dict(seed=27, affine=True, biases=True), {}),
    ("short_s63", dict(B=2, S=63, D=256, H=2, F=512, causal=True), dict(seed=83, affine=True, biases=True), {}),
    ("bq1_s70", dict(B=1, S=70, D=256, H=2, F=512, causal=True), dict(seed=13, affine=True, biases=True), {}),
    ("b3_dh64_s190", dict(B=3, S=190, D=256, H=4, F=512, causal=True), dict(seed=11, affine=True, biases=True), {}),
    ("s96_b2", dict(B=2, S=96, D=256, H=2, F=512, causal=True), dict(seed=12), {}),
    ("s160_b2", dict(B=2, S=160, D=256, H=2, F=512, causal=True), dict(seed=12), {}),
    ("repeat_s700", dict(B=2, S=700, D=256, H=4, F=512, causal=True), dict(seed=10, affine=True, biases=True), {}),
    ("smoke_s200", dict(B=1, S=200, D=256, H=2, F=512, causal=True), dict(seed=0), {}),
    ("ksplit_s512_b2", dict(B=2, S=512, D=256, H=2, F=1024, causal=True), dict(seed=14, affine=True, biases=True), {}),
]
FULL_CASES = [("workload_1b_s4096", "bf16_1b_s4096", dict(seed=0), {})]
# the input sets of the fp32 GPU parity tests
FP32_CASES = [
    ("f32_ragged_s250_h4_c", dict(B=2, S=250, D=256, H=4, F=512, causal=True), dict(seed=1, affine=True, biases=True), {}),
    ("f32_ragged_s250_h4_nc", dict(B=2, S=250, D=256, H=4, F=512, causal=False), dict(seed=1, affine=True, biases=True), {}),
    ("f32_ragged_s250_h2_c", dict(B=2, S=250, D=256, H=2, F=512, causal=True), dict(seed=1, affine=True, biases=True), {}),
    ("f32_ragged_s250_h2_nc", dict(B=2, S=250, D=256, H=2, F=512, causal=False), dict(seed=1, affine=True, biases=True), {}),
    ("f32_relu_s250", dict(B=2, S=250, D=256, H=2, F=512, causal=True), dict(seed=8, affine=True, biases=True),
     {"activation": "relu"}),
    ("f32_dropout_s250", dict(B=2, S=250, D=256, H=2, F=512, causal=True), dict(seed=9, affine=True, biases=True),
     {"dropout": 0.1}),
    ("f32_short_s1", dict(B=2, S=1, D=256, H=2, F=512, causal=True), dict(seed=21, affine=True, biases=True), {}),
    ("f32_short_s7", dict(B=2, S=7, D=256, H=2, F=512, causal=True), dict(seed=27, affine=True, biases=True), {}),
    ("f32_short_s63", dict(B=2, S=63, D=256, H=2, F=512, causal=True), dict(seed=83, affine=True, biases=True), {}),
    ("f32_s96_b2", dict(B=2, S=96, D=256, H=2, F=512, causal=True), dict(seed=12), {}),
    ("f32_s160_b2", dict(B=2, S=160, D=256, H=2, F=512, causal=True), dict(seed=12), {}),
    ("f32_ksplit_s512_b2", dict(B=2, S=512, D=256, H=2, F=1024, causal=True), dict(seed=14, affine=True, biases=True),
     {}),
]
FP32_FULL_CASES = [("f32_workload_s512", "fp32_s512_d256", dict(seed=0), {})]
FP32_VARIANTS = {
    "t64": dict(kv_tile=64, round_operands=False),
    "t128_c512_lazy_rev": dict(kv_tile=128, k_chunk=512, lazy=True, reverse=True, round_operands=False),
    "t32_c256": dict(kv_tile=32, k_chunk=256, round_operands=False),
}
# candidate thresholds tau of the fp32 elementwise check (elements with |ref| >= tau * rms(ref))
TAUS = (0.01, 0.02, 0.05, 0.1, 0.2, 0.3, 0.5)
FP32_BOUND, FP32_MARGIN = 1e-4, 4.0
DROPOUT_SEED = 0x0123456789ABCDEF


def case_inputs(wkw, ikw, extra, workload=None, dtype="bf16"):
    import oracle
    from bpt_inputs import WORKLOADS, make_inputs, small_workload
    w = WORKLOADS[workload] if workload else small_workload(dtype, **wkw)
    inp = make_inputs(w, **ikw)
    if extra.get("wq_scale"):
        inp["Wq"] = (inp["Wq"].float() * extra["wq_scale"]).to(inp["Wq"].dtype)
    p = oracle.params_from_inputs(inp, extra.get("activation", "gelu"))
    if extra.get("dropout"):
        p.dropout, p.dropout_seed = extra["dropout"], DROPOUT_SEED
    return w, inp["X"].double().numpy(), p, inp["dY"].double().numpy()


def errs(got, ref):
    got, ref = np.asarray(got, dtype=np.float64), np.asarray(ref, dtype=np.float64)
    d = np.abs(got - ref)
    r = float(np.sqrt(np.mean(ref * ref))) or 1.0
    return float(d.max()) / r, float(d.mean()) / r


def case_ratios(w, X, p, dY, variants=VARIANTS):
    """{tensor: {"model": [e_max, e_mean], variant: [ratio_max, ratio_mean], ...}}"""
    import oracle
    from oracle.bf16_model import bf16_layer_fwd_bwd
    from oracle.bf16_tiled import tiled_layer_fwd_bwd
    Y, cache = oracle.layer_fwd(X, p, w.H, w.causal)
    ref = oracle.layer_bwd(cache, p, dY)
    ref.update(Y=Y, O=cache["O"], lse=cache["lse"], Hd=cache["Hd"])
    m1 = bf16_layer_fwd_bwd(X, p, w.H, w.causal, dY)
    out = {}
    for t in TENSORS:
        if ref.get(t) is None or m1.get(t) is None:
            continue
        e1 = errs(m1[t], ref[t])
        if min(e1) < 1e-9:          # no rounding reaches it (db2 = sum of the bf16 dY): no ratio
            continue
        out[t] = {"model": list(e1)}
    for vn, kw in variants.items():
        m2 = tiled_layer_fwd_bwd(X, p, w.H, w.causal, dY, **kw)
        for t in out:
            e2 = errs(m2[t], ref[t])
            out[t][vn] = [e2[0] / out[t]["model"][0], e2[1] / out[t]["model"][1]]
    return out


def factors(all_ratios):
    """(F_max, F_mean) and the ensemble statistics from {case: case_ratios(...)}."""
    res = {}
    for j, stat in enumerate(("max", "mean")):
        lr = np.array([math.log(v[j]) for cr in all_ratios.values() for t in cr.values()
                       for k, v in t.items() if k != "model"])
        mu, sd = float(lr.mean()), float(lr.std())
        hi = float(np.exp(lr.max()))
        f = max(hi, math.exp(mu + 4.0 * sd))
        res[stat] = {"n": int(lr.size), "log_mean": mu, "log_std": sd, "largest_ratio": hi,
                     "smallest_ratio": float(np.exp(lr.min())), "four_sigma": math.exp(mu + 4.0 * sd),
                     "factor": math.ceil(f * 100) / 100}
    return res


def fp32_elementwise(w, X, p, dY):
    """For each fp32 CPU variant and tensor: the normwise error max|d| / rms(ref) and, per
    threshold tau, the largest elementwise relative error over elements |ref| >= tau rms."""
    import oracle
    from oracle.bf16_tiled import tiled_layer_fwd_bwd
    Y, cache = oracle.layer_fwd(X, p, w.H, w.causal)
    ref = oracle.layer_bwd(cache, p, dY)
    ref["Y"] = Y
    out = {}
    for vn, kw in FP32_VARIANTS.items():
        m = tiled_layer_fwd_bwd(X, p, w.H, w.causal, dY, **kw)
        for t in ("Y", "dX", "dQ", "dK", "dV", "dWq", "dWk", "dWv", "dWo", "dW1", "dW2", "db1", "db2", "dln1_g",
                  "dln1_b", "dln2_g", "dln2_b"):
            if ref.get(t) is None:
                continue
            r = np.asarray(ref[t], dtype=np.float64)
            d = np.abs(np.asarray(m[t], dtype=np.float64) - r)
            rms = float(np.sqrt(np.mean(r * r))) or 1.0
            rel = {}
            for tau in TAUS:
                big = np.abs(r) >= tau * rms
                rel[str(tau)] = float((d[big] / np.abs(r[big])).max()) if big.any() else 0.0
            out.setdefault(t, {})[vn] = {"e_max": float(d.max()) / rms, "rel": rel}
    return out


def fp32_threshold(all_fp32):
    """The smallest tau at which every fp32 CPU variant meets the elementwise bound with
    the margin: largest relative error <= FP32_BOUND / FP32_MARGIN."""
    worst = {str(t): max(v["rel"][str(t)] for cr in all_fp32.values() for tv in cr.values() for v in tv.values())
             for t in TAUS}
    ok = [t for t in TAUS if worst[str(t)] <= FP32_BOUND / FP32_MARGIN]
    e_max = max(v["e_max"] for cr in all_fp32.values() for tv in cr.values() for v in tv.values())
    return (min(ok) if ok else None), worst, e_max


def main(quick: bool = False) -> None:
    t0 = time.time()
    all_fp32 = {}
    for name, wkw, ikw, extra in FP32_CASES:
        w, X, p, dY = case_inputs(wkw, ikw, extra, dtype="f32")
        all_fp32[name] = fp32_elementwise(w, X, p, dY)
    for name, wl, ikw, extra in FP32_FULL_CASES:
        w, X, p, dY = case_inputs(None, ikw, extra, workload=wl)
        all_fp32[name] = fp32_elementwise(w, X, p, dY)
    tau, worst, e32 = fp32_threshold(all_fp32)
    print(f"fp32: tau {tau}, worst relative error per tau {worst}, largest normwise {e32:.2e}", flush=True)
    all_ratios = {}
    for name, wkw, ikw, extra in CASES:
        w, X, p, dY = case_inputs(wkw, ikw, extra)
        all_ratios[name] = case_ratios(w, X, p, dY)
        print(f"{name}: {time.time() - t0:.0f} s", flush=True)
    if not quick:
        for name, wl, ikw, extra in FULL_CASES:
            w, X, p, dY = case_inputs(None, ikw, extra, workload=wl)
            all_ratios[name] = case_ratios(w, X, p, dY)
            print(f"{name}: {time.time() - t0:.0f} s", flush=True)
    f = factors(all_ratios)
    doc = {"description": "bf16 parity-gate factors over the rounding model, from CPU rounding models only "
                          "(tests/expected/derive_model_factors.py)",
           "variants": {k: v for k, v in VARIANTS.items()}, "F_max": f["max"]["factor"],
           "F_mean": f["mean"]["factor"], "stats": f, "ratios": all_ratios,
           "fp32": {"tau": tau, "bound": FP32_BOUND, "margin": FP32_MARGIN, "worst_rel_per_tau": worst,
                    "largest_normwise": e32, "variants": FP32_VARIANTS, "cases": all_fp32}}
    with open(OUT, "w") as fh:
        json.dump(doc, fh, indent=1)
    print(json.dumps({"F_max": doc["F_max"], "F_mean": doc["F_mean"], "stats": f, "fp32_tau": tau}, indent=1))


if __name__ == "__main__":
    main(quick="--quick" in sys.argv)
