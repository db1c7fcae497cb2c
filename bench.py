#!/usr/bin/env python3
"""One-GPU benchmark of the Blockwise Parallel Transformer layer (libbpt).

A step is one forward (training mode, saving activations) plus one backward of
the layer on one batch of synthetic seeded input, all through libbpt's HIP
kernels. Default workload: the 7B-shaped layer (B=1, S=32768, D=4096, H=32,
dh=128, F=16384, causal, Bq=Bkv=1024, bf16 operands with fp32 accumulation).

Prints ONE JSON line:
  value       model TFLOP/s of fwd+bwd, with model FLOP = 3 x fwd and
              fwd = 8 B S D^2 + 4 B S D F + 2 B D S (S+1)   (causal)
  roofline    the launch class with the largest total time, its algorithmic
              flops (or bytes) per unit time measured with HIP events around
              each of its launches in the timed steps, against MI355X peak
  cpu_baseline  the float64 CPU oracle on a bounded sample of the same layer
              shape (shorter sequence), same FLOP convention
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 MFMA
PEAK_FP32_TFLOPS = 157.3
PEAK_HBM_GBS = 8000.0


def model_flops_fwd(B, S, D, F, causal=True):
    attn = 2 * B * D * S * (S + 1) if causal else 4 * B * S * S * D
    return 8 * B * S * D * D + 4 * B * S * D * F + attn


def cpu_baseline(w, sample_S: int):
    """Time the float64 oracle (untuned) on [B=1, S=sample_S] of the workload's layer shape."""
    import numpy as np
    import oracle
    from bpt_inputs import make_inputs
    try:
        from threadpoolctl import threadpool_info
        threads = max([int(i.get("num_threads", 0)) for i in threadpool_info()] + [1])
    except Exception:  # pragma: no cover
        threads = len(os.sched_getaffinity(0))
    ws = w.with_(B=1, S=sample_S, Bq=min(w.Bq, sample_S), Bkv=min(w.Bkv, sample_S), name=w.name + "_sample")
    inp = make_inputs(ws, seed=0)
    p = oracle.params_from_inputs(inp)
    X, dY = inp["X"].double().numpy(), inp["dY"].double().numpy()
    t0 = time.perf_counter()
    Y, cache = oracle.layer_fwd(X, p, ws.H, ws.causal)
    g = oracle.layer_bwd(cache, p, dY)
    dt = time.perf_counter() - t0
    assert np.isfinite(Y).all() and np.isfinite(g["dX"]).all()
    fl = 3 * model_flops_fwd(1, sample_S, ws.D, ws.F, ws.causal)
    return {"value": fl / dt / 1e12, "unit": "TFLOP/s", "cores": threads, "kind": "oracle",
            "sample": f"fwd+bwd of one sequence of {sample_S} tokens of the same layer shape "
                      f"(D={ws.D}, H={ws.H}, F={ws.F}, causal), float64 numpy, {dt:.1f} s",
            "seconds": dt, "host": host_cpu_info(threads)}


# Sources whose every byte defines a launch class's kernel, and the compile flags of its
# translation unit: a recorded HBM-traffic measurement of that class applies only while
# their hash is unchanged.
TRAFFIC_SOURCES = {
    cls: ["paper_2305_19370_amd/csrc/" + f, "paper_2305_19370_amd/csrc/attn_common.h",
          "paper_2305_19370_amd/csrc/common.h", "paper_2305_19370_amd/csrc/internal.h"]
    for cls, f in (("attn.bwd_dkdv", "attn_bwd_dkdv.hip"), ("attn.bwd_dq", "attn_bwd_dq.hip"),
                   ("attn.fwd", "attn_fwd.hip"))
}
TRAFFIC_RECORD = os.path.join(ROOT, "profiles", "attn_kernels_7b_s32768_hbm_traffic.md")


def source_hash(cls: str):
    import hashlib
    from paper_2305_19370_amd import build
    if cls not in TRAFFIC_SOURCES:
        return None
    h = hashlib.sha256()
    for f in TRAFFIC_SOURCES[cls]:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    unit = os.path.basename(TRAFFIC_SOURCES[cls][0])
    flags = build.HIP_FLAGS + build.EXTRA_FLAGS.get(unit, [])
    flags = [f for i, f in enumerate(flags) if f != "-I" and (i == 0 or flags[i - 1] != "-I")]  # no paths
    h.update(" ".join(flags).encode())
    return h.hexdigest()[:16]


def recorded_traffic(cls: str, workload: str):
    """HBM bytes per launch of a launch class, from the committed rocprofv3 counter
    summary (FETCH_SIZE + WRITE_SIZE, calibrated on a plain copy), or None when there
    is none for this class and workload or its kernel sources changed since."""
    h = source_hash(cls)
    if h is None or not os.path.exists(TRAFFIC_RECORD):
        return None
    with open(TRAFFIC_RECORD) as fh:
        for line in fh:
            # | class | workload | source hash | fetch bytes | write bytes | total bytes |
            cells = [c.strip().strip("`") for c in line.strip().strip("|").split("|")]
            if len(cells) == 6 and cells[0] == cls and cells[1] == workload and cells[2] == h:
                return int(cells[5])
    return None


def time_steps(step, steps: int):
    """Time `steps` calls of step() bracketed by device synchronisations: (ms per step from
    HIP events, wall seconds). Nothing else runs in the timed region."""
    import torch
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    e0.record()
    for _ in range(steps):
        step()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / steps, time.perf_counter() - t0


def profiled_steps(step, steps: int):
    """The same `steps` steps again with libbpt's per-launch profiler on (HIP events around
    every launch, on the stream the kernel runs on): per launch class, its launches, time
    and algorithmic work; and the step time with the events in place (their gaps make it
    slightly longer than the unprofiled one)."""
    from paper_2305_19370_amd import bpt
    bpt.profile_enable(True)
    try:
        ms, _ = time_steps(step, steps)
    finally:
        bpt.profile_enable(False)
    return bpt.profile_report(), ms


def copy_probe(nbytes: int, reps: int) -> int:
    """A plain device copy of nbytes (read nbytes, write nbytes), the calibration
    reference for the HBM byte counters."""
    import torch
    torch.cuda.set_device(0)
    src = torch.empty(nbytes // 2, dtype=torch.bfloat16, device="cuda").fill_(1.0)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes": nbytes, "reps": reps}), flush=True)
    return 0


def atomic_probe(steps: int) -> int:
    """--atomic-probe: throughput of fp32 atomic adds into device memory, the cost of
    accumulating dQ across key blocks in a fused attention backward. index_add_ along
    dim 0 adds each row of src into the row of dst its index names with one fp32 atomic
    add per element; rows of 8192 floats (32 KB, one 64 x 128 dQ tile), G source rows
    onto `tiles` destination rows (several sources per destination: contention)."""
    import torch
    torch.cuda.set_device(0)
    res = []
    for tiles, G in ((4096, 4096), (512, 8192), (64, 8192)):
        dst = torch.zeros(tiles, 8192, dtype=torch.float32, device="cuda")
        src = torch.ones(G, 8192, dtype=torch.float32, device="cuda")
        idx = torch.arange(G, device="cuda") % tiles
        dst.index_add_(0, idx, src)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(steps):
            dst.index_add_(0, idx, src)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / steps
        adds = G * 8192
        res.append({"dst_rows": tiles, "src_rows": G, "ms": round(ms, 4), "gadds_per_s": round(adds / ms / 1e6, 1),
                    "atomic_gb_per_s": round(4 * adds / ms / 1e6, 1)})
        print(f"[atomic] {tiles} destination rows, {G} source rows: {ms:.3f} ms, "
              f"{4 * adds / ms / 1e6:.0f} GB/s of fp32 atomic adds", file=sys.stderr, flush=True)
    print(json.dumps({"atomic_probe": "torch index_add_ fp32 (global atomic add per element)", "points": res}),
          flush=True)
    return 0


XENT_SHAPE = dict(T=32768, D=4096, V=50257)     # 7B-shaped tokens and width, GPT-2 vocabulary


def cpu_baseline_xent(D: int, V: int, ldw: int, sample_T: int):
    """Time the float64 cross-entropy oracle (untuned) on sample_T tokens of the LM-head shape."""
    import numpy as np
    from bpt_inputs import make_xent_inputs
    from oracle.xent import xent_bwd, xent_fwd
    try:
        from threadpoolctl import threadpool_info
        threads = max([int(i.get("num_threads", 0)) for i in threadpool_info()] + [1])
    except Exception:  # pragma: no cover
        threads = len(os.sched_getaffinity(0))
    inp = make_xent_inputs(sample_T, D, V, ldw, "bf16", seed=0)
    h, W, y = inp["h"].double().numpy(), inp["W"].double().numpy(), inp["targets"].numpy()
    t0 = time.perf_counter()
    f = xent_fwd(h, W, y, V)
    b = xent_bwd(h, W, y, V)
    dt = time.perf_counter() - t0
    assert np.isfinite(f["loss"]) and np.isfinite(b["dW"]).all()
    fl = 6.0 * sample_T * D * V
    return {"value": fl / dt / 1e12, "unit": "TFLOP/s", "cores": threads, "kind": "oracle",
            "sample": f"fwd+bwd of {sample_T} tokens of the same LM-head shape (D={D}, V={V}), "
                      f"float64 numpy, {dt:.1f} s", "seconds": dt, "host": host_cpu_info(threads)}


def bench_xent(args) -> int:
    """--xent: the blockwise LM-head cross-entropy (logits never stored whole), fwd+bwd."""
    import torch
    from bpt_inputs import make_xent_inputs
    from paper_2305_19370_amd import bpt

    T, D, V = XENT_SHAPE["T"], XENT_SHAPE["D"], XENT_SHAPE["V"]
    ldw = (V + 63) // 64 * 64
    torch.cuda.set_device(0)
    print(f"[bench] xent T={T} D={D} V={V} ldw={ldw} bf16", file=sys.stderr, flush=True)
    inp = make_xent_inputs(T, D, V, ldw, "bf16", seed=0)
    h, W, y = inp["h"].cuda(), inp["W"].cuda(), inp["targets"].cuda()
    del inp
    cfg = bpt.make_xent_config(T, D, V, ldw, 0, "bf16")
    wsf = torch.empty(bpt.xent_workspace_bytes(cfg, False), dtype=torch.uint8, device="cuda")
    wsb = torch.empty(bpt.xent_workspace_bytes(cfg, True), dtype=torch.uint8, device="cuda")
    loss = torch.empty(1, dtype=torch.float32, device="cuda")
    lse = torch.empty(T, dtype=torch.float32, device="cuda")
    dh = torch.empty_like(h)
    dW = torch.empty((D, ldw), dtype=torch.float32, device="cuda")

    def step():
        bpt.xent_fwd(cfg, h, W, y, loss, lse, wsf)
        bpt.xent_bwd(cfg, h, W, y, lse, 1.0, dh, dW, wsb)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    torch.cuda.reset_peak_memory_stats()
    ms, _ = time_steps(step, args.steps)
    peak_gib = torch.cuda.max_memory_allocated() / 2 ** 30
    prof, ms_prof = profiled_steps(step, args.steps)
    ok = bool(torch.isfinite(loss).all() and torch.isfinite(dh.float()).all())
    print(f"[bench] xent {args.steps} steps: {ms:.2f} ms/step, loss {loss.item():.4f}, finite={ok}",
          file=sys.stderr, flush=True)
    value = 6.0 * T * D * V / (ms / 1e3) / 1e12
    name, rec = max(prof.items(), key=lambda kv: kv[1]["ms"])
    achieved = rec["flops"] / (rec["ms"] / 1e3) / 1e12
    out = {
        "metric": "LM-head cross-entropy fwd+bwd TFLOP/s (blockwise over tokens, logits never stored whole)",
        "value": round(value, 2), "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms, 3), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "lmhead_xent_t32768_d4096_v50257", "T": T, "D": D, "V": V, "ldw": ldw,
                   "block_rows": min(8192, T)},
        "pct_of_peak": round(100 * value / PEAK_BF16_TFLOPS, 2),
        "tokens_per_s": round(T / (ms / 1e3), 1),
        "peak_hbm_gib": round(peak_gib, 3),
        "profiled_ms_per_step": round(ms_prof, 3),
        "roofline": {"bound": "mfma", "achieved": achieved, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": achieved / PEAK_BF16_TFLOPS, "kernel": name,
                     "launches_per_step": rec["count"] / args.steps, "avg_launch_ms": rec["ms"] / rec["count"],
                     "traffic": None, "traffic_unit": "bytes per launch"},
        "kernels": {k: {"ms_per_step": v["ms"] / args.steps,
                        "tflops": (v["flops"] / (v["ms"] / 1e3) / 1e12) if v["flops"] > 0 and v["ms"] > 0 else None,
                        "gbs": (v["bytes"] / (v["ms"] / 1e3) / 1e9) if v["ms"] > 0 else None}
                    for k, v in sorted(prof.items(), key=lambda kv: -kv[1]["ms"])},
    }
    if not args.no_cpu_baseline:
        print("[bench] cpu baseline (oracle) on 256 tokens ...", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline_xent(D, V, ldw, 256)
    else:
        out["cpu_baseline"] = None
    print(json.dumps(out), flush=True)
    return 0 if ok else 1


# GPT-XL (1B) of Table 1 / Table 4: 24 layers, width 2048, 16 heads of 128, FFN 4x,
# GPT-2 vocabulary; one 16K-token sequence per step (Table 4's batch at that length)
GPT_SHAPE = dict(L=24, B=1, S=16384, D=2048, H=16, F=8192, V=50257, Bq=1024, Bkv=1024)


def gpt_flops_step(L, B, S, D, F, V, causal=True):
    """Model FLOPs of one training step: 3x the forward of L layers plus the LM head."""
    return 3 * (L * model_flops_fwd(B, S, D, F, causal) + 2 * B * S * D * V)


def cpu_baseline_gpt(shape: dict, sample_L: int, sample_S: int):
    """Time the float64 GPT oracle (untuned) forward and backward on sample_L layers of the
    model's shape and a sample_S-token sequence, then express its FLOP rate as tokens/s of
    the full model. The oracle's AdamW is left out of the timing: its float64 temporaries
    over the 100M-entry head alone take half a minute, which would swamp the sample."""
    import numpy as np
    from bpt_inputs import make_gpt_inputs
    from oracle.gpt import GPTParams, gpt_fwd_bwd
    from oracle.layer import LayerParams
    try:
        from threadpoolctl import threadpool_info
        threads = max([int(i.get("num_threads", 0)) for i in threadpool_info()] + [1])
    except Exception:  # pragma: no cover
        threads = len(os.sched_getaffinity(0))
    D, F, V, H = shape["D"], shape["F"], shape["V"], shape["H"]
    inp = make_gpt_inputs(sample_L, 1, sample_S, D, F, V, (V + 63) // 64 * 64, dtype="bf16", seed=0)
    f = lambda k: inp[k].double().numpy()
    mats, vecs = ("Wq", "Wk", "Wv", "Wo", "W1", "W2"), ("ln1_g", "ln1_b", "ln2_g", "ln2_b", "b1", "b2")
    P = GPTParams(Wte=f("Wte"), Wpe=f("Wpe"), lnf_g=f("lnf_g"), lnf_b=f("lnf_b"), Wout=f("Wout")[:, :V],
                  layers=[LayerParams(**{k: f(f"{l}.{k}") for k in mats + vecs}) for l in range(sample_L)])
    tok = inp["tokens"].numpy().reshape(1, sample_S)
    tgt = inp["targets"].numpy().reshape(1, sample_S)
    del inp
    t0 = time.perf_counter()
    g = gpt_fwd_bwd(tok, tgt, P, H)
    dt = time.perf_counter() - t0
    assert np.isfinite(g["loss"])
    fl = gpt_flops_step(sample_L, 1, sample_S, D, F, V)
    full_per_token = gpt_flops_step(shape["L"], 1, shape["S"], D, F, V) / shape["S"]
    return {"value": fl / dt / full_per_token, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": f"fwd+bwd (AdamW not timed) of {sample_L} of the {shape['L']} layers (D={D}, F={F}, H={H}) plus the "
                      f"V={V} head on one {sample_S}-token sequence, float64 numpy, {dt:.1f} s; its FLOP rate "
                      f"({fl / dt / 1e12:.3f} TFLOP/s) divided by the full model's FLOPs per token at "
                      f"S={shape['S']}", "seconds": dt, "host": host_cpu_info(threads)}


def bench_gpt(args) -> int:
    """--gpt: one GPT-XL training step (embedding, 24 BPT layers, final LN, blockwise
    LM-head loss, backward, AdamW) on synthetic tokens."""
    import torch
    from paper_2305_19370_amd import bpt
    from paper_2305_19370_amd.gpt import GPT, GPTShape, cosine_lr

    shp = dict(GPT_SHAPE)
    if args.gpt_seq:
        shp["S"] = args.gpt_seq
    if args.gpt_batch:
        shp["B"] = args.gpt_batch
    s = GPTShape(**shp, dtype="bf16")
    torch.cuda.set_device(0)
    print(f"[bench] gpt {s}", file=sys.stderr, flush=True)
    m = GPT(s, device="cuda", seed=0)
    g = torch.Generator(device="cpu").manual_seed(0)
    tok = torch.randint(0, s.V, (s.B * s.S,), generator=g, dtype=torch.int32).cuda()
    tgt = torch.randint(0, s.V, (s.B * s.S,), generator=g, dtype=torch.int32).cuda()
    total = args.warmup + 2 * args.steps     # warm-up, timed and profiled steps
    it = [0]

    def step():
        m.train_step(tok, tgt, cosine_lr(it[0], 2e-4, 0, total))
        it[0] += 1

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    torch.cuda.reset_peak_memory_stats()
    ms, _ = time_steps(step, args.steps)
    peak_gib = torch.cuda.max_memory_allocated() / 2 ** 30
    prof, ms_prof = profiled_steps(step, args.steps)
    loss = float(m.loss.item())
    ok = bool(torch.isfinite(m.loss).all())
    print(f"[bench] gpt {args.steps} steps: {ms:.2f} ms/step, loss {loss:.4f}, finite={ok}",
          file=sys.stderr, flush=True)
    T = s.B * s.S
    fl = gpt_flops_step(s.L, s.B, s.S, s.D, s.F, s.V)
    name, rec = max(prof.items(), key=lambda kv: kv[1]["ms"])
    if rec["flops"] > 0:
        achieved = rec["flops"] / (rec["ms"] / 1e3) / 1e12
        roof = {"bound": "mfma", "achieved": achieved, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                "frac": achieved / PEAK_BF16_TFLOPS}
    else:
        achieved = rec["bytes"] / (rec["ms"] / 1e3) / 1e9
        roof = {"bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": achieved / PEAK_HBM_GBS}
    workload = f"gpt_xl_1b_s{s.S}" + (f"_b{s.B}" if s.B != 1 else "")
    roof.update({"kernel": name, "launches_per_step": rec["count"] / args.steps,
                 "avg_launch_ms": rec["ms"] / rec["count"], "traffic": recorded_traffic(name, workload),
                 "traffic_unit": "bytes per launch"})
    out = {
        "metric": "GPT training tokens/s per device (Table 4 analog: GPT-XL 1B, synthetic tokens)",
        "value": round(T / (ms / 1e3), 1), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 3), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": workload, "L": s.L, "B": s.B, "S": s.S, "D": s.D, "H": s.H, "F": s.F, "V": s.V,
                   "Bq": s.Bq, "Bkv": s.Bkv, "params": s.n_params(), "optimizer": "AdamW(0.9, 0.95, wd 0.1)"},
        "model_tflops": round(fl / (ms / 1e3) / 1e12, 2),
        "pct_of_peak": round(100 * fl / (ms / 1e3) / 1e12 / PEAK_BF16_TFLOPS, 2),
        "loss": loss,
        "peak_hbm_gib": round(peak_gib, 3),
        "profiled_ms_per_step": round(ms_prof, 3),
        "roofline": roof,
        "kernels": {k: {"ms_per_step": v["ms"] / args.steps,
                        "tflops": (v["flops"] / (v["ms"] / 1e3) / 1e12) if v["flops"] > 0 and v["ms"] > 0 else None,
                        "gbs": (v["bytes"] / (v["ms"] / 1e3) / 1e9) if v["ms"] > 0 else None}
                    for k, v in sorted(prof.items(), key=lambda kv: -kv[1]["ms"])},
    }
    if not args.no_cpu_baseline:
        print("[bench] cpu baseline (oracle) on 4 layers x 2048 tokens ...", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline_gpt(shp, 4, 2048)
    else:
        out["cpu_baseline"] = None
    print(json.dumps(out), flush=True)
    return 0 if ok else 1


# GEMM shapes (name, M, N, K, A transposed) of the 7B-shaped layer (T = 32768 tokens, D = 4096,
# F = 16384) with FFN groups of 8192 rows (the shapes the hipBLASLt comparison was taken on), as
# C[M, N] = A[M, K] B[K, N]
YARDSTICK_SHAPES = (
    ("qkv_proj", 32768, 4096, 4096, False),
    ("ffn1", 8192, 16384, 4096, False),
    ("ffn2", 8192, 4096, 16384, False),
    ("dwqkv", 4096, 4096, 32768, True),
    ("dw1", 4096, 16384, 8192, True),
    ("du", 32768, 4096, 12288, False),
)


def gemm_yardstick(args) -> int:
    """--gemm-yardstick: torch.matmul (hipBLASLt) in bf16 with fp32 accumulation on the
    7B-shaped layer's GEMM shapes, then the libbpt layer step, in one process, so that
    one counter pass sees the vendor GEMMs and the layer's kernels on the same box."""
    import torch
    torch.cuda.set_device(0)
    g = torch.Generator(device="cpu").manual_seed(0)
    res = {}
    for name, M, N, K, at in YARDSTICK_SHAPES:
        a = (torch.randn((K, M) if at else (M, K), generator=g) * 0.05).to(torch.bfloat16).cuda()
        b = (torch.randn((K, N), generator=g) * 0.05).to(torch.bfloat16).cuda()
        A = a.t() if at else a
        for _ in range(3):
            c = torch.matmul(A, b)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(args.steps):
            c = torch.matmul(A, b)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / args.steps
        res[name] = {"M": M, "N": N, "K": K, "a_transposed": at, "ms": round(ms, 4),
                     "tflops": round(2.0 * M * N * K / (ms / 1e3) / 1e12, 1)}
        print(f"[yardstick] torch.matmul {name} {M}x{N}x{K}: {ms:.3f} ms, {res[name]['tflops']} TFLOP/s",
              file=sys.stderr, flush=True)
        del a, b, c, A
    torch.cuda.empty_cache()
    print(json.dumps({"yardstick": "torch.matmul bf16 (hipBLASLt)", "shapes": res}), flush=True)
    return 0


def mfma_probe(args) -> int:
    """--mfma-probe: the matrix-core loops of libbpt_probe.so (bf16 32x32x16 products on
    register operands, and with one LDS fragment read per one or two products, at one or
    two waves per SIMD), timed over launches of about 0.2 s each: the rates the chip
    sustains for matrix work without memory traffic, beside the nominal 2.5 PFLOP/s."""
    import ctypes
    import torch
    torch.cuda.set_device(0)
    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2305_19370_amd", "libbpt_probe.so"))
    fn = lib.bpt_probe_mfma_loop
    fn.restype = ctypes.c_int32
    fn.argtypes = [ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p,
                   ctypes.c_void_p]
    seed = (torch.rand(4096, generator=torch.Generator().manual_seed(0)) * 2 - 1).cuda()
    out = torch.empty(2048 * 256, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream
    # (name, mode, workgroups, iterations): 8 resident waves per SIMD for the register loops
    # 0 and 1, two for the LDS-fed ones 2-4 (64 KiB of LDS per workgroup), one for 5-7
    # (96 KiB); about 0.2 s per launch
    modes = (("one_pair", 0, 2048, 300000), ("varied_pairs", 1, 2048, 300000), ("lds_fragment", 2, 512, 1000000),
             ("lds_fragment_ahead", 3, 512, 1000000), ("lds_half_ahead", 4, 512, 1000000),
             ("lds_fragment_ahead_1w", 5, 256, 2000000), ("lds_half_ahead_1w", 6, 256, 2000000),
             ("varied_pairs_1w", 7, 256, 2000000))
    res = {}
    for name, mode, wg, iters in modes:
        flops = float(wg) * 4 * iters * 4 * 32768
        ms = []
        for i in range(args.warmup + args.steps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            rc = fn(wg, iters, mode, seed.data_ptr(), out.data_ptr(), stream)
            e1.record()
            if rc != 0:
                raise RuntimeError(f"bpt_probe_mfma_loop returned {rc}")
            torch.cuda.synchronize()
            if i >= args.warmup:
                ms.append(e0.elapsed_time(e1))
                print(f"[mfma-probe] {name} launch {len(ms)}: {ms[-1]:.2f} ms, {flops / ms[-1] / 1e9:.1f} TFLOP/s",
                      file=sys.stderr, flush=True)
        tf = [flops / m / 1e9 for m in ms]
        res[name] = {"mode": mode, "workgroups": wg, "iters": iters, "flops_per_launch": flops,
                     "ms": [round(m, 3) for m in ms], "tflops": [round(t, 1) for t in tf],
                     "mean_tflops": round(sum(tf) / len(tf), 1), "min_tflops": round(min(tf), 1)}
    assert torch.isfinite(out).all()
    print(json.dumps({"probe": "bf16 MFMA 32x32x16 loops (libbpt_probe.so)", "peak_tflops": 2500.0, "modes": res}),
          flush=True)
    return 0


def host_cpu_info(threads: int) -> dict:
    """The host CPU model and the BLAS library numpy's oracle runs on."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    blas = "unknown"
    try:
        from threadpoolctl import threadpool_info
        libs = [i for i in threadpool_info() if i.get("user_api") == "blas"]
        if libs:
            blas = f"{libs[0].get('internal_api')} {libs[0].get('version')}"
    except Exception:  # pragma: no cover
        pass
    return {"cpu_model": model, "blas": blas, "threads": threads,
            "cpus_available": len(os.sched_getaffinity(0))}


def layer_buffers(w, cfg, bpt) -> dict:
    """Bytes of every device buffer a fwd+bwd step holds (all allocated by the caller,
    torch here; the library allocates nothing): the analytic peak HBM."""
    E = 2 if w.dtype == "bf16" else 4
    T, D, F = w.B * w.S, w.D, w.F
    wts = (4 * D * D + 2 * D * F) * E
    return {"weights": wts, "grads_fp32": (4 * D * D + 2 * D * F) * 4, "X_dY_Y_dX": 4 * T * D * E,
            "saved": bpt.saved_bytes(cfg), "workspace_fwd": bpt.workspace_bytes(cfg, False),
            "workspace_bwd": bpt.workspace_bytes(cfg, True)}


def measure_layer(w, steps: int, warmup: int, verbose: bool = True) -> dict:
    """Time `steps` fwd+bwd steps (after `warmup`) and `steps` forwards of workload w,
    with the library's per-launch profiler on during the fwd+bwd steps; peak HBM over
    the timed steps. Inputs are resident on the device before timing starts."""
    import torch
    from bpt_inputs import make_inputs
    from paper_2305_19370_amd import bpt

    dev = "cuda"
    if verbose:
        print(f"[bench] workload {w.name}: B={w.B} S={w.S} D={w.D} H={w.H} F={w.F} Bq={w.Bq} Bkv={w.Bkv} "
              f"dtype={w.dtype}", file=sys.stderr, flush=True)
    torch.cuda.empty_cache()
    torch.cuda.reset_peak_memory_stats()
    base = torch.cuda.memory_allocated()
    inp = make_inputs(w, seed=0)
    d = {k: (v.to(dev) if v is not None else None) for k, v in inp.items()}
    del inp
    cfg = bpt.make_config(w.B, w.S, w.D, w.H, w.F, w.Bq, w.Bkv, w.causal, w.dtype, w.dtype)
    wsf = torch.empty(bpt.workspace_bytes(cfg, False), dtype=torch.uint8, device=dev)
    wsb = torch.empty(bpt.workspace_bytes(cfg, True), dtype=torch.uint8, device=dev)
    out_dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    Y = torch.empty(w.B, w.S, w.D, dtype=out_dt, device=dev)
    dX = torch.empty_like(Y)
    saved = torch.empty(bpt.saved_bytes(cfg), dtype=torch.uint8, device=dev)
    shapes = {"dWq": (w.D, w.D), "dWk": (w.D, w.D), "dWv": (w.D, w.D), "dWo": (w.D, w.D),
              "dW1": (w.D, w.F), "dW2": (w.F, w.D)}
    grads = {k: torch.empty(s, dtype=torch.float32, device=dev) for k, s in shapes.items()}

    def step():
        bpt.layer_fwd(cfg, d["X"], d, Y, saved, wsf)
        bpt.layer_bwd(cfg, d["X"], d, saved, d["dY"], dX, grads, wsb)

    def fwd():
        bpt.layer_fwd(cfg, d["X"], d, Y, saved, wsf)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    if verbose:
        print(f"[bench] warmup done", file=sys.stderr, flush=True)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        fwd()
    e1.record()
    torch.cuda.synchronize()
    fwd_ms = e0.elapsed_time(e1) / steps

    ms, wall = time_steps(step, steps)
    peak = torch.cuda.max_memory_allocated() - base
    prof, ms_prof = profiled_steps(step, steps)
    ok = bool(torch.isfinite(Y.float()).all() and torch.isfinite(dX.float()).all())
    bufs = layer_buffers(w, cfg, bpt)
    group_rows = bpt.group_rows(cfg)
    del d, wsf, wsb, Y, dX, saved, grads
    torch.cuda.empty_cache()
    if verbose:
        print(f"[bench] {w.name} {steps} steps: {ms:.2f} ms/step (wall {wall / steps * 1e3:.2f}; "
              f"{ms_prof:.2f} with per-launch events), fwd {fwd_ms:.2f} ms, "
              f"peak {peak / 2 ** 30:.3f} GiB, finite={ok}", file=sys.stderr, flush=True)
    return {"ms": ms, "fwd_ms": fwd_ms, "peak": peak, "buffers": bufs, "prof": prof, "ok": ok,
            "group_rows": group_rows, "ms_profiled": ms_prof}


def linear_fit(xs, ys):
    """Least-squares y = a + b x; returns (a, b, R^2)."""
    n = len(xs)
    mx, my = sum(xs) / n, sum(ys) / n
    sxx = sum((x - mx) ** 2 for x in xs)
    sxy = sum((x - mx) * (y - my) for x, y in zip(xs, ys))
    b = sxy / sxx
    a = my - b * mx
    ss_res = sum((y - a - b * x) ** 2 for x, y in zip(xs, ys))
    ss_tot = sum((y - my) ** 2 for y in ys)
    return a, b, 1.0 - ss_res / ss_tot if ss_tot > 0 else 1.0


def peak_hbm_fit(pts) -> dict:
    """Least-squares fit of peak HBM in S over the sweep lengths at which the FFN group has
    its full size (at shorter ones the group is the whole sequence, so the constant part of
    the memory is smaller); no fit with fewer than two such lengths."""
    full = max(p["group_rows"] for p in pts)
    fit_pts = [p for p in pts if p["group_rows"] == full]
    lengths = [p["S"] for p in fit_pts]
    if len(set(lengths)) < 2:
        return {"intercept_bytes": None, "bytes_per_token": None, "r2": None, "lengths": lengths}
    a, b, r2 = linear_fit(lengths, [p["peak_hbm_bytes"] for p in fit_pts])
    return {"intercept_bytes": a, "bytes_per_token": b, "r2": r2, "lengths": lengths}


def bench_sweep(args) -> int:
    """--sweep-s: the 13B-shaped layer at each sequence length of the list: fwd and
    fwd+bwd TFLOP/s, tokens/s, peak HBM against the analytic sum of the step's buffers,
    and a linear fit of peak HBM in S."""
    import torch
    from bpt_inputs import sweep_workload
    torch.cuda.set_device(0)
    pts = []
    for S in [int(x) for x in args.sweep_s.split(",")]:
        w = sweep_workload(S)
        r = measure_layer(w, args.steps, args.warmup)
        ffwd = model_flops_fwd(w.B, w.S, w.D, w.F, w.causal)
        expected = sum(r["buffers"].values())
        pts.append({"S": S, "ms_per_step": round(r["ms"], 3), "fwd_ms": round(r["fwd_ms"], 3),
                    "tflops": round(3 * ffwd / (r["ms"] / 1e3) / 1e12, 1),
                    "fwd_tflops": round(ffwd / (r["fwd_ms"] / 1e3) / 1e12, 1),
                    "tokens_per_s": round(w.B * S / (r["ms"] / 1e3), 1),
                    "peak_hbm_bytes": int(r["peak"]), "expected_bytes": int(expected),
                    "buffers": r["buffers"], "group_rows": r["group_rows"],
                    "avoided_scores_bytes": 2 * w.B * w.H * S * S,          # one [B, H, S, S] bf16
                    "avoided_ffn_bytes": 2 * w.B * S * w.F, "finite": r["ok"]})
        del r
    fit = peak_hbm_fit(pts)
    out = {"metric": "BPT layer fwd+bwd TFLOP/s, tokens/s and peak HBM against sequence length (13B-shaped)",
           "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "dtype": "bf16", "data": "synthetic",
           "config": {"workload": "bf16_13b_sweep", "B": 1, "D": 5120, "H": 40, "F": 20480, "Bq": 2048,
                      "Bkv": 2048, "causal": True},
           "points": pts,
           "peak_hbm_fit": fit}
    print(json.dumps(out), flush=True)
    return 0 if all(p["finite"] for p in pts) else 1


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="bf16_7b_s32768")
    ap.add_argument("--cpu-sample-s", type=int, default=4096)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="BYTES",
                    help="only run a plain device copy of BYTES (counter calibration)")
    ap.add_argument("--xent", action="store_true",
                    help="measure the blockwise LM-head cross-entropy instead of the layer")
    ap.add_argument("--gpt", action="store_true",
                    help="measure a GPT-XL (1B) training step (24 layers, head, AdamW) instead of the layer")
    ap.add_argument("--gpt-seq", type=int, default=0, help="sequence length of --gpt (default 16384)")
    ap.add_argument("--gpt-batch", type=int, default=0, help="sequences per step of --gpt (default 1)")
    ap.add_argument("--atomic-probe", action="store_true",
                    help="only measure the throughput of fp32 atomic adds into device memory")
    ap.add_argument("--sweep-s", default="", metavar="S1,S2,...",
                    help="measure the 13B-shaped layer at each of these sequence lengths (peak HBM vs S)")
    ap.add_argument("--mfma-probe", action="store_true",
                    help="time the register-only matrix-core loop (the chip's sustained bf16 MFMA rate)")
    ap.add_argument("--gemm-yardstick", action="store_true",
                    help="time torch.matmul (hipBLASLt) on the 7B-shaped layer's GEMM shapes, then run the layer")
    args = ap.parse_args()
    if args.copy_probe:
        return copy_probe(args.copy_probe, 3)
    if args.atomic_probe:
        return atomic_probe(args.steps)
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}): the library runs the "
              "layer on one GPU; sharding it over several is designed, not implemented", file=sys.stderr)
        return 2
    if args.xent:
        return bench_xent(args)
    if args.gpt:
        return bench_gpt(args)
    if args.sweep_s:
        return bench_sweep(args)
    if args.mfma_probe:
        return mfma_probe(args)
    if args.gemm_yardstick:
        rc = gemm_yardstick(args)
        if rc:
            return rc

    import torch
    from bpt_inputs import workload

    w = workload(args.workload)
    torch.cuda.set_device(0)
    r = measure_layer(w, args.steps, args.warmup)
    ms, fwd_ms, prof, ok, peak_hbm = r["ms"], r["fwd_ms"], r["prof"], r["ok"], r["peak"]

    ffwd = model_flops_fwd(w.B, w.S, w.D, w.F, w.causal)
    value = 3 * ffwd / (ms / 1e3) / 1e12
    peak = PEAK_BF16_TFLOPS if w.dtype == "bf16" else PEAK_FP32_TFLOPS

    # roofline entry: the launch class with the largest total time
    top = max(prof.items(), key=lambda kv: kv[1]["ms"])
    name, rec = top
    if rec["flops"] > 0:
        achieved = rec["flops"] / (rec["ms"] / 1e3) / 1e12
        roof = {"bound": "mfma", "achieved": achieved, "peak": peak, "unit": "TFLOP/s", "frac": achieved / peak}
    else:
        achieved = rec["bytes"] / (rec["ms"] / 1e3) / 1e9
        roof = {"bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": achieved / PEAK_HBM_GBS}
    roof.update({"kernel": name, "launches_per_step": rec["count"] / args.steps,
                 "avg_launch_ms": rec["ms"] / rec["count"], "traffic": recorded_traffic(name, w.name),
                 "traffic_unit": "bytes per launch"})
    breakdown = {k: {"ms_per_step": v["ms"] / args.steps,
                     "tflops": (v["flops"] / (v["ms"] / 1e3) / 1e12) if v["flops"] > 0 and v["ms"] > 0 else None,
                     "gbs": (v["bytes"] / (v["ms"] / 1e3) / 1e9) if v["ms"] > 0 else None}
                 for k, v in sorted(prof.items(), key=lambda kv: -kv[1]["ms"])}

    out = {
        "metric": "BPT layer fwd+bwd TFLOP/s (% bf16 MFMA peak), tokens/s, peak HBM vs seq len",
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {"workload": w.name, "B": w.B, "S": w.S, "D": w.D, "H": w.H, "F": w.F, "Bq": w.Bq,
                   "Bkv": w.Bkv, "causal": w.causal, "group_rows": r["group_rows"]},
        "pct_of_peak": round(100 * value / peak, 2),
        "tokens_per_s": round(w.B * w.S / (ms / 1e3), 1),
        "fwd_ms": round(fwd_ms, 3),
        "fwd_tflops": round(ffwd / (fwd_ms / 1e3) / 1e12, 2),
        "peak_hbm_gib": round(peak_hbm / 2 ** 30, 3),
        "expected_hbm_gib": round(sum(r["buffers"].values()) / 2 ** 30, 3),
        "profiled_ms_per_step": round(r["ms_profiled"], 3),
        "roofline": roof,
        "kernels": breakdown,
    }
    if not args.no_cpu_baseline:
        print(f"[bench] cpu baseline (oracle) on S={args.cpu_sample_s} ...", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(w, args.cpu_sample_s)
    else:
        out["cpu_baseline"] = None
    print(json.dumps(out), flush=True)
    return 0 if ok else 1


if __name__ == "__main__":
    sys.exit(main())
