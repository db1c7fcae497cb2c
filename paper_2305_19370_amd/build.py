"""Build libbpt.so in-tree with hipcc for gfx950.

Usage: ``python -m paper_2305_19370_amd.build`` (or ``__graft_entry__.build()``).
Each translation unit is compiled in parallel, then linked into
``paper_2305_19370_amd/libbpt.so`` via a temporary file and an atomic rename.
"""
from __future__ import annotations

import concurrent.futures
import os
import shutil
import subprocess
import sys
import tempfile

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
SOURCES = ["libbpt.cpp", "gemm.hip", "attn_fwd.hip", "attn_bwd_dq.hip", "attn_bwd_dkdv.hip", "rowwise.hip", "gpt.hip", "dropout.hip"]
# per-source code generation options: the attention kernels keep the accumulators of
# their MFMAs in architectural VGPRs (the default placement copies them between the
# register files every iteration)
EXTRA_FLAGS = {
    "attn_fwd.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form=1"],
    "attn_bwd_dq.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form=1"],
    "attn_bwd_dkdv.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form=1"],
}
LIB = os.path.join(PKG, "libbpt.so")
# the matrix-core ceiling probe that bench.py --mfma-probe times (measurement only)
PROBE_SOURCES = ["probe_mfma.hip"]
PROBE_LIB = os.path.join(PKG, "libbpt_probe.so")
ARCH = os.environ.get("BPT_OFFLOAD_ARCH", "gfx950")

HIP_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    # keep fp32 vector math off the packed-fp32 instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", os.path.join(ROOT, "include"),
]


def _hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found")


def _compile(src: str, obj: str) -> None:
    cmd = [_hipcc(), *HIP_FLAGS, *EXTRA_FLAGS.get(src, []), "-c", os.path.join(CSRC, src), "-o", obj]
    if src.endswith(".cpp"):
        cmd[1:1] = ["-x", "hip"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stderr[-4000:]}")


def build(verbose: bool = True) -> str:
    srcs = SOURCES + PROBE_SOURCES
    with tempfile.TemporaryDirectory(prefix="bpt_build_") as tmp:
        objs = {s: os.path.join(tmp, s + ".o") for s in srcs}
        with concurrent.futures.ThreadPoolExecutor(max_workers=min(len(srcs), os.cpu_count() or 1)) as ex:
            list(ex.map(_compile, srcs, [objs[s] for s in srcs]))
        for lib, group in ((LIB, SOURCES), (PROBE_LIB, PROBE_SOURCES)):
            out_tmp = lib + ".tmp"
            r = subprocess.run([_hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", out_tmp,
                                *[objs[s] for s in group]], capture_output=True, text=True)
            if r.returncode != 0:
                raise RuntimeError(f"link of {os.path.basename(lib)} failed:\n{r.stderr[-4000:]}")
            os.replace(out_tmp, lib)
            if verbose:
                print(f"built {lib}", file=sys.stderr)
    return LIB


if __name__ == "__main__":
    build()
