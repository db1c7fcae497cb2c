"""The layer step under HIP graph capture: libbpt launches asynchronously on the caller's
stream, allocates nothing, synchronises nothing and records no memset, so a forward and
backward captured into a graph (torch.cuda.CUDAGraph) replays the same kernels on the same
buffers. Each replay, with unrelated eager work and synchronisations between replays and the
outputs cleared before each, must reproduce the eager step bitwise (the kernels are
deterministic). The forward without allocation (its workspace the library's static scratch)
is captured the same way."""
import pytest
import torch

from bpt_inputs import make_inputs, small_workload
from gpu_util import gpu_config, say
from paper_2305_19370_amd import bpt

pytestmark = pytest.mark.gpu

REPLAYS = 3


def _setup(dtype, seed):
    w = small_workload(dtype, B=2, S=700, D=256, H=2, F=1024, causal=True, Bq=128, Bkv=128)
    cfg = gpu_config(w, out_dtype=w.dtype, group_blocks=2)
    inp = make_inputs(w, seed=seed, affine=True, biases=True)
    d = {k: (v.cuda() if v is not None else None) for k, v in inp.items()}
    dt = torch.bfloat16 if dtype == "bf16" else torch.float32
    buf = {
        "Y": torch.empty(w.B, w.S, w.D, dtype=dt, device="cuda"),
        "dX": torch.empty(w.B, w.S, w.D, dtype=dt, device="cuda"),
        "saved": torch.empty(bpt.saved_bytes(cfg), dtype=torch.uint8, device="cuda"),
        "wsf": torch.empty(bpt.workspace_bytes(cfg, False), dtype=torch.uint8, device="cuda"),
        "wsb": torch.empty(bpt.workspace_bytes(cfg, True), dtype=torch.uint8, device="cuda"),
    }
    shapes = {"dWq": (w.D, w.D), "dWk": (w.D, w.D), "dWv": (w.D, w.D), "dWo": (w.D, w.D),
              "dW1": (w.D, w.F), "dW2": (w.F, w.D), "db1": (w.F,), "db2": (w.D,),
              "dln1_g": (w.D,), "dln1_b": (w.D,), "dln2_g": (w.D,), "dln2_b": (w.D,)}
    grads = {k: torch.empty(s, dtype=torch.float32, device="cuda") for k, s in shapes.items()}
    return w, cfg, d, buf, grads


def _outputs(buf, grads):
    out = {"Y": buf["Y"], "dX": buf["dX"], "saved": buf["saved"]}
    out.update(grads)
    return {k: v.clone() for k, v in out.items()}


def _clear(buf, grads):
    for t in (buf["Y"], buf["dX"], *grads.values()):
        t.fill_(float("nan"))
    buf["saved"].zero_()


def _check_replays(g, ref, buf, grads, name):
    for r in range(REPLAYS):
        _clear(buf, grads)
        x = torch.randn(4096, device="cuda")          # unrelated eager work between replays
        (x * 2).sum().item()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = _outputs(buf, grads)
        bad = [k for k in ref if not torch.equal(got[k], ref[k])]
        assert not bad, f"{name}: replay {r} differs from the eager step in {bad}"


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_layer_step_replays_from_a_graph(dtype):
    w, cfg, d, buf, grads = _setup(dtype, seed=41)
    say(f"case graph fwd+bwd {w.name}")

    def step():
        bpt.layer_fwd(cfg, d["X"], d, buf["Y"], buf["saved"], buf["wsf"])
        bpt.layer_bwd(cfg, d["X"], d, buf["saved"], d["dY"], buf["dX"], grads, buf["wsb"])

    _clear(buf, grads)
    step()
    torch.cuda.synchronize()
    ref = _outputs(buf, grads)
    assert all(torch.isfinite(v.float()).all() for k, v in ref.items() if k != "saved")
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()
    _check_replays(g, ref, buf, grads, w.name)


def test_noalloc_forward_replays_from_a_graph():
    w, cfg, d, buf, grads = _setup("bf16", seed=42)
    assert bpt.workspace_bytes(cfg, False) <= bpt.NOALLOC_SCRATCH_BYTES
    say(f"case graph noalloc forward {w.name}")

    def fwd():
        bpt.layer_fwd_noalloc(cfg, d["X"], d, buf["Y"], buf["saved"])

    _clear(buf, grads)
    fwd()
    torch.cuda.synchronize()
    ref = {"Y": buf["Y"].clone(), "saved": buf["saved"].clone()}
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fwd()
    torch.cuda.synchronize()
    for r in range(REPLAYS):
        _clear(buf, grads)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(buf["Y"], ref["Y"]) and torch.equal(buf["saved"], ref["saved"]), f"replay {r} differs"
