"""bpt_layer_fwd_noalloc (the forward with the library's static scratch as workspace)
against bpt_layer_fwd (a caller-provided workspace), through the C ABI: identical Y
and saved activations, on two calls in a row, the second with a smaller input (the
scratch keeps the first call's contents), for the bf16 and fp32 paths."""
import pytest
import torch

from bpt_inputs import make_inputs, small_workload
from gpu_util import gpu_config, say
from paper_2305_19370_amd import bpt

pytestmark = pytest.mark.gpu


def _both(w, seed, **over):
    cfg = gpu_config(w, out_dtype=w.dtype, **over)
    inp = make_inputs(w, seed=seed, affine=True, biases=True)
    d = {k: (v.cuda() if v is not None else None) for k, v in inp.items()}
    need = bpt.workspace_bytes(cfg, False)
    assert 0 < need <= bpt.NOALLOC_SCRATCH_BYTES, need
    dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    out = {}
    for mode in ("ws", "noalloc"):
        Y = torch.full((w.B, w.S, w.D), float("nan"), dtype=dt, device="cuda")
        saved = torch.zeros(max(bpt.saved_bytes(cfg), 256), dtype=torch.uint8, device="cuda")
        if mode == "ws":
            ws = torch.empty(need, dtype=torch.uint8, device="cuda")
            bpt.layer_fwd(cfg, d["X"], d, Y, saved, ws)
        else:
            bpt.layer_fwd_noalloc(cfg, d["X"], d, Y, saved)
        torch.cuda.synchronize()
        out[mode] = (Y.cpu(), saved.cpu())
    return out


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_noalloc_forward_matches_workspace_forward(dtype):
    for S, B, seed in ((700, 2, 31), (130, 1, 32)):      # the second call is smaller
        w = small_workload(dtype, B=B, S=S, D=256, H=2, F=512, causal=True, Bq=128, Bkv=128)
        say(f"case noalloc {w.name}")
        out = _both(w, seed, group_blocks=2)
        Ya, sa = out["ws"]
        Yb, sb = out["noalloc"]
        assert torch.isfinite(Yb.float()).all()
        assert torch.equal(Ya, Yb), f"{w.name}: Y differs"
        assert torch.equal(sa, sb), f"{w.name}: saved activations differ"


def test_noalloc_rejects_oversize_config():
    """A configuration whose forward workspace exceeds the static scratch is refused
    before anything is launched."""
    cfg = bpt.make_config(1, 32768, 4096, 32, 16384, 1024, 1024, True, "bf16", "bf16")
    assert bpt.workspace_bytes(cfg, False) > bpt.NOALLOC_SCRATCH_BYTES
    lib = bpt.load()
    import ctypes
    st = lib.bpt_layer_fwd_noalloc(ctypes.byref(cfg), 16, ctypes.byref(bpt.Params()), 4096, 8192, None)
    assert st == 3, st          # BPT_ERR_WORKSPACE
    assert b"static scratch" in lib.bpt_last_error()
