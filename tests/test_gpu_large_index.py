"""Index range: a batch of 4116 sequences of 2048 tokens (8,429,568 tokens; D = 256, H = 2,
F = 1024, causal, bf16, about 106 GB of device buffers), so that the activations [T, D]
and [T, 3D] and the feature-major gradients [3D, T] hold more than 2^31 elements, and
the feature-major operands of the weight-gradient GEMMs have a row stride of 8.4M
elements, 255 rows of which pass 2^31.

dY is nonzero on three sequences (the first, one in the middle and the last) and zero
elsewhere. The layer treats every sequence on its own, and a sequence with dY = 0
contributes exact zeros to every gradient, so the float64 oracle on those three
sequences gives their Y and dX and every parameter gradient of the whole batch.
Compared: Y and dX of the three sequences and every parameter gradient, under the bf16
gates of the small-size tests (the rounding model on the same three sequences); dX of
every other sequence must be exactly zero and Y finite everywhere.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

from bpt_inputs import make_inputs, small_workload
from gpu_util import GRAD_NAMES, gpu_config, run_oracle, say
from paper_2305_19370_amd import bpt
from test_gpu_parity import compare_all

pytestmark = pytest.mark.gpu

B, S, D, H, F = 4116, 2048, 256, 2, 1024
PICK = (0, B // 2, B - 1)


def test_batch_past_int32_indexing():
    free, _ = torch.cuda.mem_get_info()
    if free < 120 * 2 ** 30:
        pytest.skip(f"needs about 120 GiB of free device memory, {free / 2 ** 30:.0f} GiB free")
    w = small_workload("bf16", B=B, S=S, D=D, H=H, F=F, causal=True, Bq=S, Bkv=S)
    T = B * S
    assert T * 255 > 2 ** 31 and T * D > 2 ** 31
    say(f"case large index: B={B} S={S} D={D} H={H} F={F} ({T} tokens); drawing inputs on the host")
    inp = make_inputs(w, seed=31, affine=True, biases=True)
    pick = torch.tensor(PICK)
    dY = torch.zeros_like(inp["dY"])
    dY[pick] = inp["dY"][pick]
    sub = {k: v for k, v in inp.items()}
    sub["X"], sub["dY"] = inp["X"][pick].clone(), dY[pick].clone()
    inp["dY"] = dY
    say("copying inputs to the device")
    dev = {k: (v.cuda() if v is not None else None) for k, v in inp.items()}
    del inp, dY
    layer = bpt.Layer(gpu_config(w, "f32"))
    say("forward")
    Y, saved = layer.forward(dev["X"], dev)
    say("backward")
    dX, grads = layer.backward(dev["X"], dev, saved, dev["dY"])
    torch.cuda.synchronize()
    say("whole-batch checks")
    assert bool(torch.isfinite(Y).all()), "non-finite Y"
    others = torch.ones(B, dtype=torch.bool, device="cuda")
    others[pick.cuda()] = False
    flat = dX.view(B, -1)
    hi, lo = flat.amax(dim=1), flat.amin(dim=1)     # per sequence, without a copy of dX
    assert float(hi[others].max()) == 0.0 and float(lo[others].min()) == 0.0, \
        "dX nonzero on a sequence with dY = 0"
    assert float(hi[~others].max()) > 0.0
    gpu = {"Y": Y[pick.cuda()].cpu(), "dX": dX[pick.cuda()].cpu()}
    gpu.update({k: v.cpu() for k, v in grads.items() if k in GRAD_NAMES})
    del dev, Y, dX, saved, grads
    torch.cuda.empty_cache()
    say("oracle on the three sequences")
    w3 = small_workload("bf16", B=len(PICK), S=S, D=D, H=H, F=F, causal=True, Bq=S, Bkv=S)
    Yr, _, g = run_oracle(w3, sub)
    assert np.isfinite(Yr).all()
    compare_all(w3, sub, gpu, Yr, g, "bf16", f"large index B={B} S={S} D={D}")
