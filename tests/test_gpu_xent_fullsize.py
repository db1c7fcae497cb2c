"""Full-size parity of the LM-head cross-entropy, on sampled outputs: the GPU runs the
shape and launch configuration `bench.py --xent` times (T=32768, D=4096, V=50257 in
50304 stored columns, bf16, 8192-token blocks); the float64 oracle values at 16
sampled tokens and 16 sampled columns of dW were written by
tests/expected/make_xent_fullsize.py (oracle/ only).

Gates: loss |diff| <= 1e-5 |loss|; lse |diff| <= 1e-5 max|lse|; dh rows and dW columns
e_max <= max(2e-2, F_max x the G-rounding model's), e_mean <= max(2e-3, F_mean x), with
e = |diff| / rms(ref over the samples). Two properties that hold at any size are
checked on the whole outputs: every row of dW sums to zero over the vocabulary (the
softmax minus one-hot has zero row sums), and <dW, W> = <dh, h> (both are
sum_t sum_v G[t, v] (h_t . W_v))."""
import os

import numpy as np
import pytest
import torch

from bpt_inputs import make_xent_inputs
from gpu_util import bf16_limits, say, stats, table
from paper_2305_19370_amd import bpt

pytestmark = pytest.mark.gpu
EXPECTED = os.path.join(os.path.dirname(__file__), "expected", "xent_fullsize_t32768_d4096_v50257.npz")


def test_xent_fullsize_sampled():
    e = np.load(EXPECTED, allow_pickle=False)
    T, D, V, ldw = int(e["T"]), int(e["D"]), int(e["V"]), int(e["ldw"])
    say(f"case xent full size T={T} D={D} V={V}")
    inp = make_xent_inputs(T, D, V, ldw, "bf16", seed=0)
    h, W, y = inp["h"].cuda(), inp["W"].cuda(), inp["targets"].cuda()
    del inp
    head = bpt.LMHeadLoss(bpt.make_xent_config(T, D, V, ldw, 0, "bf16"))
    loss, lse = head.forward(h, W, y)
    dh, dW = head.backward(h, W, y, lse, 1.0)
    torch.cuda.synchronize()
    rows, cols = e["rows"], e["cols"]
    bad = []
    g_loss = float(loss.item())
    say(f"loss gpu {g_loss:.9f} oracle {float(e['loss']):.9f}")
    if not abs(g_loss - float(e["loss"])) <= 1e-5 * abs(float(e["loss"])):
        bad.append("loss")
    g_lse = lse.cpu().double().numpy()[rows]
    if not np.abs(g_lse - e["lse"]).max() <= 1e-5 * np.abs(e["lse"]).max():
        bad.append("lse")
    out = []
    for name, got, ref, model in (("dh rows", dh.float().cpu().double().numpy()[rows], e["dh"], e["dh_model"]),
                                  ("dW cols", dW.cpu().double().numpy()[:, cols], e["dW"], e["dW_model"])):
        s, ms = stats(got, ref), stats(model, ref)
        s["lim_max"], s["lim_mean"] = bf16_limits(ms)
        out.append((name, s))
        if not (s["e_max"] <= s["lim_max"] and s["e_mean"] <= s["lim_mean"]):
            bad.append(name)
    say(table(out))
    # properties of the whole outputs
    dW64 = dW[:, :V].double()
    row_sums = dW64.sum(dim=1).abs().max().item()
    scale = dW64.abs().sum(dim=1).max().item()
    lhs = (dW64 * W[:, :V].double()).sum().item()
    rhs = (dh.double() * h.double()).sum().item()
    say(f"max |row sum of dW| {row_sums:.3e} (row abs sum {scale:.3e}); <dW,W> {lhs:.6e} <dh,h> {rhs:.6e}")
    if not row_sums <= 1e-3 * scale:
        bad.append("dW row sums")
    if not abs(lhs - rhs) <= 1e-3 * max(abs(lhs), abs(rhs), 1e-30):
        bad.append("<dW,W> = <dh,h>")
    assert not bad, bad
