"""Full-size sampled parity: the 7B-, RL- and 13B-shaped layers at their full sequence
lengths, run through the C ABI in the launch configuration bench.py times (automatic
FFN grouping; outputs stored in fp32 here, which changes only the final store of Y and
dX), against float64 values the rows oracle computed on the same seeded inputs
(written by tests/expected/make_fullsize.py, which calls only oracle/ and the input
generator).

The upstream gradient is dY on a few selected rows and zero elsewhere; the rows
oracle's gradients are then the exact full backward values. Compared: Y and dX at the
selected rows (every element), dX and every parameter gradient at 2048 sampled
positions. Gate, per quantity: e_mean <= max(2e-3, 1.25 x the bf16 rounding model's
e_mean), as in the small-size bf16 parity tests, and e_max <= max(2e-2, 2 x the
model's e_max), errors normalised by the reference RMS; the model (oracle/bf16_rows.py,
every matrix-multiply operand rounded to bf16) is evaluated on the same rows and
samples by the same script. The wider factor on the maximum: with dY on a few rows,
each sampled weight-gradient element is a sum dominated by a few tokens, so its error
is set by the bf16 rounding of a handful of operands, and which elements round up or
down differs between any two implementations (the GPU's mean error stays within 1.05x
of the model's while the maximum over 2048 samples reaches 1.7x on the 7B layer).
"""
from __future__ import annotations

import os
import sys

import numpy as np
import pytest
import torch

from bpt_inputs import WORKLOADS, make_inputs
from gpu_util import GRAD_NAMES, run_gpu, say, table

sys.path.insert(0, os.path.join(os.path.dirname(os.path.abspath(__file__)), "expected"))
from make_fullsize import checks, errors, expected_path  # noqa: E402

pytestmark = pytest.mark.gpu

E_MAX, E_MEAN = 2e-2, 2e-3
MODEL_FACTOR_MAX, MODEL_FACTOR_MEAN = 2.0, 1.25


@pytest.mark.parametrize("name", ["bf16_7b_s32768", "bf16_rl_s96000", "bf16_13b_s65536"])
def test_fullsize_sampled(name):
    e = np.load(expected_path(name))
    w = WORKLOADS[name]
    say(f"case full-size {name}: B={w.B} S={w.S} D={w.D} H={w.H} F={w.F} Bq={w.Bq}")
    inp = make_inputs(w, seed=int(e["seed"]))
    rows = torch.from_numpy(e["rows"])
    dY = torch.zeros_like(inp["dY"])
    dY[:, rows] = inp["dY"][:, rows]
    inp["dY"] = dY
    gpu = run_gpu(w, inp, out_dtype="f32")
    del inp
    res = {"Y_rows": gpu["Y"][:, rows].numpy(), "dX": gpu["dX"].numpy()}
    res.update({k: gpu[k].numpy() for k in GRAD_NAMES if k in gpu})
    rows_out, bad = [], []
    for n, got, ref, norm in checks(e, res):
        assert np.isfinite(got).all(), f"non-finite values in GPU {n}"
        e_max, e_mean = errors(got, ref, norm)
        m_max, m_mean = e["model_" + n.replace(" ", "_")]
        lim_max, lim_mean = max(E_MAX, MODEL_FACTOR_MAX * m_max), max(E_MEAN, MODEL_FACTOR_MEAN * m_mean)
        d = np.abs(np.asarray(got, np.float64) - ref)
        rows_out.append((n, dict(max_abs=float(d.max()), mean_abs=float(d.mean()), rms=norm, e_max=e_max,
                                 e_mean=e_mean, lim_max=lim_max, lim_mean=lim_mean)))
        if not (e_max <= lim_max and e_mean <= lim_mean):
            bad.append(n)
    say(f"\n[{name}]\n" + table(rows_out))
    assert not bad, f"{name}: out of tolerance: {bad}"
