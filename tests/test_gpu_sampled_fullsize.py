"""Full-size sampled parity: the 7B-, RL- and 13B-shaped layers at their full sequence
lengths, the 13B-shaped layer at S = 8192 and 32768 of its sweep, and a 1B-width layer
with heads of 64 and no causal mask at S = 32768, run through the
C ABI in the launch configuration bench.py times (automatic FFN grouping; outputs
stored in fp32 here, which changes only the final store of Y and dX), against float64
values the rows oracle computed on the same seeded inputs (written by
tests/expected/make_fullsize.py, which calls only oracle/ and the input generator).

The upstream gradient is dY on about 270 selected rows (spread over the query tiles of
8192-row windows at the start, the middle and the end of the sequence) and zero
elsewhere; the rows oracle's gradients are then the exact full backward values.
Compared: Y and dX on every fourth selected row (every element, normalised by the RMS
of those rows of the reference), dX at 2048 positions sampled on the other rows (its
gradient through the keys and values only) and every parameter gradient at 2048 sampled
positions (normalised by the RMS of the reference at those positions). Gate, per quantity, as in
the small-size bf16 parity tests: e_max <= max(2e-2, F_max x the bf16 rounding model's
e_max) and e_mean <= max(2e-3, F_mean x the model's e_mean), F from
tests/expected/model_factors.json; the model (oracle/bf16_rows.py, every
matrix-multiply operand rounded to bf16) is evaluated on the same rows and samples by
the same script.
"""
from __future__ import annotations

import os
import sys

import numpy as np
import pytest
import torch

from bpt_inputs import make_inputs, workload
from gpu_util import GRAD_NAMES, bf16_limits, run_gpu, say, table

sys.path.insert(0, os.path.join(os.path.dirname(os.path.abspath(__file__)), "expected"))
from make_fullsize import FULLSIZE, checks, errors, expected_path  # noqa: E402

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name", FULLSIZE)
def test_fullsize_sampled(name):
    e = np.load(expected_path(name))
    w = workload(name)
    say(f"case full-size {name}: B={w.B} S={w.S} D={w.D} H={w.H} F={w.F} Bq={w.Bq}")
    inp = make_inputs(w, seed=int(e["seed"]))
    rows = torch.from_numpy(e["rows"])
    dY = torch.zeros_like(inp["dY"])
    dY[:, rows] = inp["dY"][:, rows]
    inp["dY"] = dY
    gpu = run_gpu(w, inp, out_dtype="f32")
    del inp
    res = {"Y_rows": gpu["Y"][:, torch.from_numpy(e["check_rows"])].numpy(), "dX": gpu["dX"].numpy()}
    res.update({k: gpu[k].numpy() for k in GRAD_NAMES if k in gpu})
    rows_out, bad = [], []
    for n, got, ref, norm in checks(e, res):
        assert np.isfinite(got).all(), f"non-finite values in GPU {n}"
        e_max, e_mean = errors(got, ref, norm)
        m_max, m_mean = e["model_" + n.replace(" ", "_")]
        lim_max, lim_mean = bf16_limits({"e_max": float(m_max), "e_mean": float(m_mean)})
        d = np.abs(np.asarray(got, np.float64) - ref)
        rows_out.append((n, dict(max_abs=float(d.max()), mean_abs=float(d.mean()), rms=norm, e_max=e_max,
                                 e_mean=e_mean, lim_max=lim_max, lim_mean=lim_mean)))
        if not (e_max <= lim_max and e_mean <= lim_mean):
            bad.append(n)
    say(f"\n[{name}]\n" + table(rows_out))
    assert not bad, f"{name}: out of tolerance: {bad}"
