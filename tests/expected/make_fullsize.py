"""Writes the expected values of the full-size sampled parity tests — run on the CPU.

For each long-context workload (the 7B-, RL- and 13B-shaped layers at their full
sequence lengths) the float64 rows oracle (``oracle/rows.py``: the plain layer
definition restricted to selected query rows) is evaluated on the seeded inputs
of ``bpt_inputs.make_inputs(w, seed=0)`` with the upstream gradient equal to dY
on the selected rows and zero elsewhere. Under that dY every gradient the rows
oracle returns is the exact full backward value, so the GPU run (same inputs,
same masked dY, full size) can be compared on:

  * Y and dX at the selected rows (every element; errors normalised by the RMS of
    those rows of the reference);
  * dX and every weight / bias / LayerNorm gradient at 2048 sampled positions
    (normalised by the RMS of the full reference tensor);

The bf16 rounding model restricted to the same rows (``oracle/bf16_rows.py``) is
evaluated too, and its normalised errors on exactly these checks are stored: they
set the floor of the tolerance for tensors whose error is dominated by bf16 operand
rounding, as in the small-size parity tests. Only ``oracle/`` and the input generator
are used; nothing here comes from the HIP path.

    python tests/expected/make_fullsize.py bf16_7b_s32768 [more workloads]
"""
from __future__ import annotations

import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

NSAMPLE = 2048
SEED = 0
GRADS = ("dWq", "dWk", "dWv", "dWo", "dW1", "dW2", "db1", "db2", "dln1_g", "dln1_b", "dln2_g", "dln2_b")


def sample_rows(S: int) -> np.ndarray:
    """First tokens, both sides of the first FFN-group boundary (8192 rows), the middle,
    and the last two tokens of the sequence."""
    return np.array(sorted({0, 1, 8191, 8192, S // 2 + 1, S - 2, S - 1}), dtype=np.int64)


def expected_path(name: str) -> str:
    return os.path.join(HERE, f"fullsize_{name}.npz")


def rms(a) -> float:
    a = np.asarray(a, dtype=np.float64)
    return float(np.sqrt(np.mean(a * a)))


def checks(e, res):
    """(name, values of `res`, reference values, normaliser) for every compared quantity.
    `e`: the stored expectations; `res`: a result dict holding Y rows ("Y_rows" [B, R, D])
    and full-size dX and gradients (numpy arrays)."""
    rows = e["rows"]
    out = [("Y rows", res["Y_rows"], e["Y_rows"], rms(e["Y_rows"])),
           ("dX rows", res["dX"][:, rows], e["dX_rows"], rms(e["dX_rows"]))]
    for k in ("dX",) + GRADS:
        if k + "_idx" not in e.files:
            continue
        got = np.asarray(res[k])
        assert tuple(got.shape) == tuple(e[k + "_shape"]), (k, got.shape)
        out.append((k, got.reshape(-1)[e[k + "_idx"]], e[k + "_val"], float(e[k + "_rms"])))
    return out


def errors(got, ref, norm):
    d = np.abs(np.asarray(got, dtype=np.float64) - np.asarray(ref, dtype=np.float64))
    norm = norm or 1.0
    return float(d.max()) / norm, float(d.mean()) / norm


def make(name: str) -> str:
    import oracle
    from oracle.bf16_rows import bf16_rows_fwd_bwd
    from bpt_inputs import WORKLOADS, make_inputs
    w = WORKLOADS[name]
    t0 = time.time()
    inp = make_inputs(w, seed=SEED)
    p = oracle.params_from_inputs(inp)
    X = inp["X"].double().numpy()
    rows = sample_rows(w.S)
    dY_rows = inp["dY"].double().numpy()[:, rows]
    del inp
    Y, g = oracle.rows_layer_fwd_bwd(X, p, w.H, w.causal, rows, dY_rows)
    rng = np.random.default_rng(1234)
    out = {"rows": rows, "seed": np.int64(SEED), "Y_rows": Y, "dX_rows": g["dX"][:, rows]}
    for k in ("dX",) + GRADS:
        v = g.get(k)
        if v is None:
            continue
        idx = rng.choice(v.size, size=min(NSAMPLE, v.size), replace=False)
        out[k + "_idx"] = idx.astype(np.int64)
        out[k + "_val"] = v.reshape(-1)[idx]
        out[k + "_rms"] = np.float64(rms(v))
        out[k + "_shape"] = np.array(v.shape, dtype=np.int64)
    del g
    t1 = time.time()
    m = bf16_rows_fwd_bwd(X, p, w.H, w.causal, rows, dY_rows)
    m["Y_rows"] = m.pop("Y")

    class _E(dict):
        files = property(lambda self: list(self.keys()))
    for n, got, ref, norm in checks(_E(out), m):
        out["model_" + n.replace(" ", "_")] = np.array(errors(got, ref, norm))
    path = expected_path(name)
    np.savez_compressed(path, **out)
    print(f"{name}: rows {rows.tolist()}, oracle {t1 - t0:.0f} s, model {time.time() - t1:.0f} s -> {path}",
          flush=True)
    return path


if __name__ == "__main__":
    for n in sys.argv[1:] or ["bf16_7b_s32768", "bf16_rl_s96000", "bf16_13b_s65536"]:
        make(n)
