"""Writes the expected values of the full-size sampled parity tests — run on the CPU.

For each long-context workload (the 7B-, RL- and 13B-shaped layers at their full
sequence lengths, the 13B-shaped layer at two shorter lengths of its sweep, and a
1B-width layer with heads of 64 and no causal mask at S = 32768) the
float64 rows oracle (``oracle/rows.py``: the plain layer definition restricted to
selected query rows) is evaluated on the seeded inputs of
``bpt_inputs.make_inputs(w, seed=0)`` with the upstream gradient equal to dY on the
selected rows and zero elsewhere. Under that dY every gradient the rows oracle
returns is the exact full backward value, so the GPU run (same inputs, same masked
dY, full size) can be compared on:

  * Y and dX on every fourth selected row (every element; errors normalised by the RMS
    of those rows of the reference; stored in float32, whose rounding, 6e-8 relative,
    is far below any bf16 tolerance);
  * dX at 2048 positions sampled on the other rows (whose gradient comes only through
    the keys and values), and every weight / bias / LayerNorm gradient at 2048 sampled
    positions (errors normalised by the RMS of the reference at the sampled positions);

The selected rows (about 270) are spread over the query tiles of three windows of
8192 rows (half an automatic FFN group at the 7B and 13B shapes, a quarter of one at the
RL shape): the start, the middle and the end of the sequence, plus the first and last two
tokens, so that the attention backward sees nonzero gradients on query tiles of every
part of the causal triangle.

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


GROUP_ROWS = 8192          # window rows (half an automatic FFN group at F >= 8192)
PER_WINDOW = 88


def sample_rows(S: int) -> np.ndarray:
    """PER_WINDOW rows in each of three windows of GROUP_ROWS rows (start, middle and end
    of the sequence), one per stride of GROUP_ROWS / PER_WINDOW at a seeded offset inside
    the stride, plus tokens 0, 1, S-2, S-1 and both sides of row GROUP_ROWS."""
    rng = np.random.default_rng(S)
    rows = {0, 1, S - 2, S - 1, GROUP_ROWS - 1, GROUP_ROWS}
    for w0 in (0, max(0, S // 2 - GROUP_ROWS // 2), max(0, S - GROUP_ROWS)):
        n = min(GROUP_ROWS, S - w0)
        stride = n // PER_WINDOW
        for i in range(PER_WINDOW):
            rows.add(w0 + i * stride + int(rng.integers(0, stride)))
    return np.array(sorted(r for r in rows if 0 <= r < S), dtype=np.int64)


FULLSIZE = ("bf16_7b_s32768", "bf16_rl_s96000", "bf16_13b_s65536", "bf16_13b_s8192", "bf16_13b_s32768",
            "bf16_dh64_nc_s32768")


def expected_path(name: str) -> str:
    return os.path.join(HERE, f"fullsize_{name}.npz")


def rms(a) -> float:
    a = np.asarray(a, dtype=np.float64)
    return float(np.sqrt(np.mean(a * a)))


def checks(e, res):
    """(name, values of `res`, reference values, normaliser) for every compared quantity.
    `e`: the stored expectations; `res`: a result dict holding Y at the checked rows
    ("Y_rows" [B, R, D], R = len(e["check_rows"])) and full-size dX and gradients (numpy
    arrays)."""
    rows = e["check_rows"]
    out = [("Y rows", res["Y_rows"], e["Y_rows"], rms(e["Y_rows"])),
           ("dX rows", res["dX"][:, rows], e["dX_rows"], rms(e["dX_rows"]))]
    for k in ("dX",) + GRADS:
        if k + "_idx" not in e.files:
            continue
        got = np.asarray(res[k])
        assert tuple(got.shape) == tuple(e[k + "_shape"]), (k, got.shape)
        out.append((k, got.reshape(-1)[e[k + "_idx"]], e[k + "_val"], rms(e[k + "_val"])))
    return out


def errors(got, ref, norm):
    d = np.abs(np.asarray(got, dtype=np.float64) - np.asarray(ref, dtype=np.float64))
    norm = norm or 1.0
    return float(d.max()) / norm, float(d.mean()) / norm


def make(name: str) -> str:
    import oracle
    from oracle.bf16_rows import bf16_rows_fwd_bwd
    from bpt_inputs import make_inputs, workload
    w = workload(name)
    t0 = time.time()
    inp = make_inputs(w, seed=SEED)
    p = oracle.params_from_inputs(inp)
    X = inp["X"].double().numpy()
    rows = sample_rows(w.S)
    dY_rows = inp["dY"].double().numpy()[:, rows]
    del inp
    Y, g = oracle.rows_layer_fwd_bwd(X, p, w.H, w.causal, rows, dY_rows)
    rng = np.random.default_rng(1234)
    sel = np.arange(0, rows.size, 4)                 # Y and dX compared in full on these rows
    check_rows = rows[sel]
    out = {"rows": rows, "check_rows": check_rows, "seed": np.int64(SEED),
           "Y_rows": Y[:, sel].astype(np.float32), "dX_rows": g["dX"][:, check_rows].astype(np.float32)}
    for k in ("dX",) + GRADS:
        v = g.get(k)
        if v is None:
            continue
        if k == "dX":
            # positions on rows outside the selected ones: the selected rows are compared in
            # full above, and mixing the two populations would leave the statistics of the
            # sample to the few positions that fall on selected rows
            B_, S_, D_ = v.shape
            off = np.setdiff1d(np.arange(S_), rows)
            j = rng.choice(B_ * off.size * D_, size=min(NSAMPLE, B_ * off.size * D_), replace=False)
            bb, rem = j // (off.size * D_), j % (off.size * D_)
            idx = (bb * S_ + off[rem // D_]) * D_ + rem % D_
        else:
            idx = rng.choice(v.size, size=min(NSAMPLE, v.size), replace=False)
        out[k + "_idx"] = idx.astype(np.int64)
        out[k + "_val"] = v.reshape(-1)[idx]
        out[k + "_shape"] = np.array(v.shape, dtype=np.int64)
    del g
    t1 = time.time()
    m = bf16_rows_fwd_bwd(X, p, w.H, w.causal, rows, dY_rows)
    m["Y_rows"] = m.pop("Y")[:, sel]

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
    for n in sys.argv[1:] or FULLSIZE:
        make(n)
