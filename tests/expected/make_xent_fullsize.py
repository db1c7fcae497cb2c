"""Writes the expected values of the full-size sampled parity test of the LM-head
cross-entropy — run on the CPU.

Shape: the one `bench.py --xent` times (T=32768 tokens, D=4096, V=50257 stored with
50304 columns), inputs from ``bpt_inputs.make_xent_inputs(..., seed=0)``. With the
float64 oracle (``oracle/xent.py``) it stores:

  * the mean loss, from the exact log-sum-exp of every token (computed 1024 tokens at
    a time; each token is independent);
  * lse and dh at 16 sampled tokens (block boundaries of the 8192-token blocks, the
    ends, random others);
  * 16 sampled columns of dW (first, last, around 64-column boundaries, random);
  * dh and dW at the same samples under the rounding model (G rounded to bf16), which
    sets the tolerance floor as in the small-size tests.

Only ``oracle/`` and the input generator are used; nothing here comes from the HIP path.

    python tests/expected/make_xent_fullsize.py
"""
from __future__ import annotations

import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

from bpt_inputs import make_xent_inputs  # noqa: E402
from oracle.bf16_model import to_bf16  # noqa: E402
from oracle.xent import xent_dh_rows, xent_dW_cols, xent_lse_rows  # noqa: E402

T, D, V = 32768, 4096, 50257
LDW = (V + 63) // 64 * 64
OUT = os.path.join(HERE, "xent_fullsize_t32768_d4096_v50257.npz")


def main() -> None:
    t0 = time.time()
    inp = make_xent_inputs(T, D, V, LDW, "bf16", seed=0)
    h, W, y = inp["h"].double().numpy(), inp["W"].double().numpy(), inp["targets"].numpy()
    del inp
    rng = np.random.default_rng(12345)
    rows = np.unique(np.concatenate([[0, 1, 8191, 8192, 16383, 16384, 24576, T - 2, T - 1],
                                     rng.choice(T, 7, replace=False)]))
    cols = np.unique(np.concatenate([[0, 1, 63, 64, 127, 25000, V - 2, V - 1],
                                     rng.choice(V, 8, replace=False)]))
    lse = xent_lse_rows(h, W, V)
    zy = np.einsum("td,td->t", h, W[:, y].T)
    loss = float(np.mean(lse - zy))
    print(f"lse of all tokens: {time.time() - t0:.1f} s, loss {loss:.9f}", flush=True)
    dh = xent_dh_rows(h, W, y, V, rows, T)
    dh_model = xent_dh_rows(h, W, y, V, rows, T, round_g=to_bf16)
    dW = xent_dW_cols(h, W, y, lse, cols)
    dW_model = xent_dW_cols(h, W, y, lse, cols, round_g=to_bf16)
    np.savez_compressed(OUT, rows=rows, cols=cols, loss=loss, lse=lse[rows], dh=dh, dh_model=dh_model,
                        dW=dW, dW_model=dW_model, T=T, D=D, V=V, ldw=LDW)
    print(f"wrote {OUT} in {time.time() - t0:.1f} s", flush=True)


if __name__ == "__main__":
    main()
