"""Dropout masks of the layer's residual branches, float64 side — TEST INFRASTRUCTURE ONLY.

The paper's memory accounting of a BPT layer keeps one dropout mask for the output
projection and one for the FFN output, and its RL runs use a rate of 0.1. The mask is
random, so both sides draw it from one counter-based generator written from its
published definition: Philox4x32 with 10 rounds (Salmon, Moraes, Dror and Shaw,
"Parallel random numbers: as easy as 1, 2, 3", SC 2011). The oracle and the GPU
library each implement it on their own.

Element (t, n) of a [T, D] branch output (t the token index over the whole batch,
b*S + s; n the column) at site k (0: the attention output projection, 1: the FFN
output) takes word n mod 4 of Philox4x32-10 with counter (n div 4, t, k, 0) and key
(seed mod 2^32, seed div 2^32). It is kept iff that word is >= floor(p * 2^32),
and a kept value is scaled by 1 / (1 - p).
"""
from __future__ import annotations

import numpy as np

_M0, _M1 = 0xD2511F53, 0xCD9E8D57          # round multipliers
_W0, _W1 = 0x9E3779B9, 0xBB67AE85          # Weyl key increments
_MASK = np.uint64(0xFFFFFFFF)


def philox4x32_10(c0, c1, c2, c3, k0: int, k1: int):
    """Philox4x32-10 on arrays of 32-bit counter words (any common shape); returns the
    four output words as uint64 arrays holding 32-bit values."""
    c = [np.asarray(x, dtype=np.uint64) & _MASK for x in (c0, c1, c2, c3)]
    k0, k1 = np.uint64(k0 & 0xFFFFFFFF), np.uint64(k1 & 0xFFFFFFFF)
    for r in range(10):
        if r:
            k0 = (k0 + np.uint64(_W0)) & _MASK
            k1 = (k1 + np.uint64(_W1)) & _MASK
        p0 = np.uint64(_M0) * c[0]           # < 2^64: exact in uint64
        p1 = np.uint64(_M1) * c[2]
        c = [((p1 >> np.uint64(32)) ^ c[1] ^ k0) & _MASK, p1 & _MASK,
             ((p0 >> np.uint64(32)) ^ c[3] ^ k1) & _MASK, p0 & _MASK]
    return c


def threshold(p: float) -> int:
    """floor(p * 2^32) for the rate p as a float32 value."""
    return int(np.floor(float(np.float32(p)) * 2.0 ** 32))


def keep_mask(T: int, D: int, seed: int, site: int, p: float) -> np.ndarray:
    """Boolean [T, D]: which elements of a branch output survive dropout at rate p."""
    if p <= 0.0:
        return np.ones((T, D), dtype=bool)
    t = np.arange(T, dtype=np.uint64)[:, None]
    n = np.arange(D, dtype=np.uint64)[None, :]
    words = philox4x32_10(n // np.uint64(4), np.broadcast_to(t, (T, D)), np.full((T, D), site, np.uint64),
                          np.zeros((T, D), np.uint64), seed & 0xFFFFFFFF, (seed >> 32) & 0xFFFFFFFF)
    w = np.select([(n % np.uint64(4)) == np.uint64(i) for i in range(4)], words)
    return w >= np.uint64(threshold(p))


def dropout_factor(T: int, D: int, seed: int, site: int, p: float) -> np.ndarray:
    """float64 [T, D]: 0 where dropped, 1 / (1 - p) where kept."""
    return keep_mask(T, D, seed, site, p) / (1.0 - float(np.float32(p)))
