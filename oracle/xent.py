"""Cross-entropy of a language-model head, float64 — TEST INFRASTRUCTURE ONLY.

Section 3 of the paper remarks that the blockwise scheme carries over to the final
cross-entropy loss: the [T, V] logits of the vocabulary projection never need to
exist at once. The result it must reproduce is the plain definition, written out
unblocked here:

    logits = h W                      h[T, D], W[D, V] (y = x @ W); a W stored with
                                      more columns than V has them ignored
    lse_t  = log sum_v exp(logits[t, v])
    loss   = (1/T) sum_t (lse_t - logits[t, y_t])

and, for an upstream gradient g of the loss,

    G  = (g / T) (softmax(logits) - onehot(y))        [T, V]
    dh = G W^T,    dW = h^T G.

A target outside [0, V) gives that token a NaN loss (so the mean is NaN) and no
one-hot term in G; the GPU library documents the same behaviour.
"""
from __future__ import annotations

from typing import Dict

import numpy as np


def xent_logits(h: np.ndarray, W: np.ndarray, V: int) -> np.ndarray:
    """h[T, D] @ W[D, >= V], the first V columns, float64."""
    return np.asarray(h, dtype=np.float64) @ np.asarray(W, dtype=np.float64)[:, :V]


def xent_fwd(h: np.ndarray, W: np.ndarray, targets: np.ndarray, V: int) -> Dict[str, np.ndarray]:
    """Returns loss (scalar), lse [T] and the per-token losses [T]."""
    z = xent_logits(h, W, V)
    T = z.shape[0]
    m = z.max(axis=1)
    lse = m + np.log(np.exp(z - m[:, None]).sum(axis=1))
    y = np.asarray(targets, dtype=np.int64)
    ok = (y >= 0) & (y < V)
    zy = np.where(ok, z[np.arange(T), np.clip(y, 0, V - 1)], np.nan)
    tok = lse - zy
    return dict(loss=tok.sum() / T, lse=lse, token_loss=tok)


def xent_grad_logits(z: np.ndarray, lse: np.ndarray, targets: np.ndarray, g: float) -> np.ndarray:
    """G = (g / T) (softmax(z) - onehot(y)) from the logits and their log-sum-exp."""
    T, V = z.shape
    G = np.exp(z - lse[:, None])
    y = np.asarray(targets, dtype=np.int64)
    ok = (y >= 0) & (y < V)
    G[np.arange(T)[ok], y[ok]] -= 1.0
    return G * (g / T)


def xent_bwd(h: np.ndarray, W: np.ndarray, targets: np.ndarray, V: int, g: float = 1.0,
             round_g=None) -> Dict[str, np.ndarray]:
    """dh [T, D] and dW [D, V] of the mean loss times g. ``round_g``, if given, is
    applied to G before the two products (the bf16 rounding model passes its
    rounding function)."""
    z = xent_logits(h, W, V)
    lse = xent_fwd(h, W, targets, V)["lse"]
    G = xent_grad_logits(z, lse, targets, g)
    if round_g is not None:
        G = round_g(G)
    h64 = np.asarray(h, dtype=np.float64)
    return dict(dh=G @ np.asarray(W, dtype=np.float64)[:, :V].T, dW=h64.T @ G, G=G)


# ---------------------------------------------------------------- restricted to rows / columns
def xent_lse_rows(h: np.ndarray, W: np.ndarray, V: int, chunk: int = 1024) -> np.ndarray:
    """lse of every token, computed chunk by chunk of tokens (each row is independent,
    so this is the plain definition; it only bounds the memory of the logits)."""
    out = np.empty(h.shape[0])
    for t0 in range(0, h.shape[0], chunk):
        z = xent_logits(h[t0:t0 + chunk], W, V)
        m = z.max(axis=1)
        out[t0:t0 + chunk] = m + np.log(np.exp(z - m[:, None]).sum(axis=1))
    return out


def xent_dh_rows(h: np.ndarray, W: np.ndarray, targets: np.ndarray, V: int, rows: np.ndarray, T: int,
                 g: float = 1.0, round_g=None) -> np.ndarray:
    """dh of the selected tokens (T = all tokens, for the 1/T of the mean)."""
    z = xent_logits(h[rows], W, V)
    m = z.max(axis=1)
    lse = m + np.log(np.exp(z - m[:, None]).sum(axis=1))
    G = np.exp(z - lse[:, None])
    y = np.asarray(targets, dtype=np.int64)[rows]
    ok = (y >= 0) & (y < V)
    G[np.arange(len(rows))[ok], y[ok]] -= 1.0
    G *= g / T
    if round_g is not None:
        G = round_g(G)
    return G @ np.asarray(W, dtype=np.float64)[:, :V].T


def xent_dW_cols(h: np.ndarray, W: np.ndarray, targets: np.ndarray, lse: np.ndarray, cols: np.ndarray,
                 g: float = 1.0, round_g=None) -> np.ndarray:
    """Columns `cols` of dW = h^T G, from the exact lse of every token."""
    h64 = np.asarray(h, dtype=np.float64)
    T = h64.shape[0]
    z = h64 @ np.asarray(W, dtype=np.float64)[:, cols]            # [T, len(cols)]
    G = np.exp(z - lse[:, None])
    y = np.asarray(targets, dtype=np.int64)
    G -= (y[:, None] == np.asarray(cols)[None, :])
    G *= g / T
    if round_g is not None:
        G = round_g(G)
    return h64.T @ G
