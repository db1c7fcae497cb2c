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
