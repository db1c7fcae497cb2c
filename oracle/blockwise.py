"""Algorithm 1 of the paper in float64 — TEST INFRASTRUCTURE (see ``oracle/__init__.py``).

Attention of a query block is assembled from its key/value blocks the way Section 3
combines blocks (eq. 3 and the rescaling that follows it): each key/value block j
on its own yields, per query row, a summary triple

    m_j = max_k s_k,   l_j = sum_k exp(s_k - m_j),   a_j = sum_k exp(s_k - m_j) v_k

over its keys k (s the scaled scores), and two summaries merge exactly into the
summary of their union by bringing both to the larger maximum:

    m = max(m_1, m_2),   l = l_1 e^(m_1 - m) + l_2 e^(m_2 - m),   a = a_1 e^(m_1 - m) + a_2 e^(m_2 - m).

Folding the blocks in key order and reading out a / l gives the query block's
attention, and m + log l its log-sum-exp. Then the output projection, the FFN and
both residuals are applied to that query block before the next one starts
(Algorithm 1's outer loop).

Bq and Bkv are block LENGTHS in tokens and need not divide S: the last block of a
sequence is shorter. Blocks are contiguous token ranges. A row whose keys in a
block are all masked has the empty summary (m = -inf, l = 0, a = 0), which the
merge leaves unchanged.

This is a second, independently structured route to the same numbers as
``oracle.layer``; the tests require the two to agree to ~1e-12 for many
(Bq, Bkv), which is the method's exactness claim.
"""
from __future__ import annotations

import math

import numpy as np

from .layer import LayerParams, act_fwd, layer_norm_fwd


def _block_summary(s, v):
    """(m, l, a) of one key/value block for every query row; s [nq, nk] scaled scores
    (-inf where masked), v [nk, dh]."""
    m = s.max(axis=1)
    e = np.exp(s - np.where(np.isfinite(m), m, 0.0)[:, None])     # 0 wherever s = -inf
    return m, e.sum(axis=1), e @ v


def _merge(x, y):
    """Summary of the union of two disjoint key sets from their summaries."""
    (m1, l1, a1), (m2, l2, a2) = x, y
    m = np.maximum(m1, m2)
    ref = np.where(np.isfinite(m), m, 0.0)
    c1, c2 = np.exp(m1 - ref), np.exp(m2 - ref)                     # exp(-inf) = 0 for empty ones
    return m, l1 * c1 + l2 * c2, a1 * c1[:, None] + a2 * c2[:, None]


def _attend_query_block(q_scaled, K, V, rows, causal, Bkv):
    """Attention of one query block (queries already divided by sqrt(dh); rows their
    absolute positions) against every key/value block. Returns (O [nq, dh], lse [nq])."""
    nq, dh = q_scaled.shape
    acc = (np.full(nq, -np.inf), np.zeros(nq), np.zeros((nq, dh)))   # the empty summary
    for k0 in range(0, K.shape[0], Bkv):
        k1 = min(k0 + Bkv, K.shape[0])
        s = q_scaled @ K[k0:k1].T
        if causal:
            s = np.where(np.arange(k0, k1)[None, :] <= rows[:, None], s, -np.inf)
        acc = _merge(acc, _block_summary(s, V[k0:k1]))
    m, l, a = acc
    return a / l[:, None], m + np.log(l)


def blockwise_attention_head(Q, K, V, causal: bool, Bq: int, Bkv: int):
    """Blockwise attention for one head; same contract as ``layer.attention_head``
    without P. Returns (O [S, dh], lse [S])."""
    S, dh = Q.shape
    O = np.empty_like(Q)
    lse = np.empty(S)
    for q0 in range(0, S, Bq):
        q1 = min(q0 + Bq, S)
        O[q0:q1], lse[q0:q1] = _attend_query_block(Q[q0:q1] / math.sqrt(dh), K, V,
                                                   np.arange(q0, q1), causal, Bkv)
    return O, lse


def blockwise_layer_fwd(X: np.ndarray, p: LayerParams, H: int, causal: bool, Bq: int, Bkv: int,
                        eps: float = 1e-5):
    """Algorithm 1 for the whole layer on X[B, S, D]. Returns (Y, O, lse)."""
    B, S, D = X.shape
    dh = D // H
    U, _, _ = layer_norm_fwd(X, p.ln1_g, p.ln1_b, eps)
    Q, K, V = U @ p.Wq, U @ p.Wk, U @ p.Wv          # project the input sequence
    Y = np.empty_like(X)
    O = np.empty_like(X)
    lse = np.empty((B, H, S))
    for b in range(B):
        for q0 in range(0, S, Bq):                  # outer loop over query blocks
            q1 = min(q0 + Bq, S)
            rows = np.arange(q0, q1)
            for h in range(H):                      # inner loop over key/value blocks
                cols = slice(h * dh, (h + 1) * dh)
                O[b, q0:q1, cols], lse[b, h, q0:q1] = _attend_query_block(
                    Q[b, q0:q1, cols] / math.sqrt(dh), K[b, :, cols], V[b, :, cols],
                    rows, causal, Bkv)
            # feed-forward and residuals on this query block before the next one
            hd = X[b, q0:q1] + O[b, q0:q1] @ p.Wo
            vn, _, _ = layer_norm_fwd(hd, p.ln2_g, p.ln2_b, eps)
            z = vn @ p.W1
            if p.b1 is not None:
                z = z + p.b1
            y = hd + act_fwd(p, z) @ p.W2
            if p.b2 is not None:
                y = y + p.b2
            Y[b, q0:q1] = y
    return Y, O, lse
