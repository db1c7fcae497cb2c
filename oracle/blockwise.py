"""Algorithm 1 of the paper in float64 — TEST INFRASTRUCTURE (see ``oracle/__init__.py``).

For each query block (rows [i*Bq, min((i+1)*Bq, S)) of one sequence), iterate
over the key/value blocks (rows [j*Bkv, ...)), keep per query row a running
maximum, a running numerator and a running denominator, and rescale them by
exp(old_max - new_max) whenever the maximum grows (the carry update of
Section 3 and Fig. 3: numerator * correction + exp(scores - max) V, likewise
for the denominator). Once every key/value block has been visited the block's
attention is numerator / denominator, after which the output projection, the
FFN and both residuals are applied to that query block before the next query
block starts (Algorithm 1, last two steps of the outer loop).

Bq and Bkv are block LENGTHS in tokens and need not divide S: the last block
of a sequence is shorter. Blocks are contiguous token ranges.

This is a second, independently structured route to the same numbers as
``oracle.layer``; the tests require the two to agree to ~1e-12 for many
(Bq, Bkv), which is the method's exactness claim.
"""
from __future__ import annotations

import math

import numpy as np

from .layer import LayerParams, act_fwd, layer_norm_fwd


def _attend_query_block(q_scaled, K, V, rows, causal, Bkv):
    """Online-softmax attention of one query block against all key/value blocks.

    q_scaled: [nq, dh] queries already divided by sqrt(dh) (the listing scales
    the query once up front). rows: absolute positions of the queries.
    Returns (attention [nq, dh], log-sum-exp [nq])."""
    nq, dh = q_scaled.shape
    S_kv = K.shape[0]
    numerator = np.zeros((nq, dh))
    denominator = np.zeros(nq)
    running_max = np.full(nq, -np.inf)
    for k0 in range(0, S_kv, Bkv):
        k1 = min(k0 + Bkv, S_kv)
        scores = q_scaled @ K[k0:k1].T                       # scores of this block pair
        if causal:
            keys = np.arange(k0, k1)
            scores = np.where(keys[None, :] <= rows[:, None], scores, -np.inf)
        new_max = np.maximum(running_max, scores.max(axis=1))
        # A row that has seen only masked keys so far keeps max = -inf; its weights
        # and its correction are exactly 0 (avoids -inf - -inf).
        ref = np.where(np.isfinite(new_max), new_max, 0.0)
        weights = np.exp(scores - ref[:, None])
        correction = np.exp(running_max - ref)
        numerator = numerator * correction[:, None] + weights @ V[k0:k1]
        denominator = denominator * correction + weights.sum(axis=1)
        running_max = new_max
    return numerator / denominator[:, None], running_max + np.log(denominator)


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
