"""The bf16-operand rounding model restricted to selected query rows — TEST INFRASTRUCTURE.

(See ``oracle/__init__.py``.) ``oracle/bf16_model.py`` evaluated only where
``oracle/rows.py`` evaluates the plain definition: the forward of the selected
query rows (their attention over every key they may see) and the backward for an
upstream gradient that is zero outside those rows. Every matrix-multiply operand
is rounded to bfloat16 at the same points as in ``bf16_model``; accumulations and
softmax / LayerNorm statistics stay in float64. With dY zero outside the rows, the
rows that are not selected carry zero dO and dS, so every returned gradient equals
the full model's (pinned against ``bf16_model`` on small inputs). It exists to
measure, at the full sizes where the full model cannot run, how far from the exact
result any bf16-operand implementation lands.
"""
from __future__ import annotations

import math
from typing import Dict

import numpy as np

from .bf16_model import to_bf16
from .layer import LayerParams, act_fwd, act_grad, layer_norm_bwd, layer_norm_fwd


def bf16_rows_fwd_bwd(X: np.ndarray, p: LayerParams, H: int, causal: bool, rows: np.ndarray,
                      dY_rows: np.ndarray, eps: float = 1e-5,
                      round_operands: bool = True) -> Dict[str, np.ndarray]:
    """Returns Y at ``rows`` [B, R, D] and every gradient (dX [B, S, D], weights, biases,
    LayerNorm parameters) for the upstream gradient ``dY_rows`` at ``rows``, zero elsewhere."""
    r = to_bf16 if round_operands else (lambda a: a)
    B, S, D = X.shape
    dh = D // H
    scale = 1.0 / math.sqrt(dh)
    rows = np.asarray(rows)
    R = rows.size
    T = int(rows.max()) + 1 if causal else S          # keys that can matter
    flat = lambda a: a.reshape(-1, a.shape[-1])

    U, xhat1, rstd1 = layer_norm_fwd(X[:, :T], p.ln1_g, p.ln1_b, eps)
    U = r(U)
    Ur = U[:, rows]
    Q, K, V = r(Ur @ p.Wq), r(U @ p.Wk), r(U @ p.Wv)
    O = np.empty((B, R, D))
    lse = np.empty((B, H, R))
    vis = (np.arange(T)[None, :] <= rows[:, None]) if causal else np.ones((R, T), dtype=bool)
    for b in range(B):
        for h in range(H):
            c = slice(h * dh, (h + 1) * dh)
            sc = np.where(vis, Q[b, :, c] @ K[b, :, c].T, -np.inf)
            m = sc.max(axis=1, keepdims=True)
            e = np.exp((sc - m) * scale)
            den = e.sum(axis=1, keepdims=True)
            O[b, :, c] = r((r(e) @ V[b, :, c]) / den)
            lse[b, h] = (m * scale + np.log(den))[:, 0]
    Hd = X[:, rows] + O @ p.Wo
    Vn, xhat2, rstd2 = layer_norm_fwd(Hd, p.ln2_g, p.ln2_b, eps)
    Vn = r(Vn)
    Z = Vn @ p.W1
    if p.b1 is not None:
        Z = Z + p.b1
    G = r(act_fwd(p, Z))
    Y = Hd + G @ p.W2
    if p.b2 is not None:
        Y = Y + p.b2

    dY = dY_rows
    dZ = r((dY @ p.W2.T) * act_grad(p, Z))
    out = dict(Y=Y)
    out["dW2"] = flat(G).T @ flat(dY)
    out["dW1"] = flat(Vn).T @ flat(dZ)
    out["db1"] = dZ.sum(axis=(0, 1)) if p.b1 is not None else None
    out["db2"] = dY.sum(axis=(0, 1)) if p.b2 is not None else None
    dz2, dg2, dbeta2 = layer_norm_bwd(dZ @ p.W1.T, xhat2, rstd2, p.ln2_g)
    dHd = dY + dz2
    dHe = r(dHd)
    dO = r(dHe @ p.Wo.T)
    out["dWo"] = flat(O).T @ flat(dHe)
    dQ = np.empty((B, R, D))
    dK = np.zeros((B, T, D))
    dV = np.zeros((B, T, D))
    for b in range(B):
        for h in range(H):
            c = slice(h * dh, (h + 1) * dh)
            q, k, v, do = Q[b, :, c], K[b, :, c], V[b, :, c], dO[b, :, c]
            sc = np.where(vis, q @ k.T, -np.inf)
            P = np.exp(sc * scale - lse[b, h][:, None])
            delta = (do * O[b, :, c]).sum(axis=1, keepdims=True)
            dS = r(P * (do @ v.T - delta))
            dV[b, :, c] = r(r(P).T @ do)
            dK[b, :, c] = r(scale * (dS.T @ q))
            dQ[b, :, c] = r(scale * (dS @ k))
    out["dWq"] = flat(Ur).T @ flat(dQ)
    out["dWk"] = flat(U).T @ flat(dK)
    out["dWv"] = flat(U).T @ flat(dV)
    dU = dK @ p.Wk.T + dV @ p.Wv.T
    dU[:, rows] += dQ @ p.Wq.T
    dz1, dg1, dbeta1 = layer_norm_bwd(dU, xhat1, rstd1, p.ln1_g)
    dX = np.zeros_like(X)
    dX[:, :T] = dz1
    dX[:, rows] += dHd
    out["dX"] = dX
    out["dln1_g"] = dg1 if p.ln1_g is not None else None
    out["dln1_b"] = dbeta1 if p.ln1_b is not None else None
    out["dln2_g"] = dg2 if p.ln2_g is not None else None
    out["dln2_b"] = dbeta2 if p.ln2_b is not None else None
    return out
