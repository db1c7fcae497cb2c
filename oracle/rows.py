"""The plain layer definition restricted to selected query rows — TEST INFRASTRUCTURE.

(See ``oracle/__init__.py``.) Used to check full-size GPU runs element by element
on a sample of outputs without materialising an SxS matrix over the whole
sequence.

Forward: Y[b, r] for each selected row r needs LN1/Q of that row, K and V of
every key the row may see (all keys; keys 0..r when causal), the attention row
P[r, :], then the output projection and FFN of that row. Nothing is blocked
or reordered: it is ``layer.layer_fwd`` evaluated only where asked.

Backward: if the upstream gradient dY is zero outside the selected rows, the
loss only reaches the parameters and X through those rows, so every gradient
(dX everywhere, every weight gradient) is exactly the full backward's value
for that dY. Keys beyond the last selected row receive no gradient in the
causal case and are skipped.
"""
from __future__ import annotations

import math
from typing import Dict, Optional

import numpy as np

from .layer import LayerParams, act_fwd, act_grad, layer_norm_bwd, layer_norm_fwd


def rows_layer_fwd_bwd(X: np.ndarray, p: LayerParams, H: int, causal: bool,
                       rows: np.ndarray, dY_rows: Optional[np.ndarray] = None,
                       eps: float = 1e-5):
    """X[B, S, D] float64; ``rows``: sorted 1-D positions (the same for every batch entry).

    Returns (Y_rows [B, R, D], grads or None). ``grads`` holds dX [B, S, D] and every
    weight gradient for the upstream gradient that equals ``dY_rows`` at ``rows``
    and zero elsewhere."""
    B, S, D = X.shape
    dh = D // H
    scale = 1.0 / math.sqrt(dh)
    rows = np.asarray(rows)
    R = rows.size
    T = int(rows.max()) + 1 if causal else S          # keys that can matter
    Xk = X[:, :T]
    U, xhat1, rstd1 = layer_norm_fwd(Xk, p.ln1_g, p.ln1_b, eps)
    Ur = U[:, rows]
    Q = Ur @ p.Wq
    K = U @ p.Wk
    V = U @ p.Wv
    O = np.empty((B, R, D))
    Ps = {}
    for b in range(B):
        for h in range(H):
            c = slice(h * dh, (h + 1) * dh)
            sc = scale * (Q[b, :, c] @ K[b, :, c].T)        # [R, T]
            if causal:
                sc = np.where(np.arange(T)[None, :] <= rows[:, None], sc, -np.inf)
            m = sc.max(axis=1, keepdims=True)
            e = np.exp(sc - m)
            P = e / e.sum(axis=1, keepdims=True)
            O[b, :, c] = P @ V[b, :, c]
            if dY_rows is not None:
                Ps[b, h] = P
    Xr = X[:, rows]
    Hd = Xr + O @ p.Wo
    Vn, xhat2, rstd2 = layer_norm_fwd(Hd, p.ln2_g, p.ln2_b, eps)
    Z = Vn @ p.W1
    if p.b1 is not None:
        Z = Z + p.b1
    G = act_fwd(p, Z)
    Y = Hd + G @ p.W2
    if p.b2 is not None:
        Y = Y + p.b2
    if dY_rows is None:
        return Y, None

    dY = dY_rows
    flat = lambda a: a.reshape(-1, a.shape[-1])
    dW2 = flat(G).T @ flat(dY)
    dZ = (dY @ p.W2.T) * act_grad(p, Z)
    dW1 = flat(Vn).T @ flat(dZ)
    dz2, dg2, dbeta2 = layer_norm_bwd(dZ @ p.W1.T, xhat2, rstd2, p.ln2_g)
    dHd = dY + dz2
    dWo = flat(O).T @ flat(dHd)
    dO = dHd @ p.Wo.T
    dQ = np.empty((B, R, D))
    dK = np.zeros((B, T, D))
    dV = np.zeros((B, T, D))
    for b in range(B):
        for h in range(H):
            c = slice(h * dh, (h + 1) * dh)
            P = Ps[b, h]
            do = dO[b, :, c]
            dV[b, :, c] = P.T @ do
            dP = do @ V[b, :, c].T
            dSc = P * (dP - (P * dP).sum(axis=1, keepdims=True))
            dQ[b, :, c] = scale * (dSc @ K[b, :, c])
            dK[b, :, c] = scale * (dSc.T @ Q[b, :, c])
    dWq = flat(Ur).T @ flat(dQ)
    dWk = flat(U).T @ flat(dK)
    dWv = flat(U).T @ flat(dV)
    dU = dK @ p.Wk.T + dV @ p.Wv.T
    dU[:, rows] += dQ @ p.Wq.T
    dz1, dg1, dbeta1 = layer_norm_bwd(dU, xhat1, rstd1, p.ln1_g)
    dX = np.zeros_like(X)
    dX[:, :T] = dz1
    dX[:, rows] += dHd
    grads: Dict[str, Optional[np.ndarray]] = dict(
        dX=dX, dWq=dWq, dWk=dWk, dWv=dWv, dWo=dWo, dW1=dW1, dW2=dW2,
        db1=dZ.sum(axis=(0, 1)) if p.b1 is not None else None,
        db2=dY.sum(axis=(0, 1)) if p.b2 is not None else None,
        dln1_g=dg1 if p.ln1_g is not None else None,
        dln1_b=dbeta1 if p.ln1_b is not None else None,
        dln2_g=dg2 if p.ln2_g is not None else None,
        dln2_b=dbeta2 if p.ln2_b is not None else None,
    )
    return Y, grads
