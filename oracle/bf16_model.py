"""Rounding model of a bf16-operand implementation of the layer — TEST INFRASTRUCTURE.

(See ``oracle/__init__.py``.) The plain definition of ``oracle.layer`` computed in
float64, except that every tensor a bf16 matrix-core implementation must hand to
a matrix multiply as an operand is rounded to bfloat16 (round to nearest even)
first: the LayerNorm outputs, Q, K, V, the exp-weights before they multiply V,
the attention output, the FFN activation output, and in the backward dO, dS, dZ, the
upstream gradient into the output projection and the Q/K/V gradients.
Accumulations, softmax statistics and LayerNorm statistics stay in high
precision, as the hardware's fp32 accumulators do.

It shares no code with the HIP path. Its only use is to measure how far from
the exact result ANY implementation with bf16 operands lands on a given input,
which sets the parity tolerance for tensors whose exact-result error is
dominated by that rounding (sums over every token of products of rounded
operands, such as the weight gradients). With ``round_operands=False`` it
reduces exactly to ``oracle.layer`` (pinned by the tests).
"""
from __future__ import annotations

import math
from typing import Dict

import numpy as np

from .layer import LayerParams, act_fwd, act_grad, layer_norm_bwd, layer_norm_fwd


def to_bf16(x: np.ndarray) -> np.ndarray:
    """Round to the nearest bfloat16 (ties to even), returned as float64."""
    f = np.ascontiguousarray(x, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    u = ((u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000).astype(np.uint32)
    return u.view(np.float32).astype(np.float64)


def bf16_layer_fwd_bwd(X: np.ndarray, p: LayerParams, H: int, causal: bool, dY: np.ndarray,
                       eps: float = 1e-5, round_operands: bool = True) -> Dict[str, np.ndarray]:
    r = to_bf16 if round_operands else (lambda a: a)
    B, S, D = X.shape
    dh = D // H
    scale = 1.0 / math.sqrt(dh)
    flat = lambda a: a.reshape(-1, a.shape[-1])

    U, xhat1, rstd1 = layer_norm_fwd(X, p.ln1_g, p.ln1_b, eps)
    U = r(U)
    Q, K, V = r(U @ p.Wq), r(U @ p.Wk), r(U @ p.Wv)
    O = np.empty_like(X)
    lse = np.empty((B, H, S))
    mask = np.tri(S, dtype=bool) if causal else np.ones((S, S), dtype=bool)
    for b in range(B):
        for h in range(H):
            c = slice(h * dh, (h + 1) * dh)
            sc = np.where(mask, Q[b, :, c] @ K[b, :, c].T, -np.inf)
            m = sc.max(axis=1, keepdims=True)
            e = np.exp((sc - m) * scale)
            den = e.sum(axis=1, keepdims=True)
            O[b, :, c] = r((r(e) @ V[b, :, c]) / den)
            lse[b, h] = (m * scale + np.log(den))[:, 0]
    Hd = X + O @ p.Wo
    Vn, xhat2, rstd2 = layer_norm_fwd(Hd, p.ln2_g, p.ln2_b, eps)
    Vn = r(Vn)
    Z = Vn @ p.W1
    if p.b1 is not None:
        Z = Z + p.b1
    G = r(act_fwd(p, Z))
    Y = Hd + G @ p.W2
    if p.b2 is not None:
        Y = Y + p.b2

    dZ = r((dY @ p.W2.T) * act_grad(p, Z))
    out = dict(Y=Y, O=O, lse=lse, Hd=Hd)
    out["dW2"] = flat(G).T @ flat(dY)
    out["dW1"] = flat(Vn).T @ flat(dZ)
    out["db1"] = dZ.sum(axis=(0, 1)) if p.b1 is not None else None
    out["db2"] = dY.sum(axis=(0, 1)) if p.b2 is not None else None
    dz2, out["dln2_g"], out["dln2_b"] = layer_norm_bwd(dZ @ p.W1.T, xhat2, rstd2, p.ln2_g)
    dHd = dY + dz2
    dHe = r(dHd)
    dO = r(dHe @ p.Wo.T)
    out["dWo"] = flat(O).T @ flat(dHe)
    dQ, dK, dV = np.empty_like(Q), np.empty_like(K), np.empty_like(V)
    for b in range(B):
        for h in range(H):
            c = slice(h * dh, (h + 1) * dh)
            q, k, v, do = Q[b, :, c], K[b, :, c], V[b, :, c], dO[b, :, c]
            sc = np.where(mask, q @ k.T, -np.inf)
            P = np.exp(sc * scale - lse[b, h][:, None])
            delta = (do * O[b, :, c]).sum(axis=1, keepdims=True)
            dS = r(P * (do @ v.T - delta))
            dV[b, :, c] = r(r(P).T @ do)
            dK[b, :, c] = r(scale * (dS.T @ q))
            dQ[b, :, c] = r(scale * (dS @ k))
    fU = flat(U)
    out["dWq"], out["dWk"], out["dWv"] = fU.T @ flat(dQ), fU.T @ flat(dK), fU.T @ flat(dV)
    dU = dQ @ p.Wq.T + dK @ p.Wk.T + dV @ p.Wv.T
    dz1, out["dln1_g"], out["dln1_b"] = layer_norm_bwd(dU, xhat1, rstd1, p.ln1_g)
    out["dX"] = dHd + dz1
    if p.ln1_g is None:
        out["dln1_g"] = None
    if p.ln1_b is None:
        out["dln1_b"] = None
    if p.ln2_g is None:
        out["dln2_g"] = None
    if p.ln2_b is None:
        out["dln2_b"] = None
    return out
