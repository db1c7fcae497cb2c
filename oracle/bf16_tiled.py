"""A second rounding model: the layer in float32 arithmetic, blockwise — TEST INFRASTRUCTURE.

(See ``oracle/__init__.py``.) ``oracle/bf16_model.py`` rounds the matrix-multiply
operands of the plain definition to bfloat16 but accumulates in float64. A real
bf16-operand implementation also accumulates in float32, in some order of its own.
This model is such an implementation, written plainly on the CPU: the same operand
rounding sites as ``bf16_model.SITES``, float32 everywhere else, and attention as the
blockwise method computes it (Section 3, eq. 3): for each key tile a running
maximum, a running sum and a running numerator, rescaled by exp(m_old - m_new) when
the maximum grows, with the un-normalised weights rounded to bf16 before they
multiply V; the backward visits the same key tiles, rebuilds P from the saved
log-sum-exp and accumulates dQ over the tiles in float32.

Its only use is to measure, on the CPU, how much the error statistics of two valid
bf16-operand implementations differ from each other: the spread of (this model's
error) / (``bf16_model``'s error) over inputs and over the variants below bounds the
factor by which a parity gate may exceed ``bf16_model``'s error
(``tests/expected/derive_model_factors.py``). Variants change only the order and
form of the float32 arithmetic:

    kv_tile   keys per attention tile (the blockwise method's key-value block)
    k_chunk   if set, every product accumulates over its contraction in chunks of this
              length, one after the other, instead of one float32 matmul
    lazy      the running maximum of a row moves only when a tile's maximum exceeds it
              by more than 8 octaves (weights up to 2^8 against a stale maximum)
    base2     scores in base 2: the query is stored times log2(e)/sqrt(dh) (rounded to
              bf16 after the scaling) and the weights are exp2 of the scores
    reverse   key tiles visited from the last one down in the backward

It shares no code with the HIP path.
"""
from __future__ import annotations

import math
from typing import Dict, Optional

import numpy as np
import torch

from .dropout import dropout_factor
from .layer import LayerParams

LOG2E = 1.4426950408889634
LN2 = 0.6931471805599453


def tiled_layer_fwd_bwd(X: np.ndarray, p: LayerParams, H: int, causal: bool, dY: np.ndarray, eps: float = 1e-5,
                        kv_tile: int = 64, k_chunk: Optional[int] = None, lazy: bool = False,
                        base2: bool = False, reverse: bool = False,
                        round_operands: bool = True) -> Dict[str, Optional[np.ndarray]]:
    """Forward and backward; returns Y, O, lse (natural log), Hd, dX, dQ, dK, dV and every
    parameter gradient as float64 arrays. ``round_operands=False`` leaves out the bf16
    rounding (float32 throughout)."""
    # float32 -> nearest bfloat16 (ties to even) -> float32
    _rb = (lambda t: t.to(torch.bfloat16).to(torch.float32)) if round_operands else (lambda t: t)
    f32 = lambda a: None if a is None else torch.from_numpy(np.asarray(a, dtype=np.float32).copy())
    Xt, dYt = f32(X), f32(dY)
    W = {k: f32(getattr(p, k)) for k in ("Wq", "Wk", "Wv", "Wo", "W1", "W2", "ln1_g", "ln1_b", "ln2_g",
                                         "ln2_b", "b1", "b2")}
    B, S, D = X.shape
    dh = D // H
    scale = 1.0 / math.sqrt(dh)
    T = B * S

    def mm(a: torch.Tensor, b: torch.Tensor) -> torch.Tensor:
        if k_chunk is None or a.shape[-1] <= k_chunk:
            return a @ b
        acc = torch.zeros(a.shape[:-1] + (b.shape[-1],), dtype=torch.float32)
        for c0 in range(0, a.shape[-1], k_chunk):
            acc = acc + a[..., c0:c0 + k_chunk] @ b[c0:c0 + k_chunk]
        return acc

    def ln(z, g, b):
        mu = z.mean(-1, keepdim=True)
        var = ((z - mu) ** 2).mean(-1, keepdim=True)
        rs = torch.rsqrt(var + eps)
        xh = (z - mu) * rs
        out = xh if g is None else xh * g
        return (out if b is None else out + b), xh, rs

    def ln_bwd(dout, xh, rs, g):
        gd = dout if g is None else dout * g
        dz = rs * (gd - gd.mean(-1, keepdim=True) - xh * (gd * xh).mean(-1, keepdim=True))
        return dz, (dout * xh).sum(0), dout.sum(0)

    def act(z):
        return torch.relu(z) if p.activation == "relu" else 0.5 * z * (1.0 + torch.erf(z / math.sqrt(2.0)))

    def dact(z):
        if p.activation == "relu":
            return (z > 0).to(torch.float32)
        return 0.5 * (1.0 + torch.erf(z / math.sqrt(2.0))) + z * torch.exp(-0.5 * z * z) / math.sqrt(2 * math.pi)

    x = Xt.reshape(T, D)
    U, xh1, rs1 = ln(x, W["ln1_g"], W["ln1_b"])
    U = _rb(U)
    qs = LOG2E * scale if base2 else 1.0              # factor stored into the query
    Q = _rb(mm(U, W["Wq"]) * qs)
    K, V = _rb(mm(U, W["Wk"])), _rb(mm(U, W["Wv"]))
    ex = torch.exp2 if base2 else torch.exp
    ss = 1.0 if base2 else scale                      # score scale applied after Q K^T
    jump = 8.0 if base2 else 8.0 * math.log(2.0)      # "8 octaves" in score units

    O = torch.empty(T, D)
    lse = torch.empty(B, H, S)                        # in score units (base 2 or e)
    qi = torch.arange(S)[:, None]
    tiles = [(k0, min(k0 + kv_tile, S)) for k0 in range(0, S, kv_tile)]
    for b in range(B):
        for h in range(H):
            rows, cols = slice(b * S, (b + 1) * S), slice(h * dh, (h + 1) * dh)
            q, k, v = Q[rows, cols], K[rows, cols], V[rows, cols]
            m = torch.full((S, 1), -math.inf)
            l = torch.zeros(S, 1)
            acc = torch.zeros(S, dh)
            for k0, k1 in tiles:
                s = mm(q, k[k0:k1].T) * ss
                if causal:
                    s = s.masked_fill(torch.arange(k0, k1)[None, :] > qi, -math.inf)
                tmax = s.max(1, keepdim=True).values
                if lazy:
                    move = (m == -math.inf) | (tmax > m + jump)
                    m_new = torch.where(move, torch.maximum(m, tmax), m)
                else:
                    m_new = torch.maximum(m, tmax)
                corr = torch.where(m_new == -math.inf, torch.zeros_like(m), ex(m - m_new))
                w = torch.where(m_new == -math.inf, torch.zeros_like(s), ex(s - m_new))
                l = l * corr + w.sum(1, keepdim=True)
                acc = acc * corr + mm(_rb(w), v[k0:k1])
                m = m_new
            O[rows, cols] = _rb(acc / l)
            lse[b, h] = (m + torch.log(l) / math.log(2.0 if base2 else math.e))[:, 0]
    dm0 = f32(dropout_factor(T, D, p.dropout_seed, 0, p.dropout))
    dm1 = f32(dropout_factor(T, D, p.dropout_seed, 1, p.dropout))
    Hd = x + dm0 * mm(O, W["Wo"])
    Vn, xh2, rs2 = ln(Hd, W["ln2_g"], W["ln2_b"])
    Vn = _rb(Vn)
    Z = mm(Vn, W["W1"])
    if W["b1"] is not None:
        Z = Z + W["b1"]
    G = _rb(act(Z))
    F2 = mm(G, W["W2"])
    if W["b2"] is not None:
        F2 = F2 + W["b2"]
    Y = Hd + dm1 * F2

    # backward
    dy = dYt.reshape(T, D)
    dYm = _rb(dm1 * dy)
    dZ = _rb(mm(dYm, W["W2"].T) * dact(Z))
    out = {"dW2": mm(G.T, dYm), "dW1": mm(Vn.T, dZ),
           "db1": dZ.sum(0) if W["b1"] is not None else None, "db2": dYm.sum(0) if W["b2"] is not None else None}
    dz2, out["dln2_g"], out["dln2_b"] = ln_bwd(mm(dZ, W["W1"].T), xh2, rs2, W["ln2_g"])
    dHd = dy + dz2
    dHe = _rb(dm0 * dHd)
    dO = _rb(mm(dHe, W["Wo"].T))
    out["dWo"] = mm(O.T, dHe)
    dQ, dK, dV = torch.empty(T, D), torch.empty(T, D), torch.empty(T, D)
    # dK = scale dS^T Q; with a base-2 query Q2 = Q log2(e) scale it is ln(2) dS^T Q2
    kscale = LN2 if base2 else scale
    for b in range(B):
        for h in range(H):
            rows, cols = slice(b * S, (b + 1) * S), slice(h * dh, (h + 1) * dh)
            q, k, v, do, o = Q[rows, cols], K[rows, cols], V[rows, cols], dO[rows, cols], O[rows, cols]
            delta = (do * o).sum(1, keepdim=True)
            ls = lse[b, h][:, None]
            dq = torch.zeros(S, dh)
            for k0, k1 in (reversed(tiles) if reverse else tiles):
                s = mm(q, k[k0:k1].T) * ss
                if causal:
                    s = s.masked_fill(torch.arange(k0, k1)[None, :] > qi, -math.inf)
                P = ex(s - ls)
                dS = _rb(P * (mm(do, v[k0:k1].T) - delta))
                dV[b * S + k0:b * S + k1, cols] = _rb(mm(_rb(P).T, do))
                dK[b * S + k0:b * S + k1, cols] = _rb(kscale * mm(dS.T, q))
                dq = dq + mm(dS, k[k0:k1])
            dQ[rows, cols] = _rb(dq * scale)
    out["dWq"], out["dWk"], out["dWv"] = mm(U.T, dQ), mm(U.T, dK), mm(U.T, dV)
    dU = mm(dQ, W["Wq"].T) + mm(dK, W["Wk"].T) + mm(dV, W["Wv"].T)
    dz1, out["dln1_g"], out["dln1_b"] = ln_bwd(dU, xh1, rs1, W["ln1_g"])
    out["dX"] = dHd + dz1
    for k in ("ln1_g", "ln1_b", "ln2_g", "ln2_b"):
        if W[k] is None:
            out["d" + k] = None
    lse_nat = lse * (LN2 if base2 else 1.0)
    res = {k: (None if v is None else v.double().numpy()) for k, v in out.items()}
    shp = lambda t: t.double().numpy().reshape(B, S, D)
    res.update(Y=shp(Y), dX=shp(out["dX"]), O=shp(O), Hd=shp(Hd), dQ=shp(dQ), dK=shp(dK), dV=shp(dV),
               lse=lse_nat.double().numpy())
    return res
