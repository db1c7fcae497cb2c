"""Rounding model of a bf16-operand implementation of the layer — TEST INFRASTRUCTURE.

(See ``oracle/__init__.py``.) The plain definition of ``oracle.layer`` computed in
float64, except that every tensor a bf16 matrix-core implementation must hand to
a matrix multiply as an operand is rounded to bfloat16 (round to nearest even,
from the float32 value an fp32 accumulator would hold) first. Accumulations,
softmax statistics and LayerNorm statistics stay in high precision, as the
hardware's fp32 accumulators do. Inputs (X, the weights, dY) are bf16 already.

The rounding sites, one per matrix-multiply operand of the layer that is not an
input (``SITES``; each name is the tensor as the method forms it):

    forward   U      LN1 output, operand of the Q/K/V projections and of dWq/dWk/dWv
              Q, K, V  projections: operands of the scores, P V and the backward products
              W      the exponentiated scores exp(s - m) of a row before they multiply V.
                     Section 3 accumulates the numerator sum_j exp(s_j - m) V_j and divides
                     by the denominator only at the end, so the operand of the P V product is
                     the un-normalised weight, not the probability
              O      attention output (numerator / denominator), operand of O Wo and dWo
              Vn     LN2 output, operand of the FFN1 product and of dW1
              G      FFN activation output, operand of G W2 and dW2
    backward  dYm    dY through the FFN branch's dropout (identity without dropout)
              dZ     gradient of the FFN pre-activation, operand of dW1 and dZ W1^T
              dHe    gradient entering the output projection, operand of dO = dHe Wo^T, dWo
              dO     gradient of the attention output, operand of dP = dO V^T and dV
              P      probabilities rebuilt from the saved log-sum-exp, operand of dV = P^T dO
              dS     softmax gradient P * (dP - Delta), operand of dQ and dK
              dQ, dK, dV  operands of the weight gradients and of dU

The row statistic Delta = rowsum(dO * O) is formed from the rounded dO and O, the
only dO and O that a bf16 implementation holds; it is not an operand, so it is not
rounded. ``sites`` selects a subset (or extra candidate sites, ``EXTRA_SITES``),
which is how the tests show that the model's result depends on every site it
claims and on no other. With no site it reduces exactly to ``oracle.layer``.

It shares no code with the HIP path. Its only use is to measure how far from the
exact result ANY implementation with bf16 operands lands on a given input, which
sets the parity tolerance for tensors whose exact-result error is dominated by
that rounding (sums over every token of products of rounded operands, such as the
weight gradients).
"""
from __future__ import annotations

import math
from typing import Dict, Iterable, Optional

import numpy as np

from .dropout import dropout_factor
from .layer import LayerParams, act_fwd, act_grad, layer_norm_bwd, layer_norm_fwd

SITES = ("U", "Q", "K", "V", "W", "O", "Vn", "G", "dYm", "dZ", "dHe", "dO", "P", "dS", "dQ", "dK", "dV")
# tensors a bf16 implementation keeps in fp32 (or never forms): rounding one of them
# is a site the model must NOT have
EXTRA_SITES = ("Hd", "Z", "F2", "Pn", "delta", "dP", "dG", "dVn", "dU", "dHd", "lse")


def to_bf16(x: np.ndarray) -> np.ndarray:
    """Round to the nearest bfloat16 (ties to even), returned as float64."""
    f = np.ascontiguousarray(x, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    u = ((u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000).astype(np.uint32)
    return u.view(np.float32).astype(np.float64)


class _Rounder:
    """Rounds a named tensor to bf16 iff its site is on."""

    def __init__(self, sites: Optional[Iterable[str]], round_operands: bool):
        self.on = set(SITES if sites is None else sites) if round_operands else set()
        unknown = self.on - set(SITES) - set(EXTRA_SITES)
        if unknown:
            raise ValueError(f"unknown rounding sites {sorted(unknown)}")

    def __call__(self, name: str, a: np.ndarray) -> np.ndarray:
        return to_bf16(a) if name in self.on else a


def bf16_layer_fwd(X: np.ndarray, p: LayerParams, H: int, causal: bool, eps: float = 1e-5,
                   round_operands: bool = True, sites: Optional[Iterable[str]] = None):
    """Forward of the rounding model. Returns (Y, cache) like ``oracle.layer.layer_fwd``."""
    r = _Rounder(sites, round_operands)
    B, S, D = X.shape
    dh = D // H
    scale = 1.0 / math.sqrt(dh)
    U, xhat1, rstd1 = layer_norm_fwd(X, p.ln1_g, p.ln1_b, eps)
    U = r("U", U)
    Q, K, V = r("Q", U @ p.Wq), r("K", U @ p.Wk), r("V", U @ p.Wv)
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
            w = r("W", e)
            if "Pn" in r.on:            # extra site: the normalised probabilities rounded too
                w = to_bf16(w / den) * den
            O[b, :, c] = r("O", (w @ V[b, :, c]) / den)
            lse[b, h] = r("lse", (m * scale + np.log(den)))[:, 0]
    dm0 = dropout_factor(B * S, D, p.dropout_seed, 0, p.dropout).reshape(B, S, D)
    dm1 = dropout_factor(B * S, D, p.dropout_seed, 1, p.dropout).reshape(B, S, D)
    Hd = r("Hd", X + dm0 * (O @ p.Wo))
    Vn, xhat2, rstd2 = layer_norm_fwd(Hd, p.ln2_g, p.ln2_b, eps)
    Vn = r("Vn", Vn)
    Z = Vn @ p.W1
    if p.b1 is not None:
        Z = Z + p.b1
    Z = r("Z", Z)
    G = r("G", act_fwd(p, Z))
    F2 = G @ p.W2
    if p.b2 is not None:
        F2 = F2 + p.b2
    Y = Hd + dm1 * r("F2", F2)
    cache = dict(X=X, U=U, xhat1=xhat1, rstd1=rstd1, Q=Q, K=K, V=V, O=O, lse=lse, Hd=Hd, Vn=Vn,
                 xhat2=xhat2, rstd2=rstd2, Z=Z, G=G, H=H, causal=causal, dm0=dm0, dm1=dm1, r=r)
    return Y, cache


def bf16_layer_bwd(cache: Dict, p: LayerParams, dY: np.ndarray) -> Dict[str, Optional[np.ndarray]]:
    """Backward of the rounding model for upstream dY (bf16-valued). Returns dX, every
    parameter gradient and the attention-input gradients dQ, dK, dV (as rounded)."""
    r = cache["r"]
    H, causal = cache["H"], cache["causal"]
    X, U, Q, K, V, O, lse = (cache[k] for k in ("X", "U", "Q", "K", "V", "O", "lse"))
    B, S, D = X.shape
    dh = D // H
    scale = 1.0 / math.sqrt(dh)
    flat = lambda a: a.reshape(-1, a.shape[-1])
    mask = np.tri(S, dtype=bool) if causal else np.ones((S, S), dtype=bool)

    dYm = r("dYm", cache["dm1"] * dY)
    dG = r("dG", dYm @ p.W2.T)
    dZ = r("dZ", dG * act_grad(p, cache["Z"]))
    out = {}
    out["dW2"] = flat(cache["G"]).T @ flat(dYm)
    out["dW1"] = flat(cache["Vn"]).T @ flat(dZ)
    out["db1"] = dZ.sum(axis=(0, 1)) if p.b1 is not None else None
    out["db2"] = dYm.sum(axis=(0, 1)) if p.b2 is not None else None
    dz2, out["dln2_g"], out["dln2_b"] = layer_norm_bwd(r("dVn", dZ @ p.W1.T), cache["xhat2"], cache["rstd2"],
                                                       p.ln2_g)
    dHd = r("dHd", dY + dz2)
    dHe = r("dHe", cache["dm0"] * dHd)
    dO = r("dO", dHe @ p.Wo.T)
    out["dWo"] = flat(O).T @ flat(dHe)
    dQ, dK, dV = np.empty_like(Q), np.empty_like(K), np.empty_like(V)
    for b in range(B):
        for h in range(H):
            c = slice(h * dh, (h + 1) * dh)
            q, k, v, do = Q[b, :, c], K[b, :, c], V[b, :, c], dO[b, :, c]
            sc = np.where(mask, q @ k.T, -np.inf)
            P = np.exp(sc * scale - lse[b, h][:, None])
            delta = r("delta", (do * O[b, :, c]).sum(axis=1, keepdims=True))
            dS = r("dS", P * (r("dP", do @ v.T) - delta))
            dV[b, :, c] = r("dV", r("P", P).T @ do)
            dK[b, :, c] = r("dK", scale * (dS.T @ q))
            dQ[b, :, c] = r("dQ", scale * (dS @ k))
    fU = flat(U)
    out["dWq"], out["dWk"], out["dWv"] = fU.T @ flat(dQ), fU.T @ flat(dK), fU.T @ flat(dV)
    dU = r("dU", dQ @ p.Wq.T + dK @ p.Wk.T + dV @ p.Wv.T)
    dz1, out["dln1_g"], out["dln1_b"] = layer_norm_bwd(dU, cache["xhat1"], cache["rstd1"], p.ln1_g)
    out["dX"] = dHd + dz1
    for k in ("ln1_g", "ln1_b", "ln2_g", "ln2_b"):
        if getattr(p, k) is None:
            out["d" + k] = None
    out["dQ"], out["dK"], out["dV"] = dQ, dK, dV
    return out


def bf16_layer_fwd_bwd(X: np.ndarray, p: LayerParams, H: int, causal: bool, dY: np.ndarray,
                       eps: float = 1e-5, round_operands: bool = True,
                       sites: Optional[Iterable[str]] = None) -> Dict[str, np.ndarray]:
    """Forward and backward of the rounding model: Y, O, lse, Hd and every gradient."""
    Y, cache = bf16_layer_fwd(X, p, H, causal, eps, round_operands, sites)
    out = bf16_layer_bwd(cache, p, dY)
    out.update(Y=Y, O=cache["O"], lse=cache["lse"], Hd=cache["Hd"])
    return out
