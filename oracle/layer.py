"""Plain float64 definition of one BPT layer, forward and backward.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

The layer (pre-LayerNorm GPT block; the paper builds on the GPT architecture,
Section 4 "Model Configuration"):

    U  = LN1(X)                      LayerNorm over D, biased variance, eps
    Q  = U Wq,  K = U Wk,  V = U Wv  "project input sequence into query, key
                                     and value" (Algorithm 1); W[D_in, D_out]
    O  = concat_h softmax(Q_h K_h^T / sqrt(dh) + mask) V_h     (eq. 1)
    Hd = X + O Wo                    residual 1
    Vn = LN2(Hd)
    Z  = Vn W1 + b1,  G = act(Z)     FFN first linear + activation: eq. 2's
                                     ReLU, or the exact-erf GELU of GPT models
                                     (``LayerParams.activation``)
    Y  = Hd + G W2 + b2              FFN second linear + residual 2

The paper's per-block output (Section 3) is the FFN of (attention + input)
added to (attention + input); read as the pre-LN block above, with the
projection Wo and the two LayerNorms of the GPT block. The causal mask lets
query q see key k iff k <= q within the same sequence; masked scores are -inf.

Everything is unblocked: each (batch, head) materialises its full SxS score and
probability matrices, and the FFN materialises the full SxF intermediate.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, Optional

import numpy as np

from .dropout import dropout_factor
from scipy.special import erf

SQRT2 = math.sqrt(2.0)
INV_SQRT_2PI = 1.0 / math.sqrt(2.0 * math.pi)


@dataclasses.dataclass
class LayerParams:
    """float64 parameters; y = x @ W with W[D_in, D_out]. Optional entries may be None
    (LayerNorm gamma None = 1, beta None = 0, FFN bias None = absent)."""
    Wq: np.ndarray
    Wk: np.ndarray
    Wv: np.ndarray
    Wo: np.ndarray
    W1: np.ndarray
    W2: np.ndarray
    ln1_g: Optional[np.ndarray] = None
    ln1_b: Optional[np.ndarray] = None
    ln2_g: Optional[np.ndarray] = None
    ln2_b: Optional[np.ndarray] = None
    b1: Optional[np.ndarray] = None
    b2: Optional[np.ndarray] = None
    activation: str = "gelu"          # FFN activation: "gelu" or "relu" (eq. 2)
    dropout: float = 0.0              # rate of the two residual-branch dropouts (0: none)
    dropout_seed: int = 0             # 64-bit key of their masks (``oracle/dropout.py``)


PARAM_NAMES = ("ln1_g", "ln1_b", "Wq", "Wk", "Wv", "Wo", "ln2_g", "ln2_b", "W1", "b1", "W2", "b2")


def _f64(t) -> Optional[np.ndarray]:
    if t is None:
        return None
    if isinstance(t, np.ndarray):
        return t.astype(np.float64)
    return t.detach().to("cpu").double().numpy()   # exact for bf16 / fp32 values


def params_from_inputs(inputs: Dict, activation: str = "gelu") -> LayerParams:
    """Build float64 parameters from a dict of tensors (exact upcast)."""
    return LayerParams(**{k: _f64(inputs.get(k)) for k in PARAM_NAMES}, activation=activation)


# --------------------------------------------------------------------------- LayerNorm
def layer_norm_fwd(z: np.ndarray, g: Optional[np.ndarray], b: Optional[np.ndarray], eps: float):
    """LayerNorm over the last axis: gamma * (z - mean) / sqrt(var + eps) + beta.
    Returns (out, xhat, rstd)."""
    mu = z.mean(axis=-1, keepdims=True)
    var = ((z - mu) ** 2).mean(axis=-1, keepdims=True)
    rstd = 1.0 / np.sqrt(var + eps)
    xhat = (z - mu) * rstd
    out = xhat if g is None else xhat * g
    if b is not None:
        out = out + b
    return out, xhat, rstd


def layer_norm_bwd(dout: np.ndarray, xhat: np.ndarray, rstd: np.ndarray, g: Optional[np.ndarray]):
    """Chain rule of ``layer_norm_fwd``. Returns (dz, dgamma, dbeta); dgamma/dbeta are
    summed over every leading axis."""
    gd = dout if g is None else dout * g
    dz = rstd * (gd - gd.mean(axis=-1, keepdims=True)
                 - xhat * (gd * xhat).mean(axis=-1, keepdims=True))
    lead = tuple(range(dout.ndim - 1))
    return dz, (dout * xhat).sum(axis=lead), dout.sum(axis=lead)


# --------------------------------------------------------------------------- GELU
def gelu(z: np.ndarray) -> np.ndarray:
    """Exact GELU: z * Phi(z) with Phi the standard normal CDF."""
    return 0.5 * z * (1.0 + erf(z / SQRT2))


def gelu_grad(z: np.ndarray) -> np.ndarray:
    """d/dz GELU(z) = Phi(z) + z * phi(z)."""
    return 0.5 * (1.0 + erf(z / SQRT2)) + z * INV_SQRT_2PI * np.exp(-0.5 * z * z)


def relu(z: np.ndarray) -> np.ndarray:
    """Eq. (2)'s max(0, z)."""
    return np.maximum(z, 0.0)


def relu_grad(z: np.ndarray) -> np.ndarray:
    """d/dz max(0, z): 1 for z > 0, else 0 (the value 0 taken at z = 0)."""
    return (z > 0).astype(np.float64)


def act_fwd(p: "LayerParams", z: np.ndarray) -> np.ndarray:
    return relu(z) if p.activation == "relu" else gelu(z)


def act_grad(p: "LayerParams", z: np.ndarray) -> np.ndarray:
    return relu_grad(z) if p.activation == "relu" else gelu_grad(z)


# --------------------------------------------------------------------------- attention
def attention_head(Q: np.ndarray, K: np.ndarray, V: np.ndarray, causal: bool):
    """Eq. (1) for one head: softmax(Q K^T / sqrt(dh)) V, softmax row-wise.

    Q, K, V: [S, dh]. Returns (O [S, dh], P [S, S], lse [S]) where
    lse = log sum_k exp(score[q, k]) over the visible keys."""
    S, dh = Q.shape
    sc = (Q @ K.T) / math.sqrt(dh)
    if causal:
        sc = np.where(np.tri(S, K.shape[0], dtype=bool), sc, -np.inf)
    m = sc.max(axis=1, keepdims=True)
    e = np.exp(sc - m)
    den = e.sum(axis=1, keepdims=True)
    P = e / den
    return P @ V, P, (m + np.log(den))[:, 0]


def attention_head_bwd(Q, K, V, P, dO):
    """Chain rule of ``attention_head`` given its probabilities P. Returns dQ, dK, dV."""
    dh = Q.shape[1]
    scale = 1.0 / math.sqrt(dh)
    dV = P.T @ dO
    dP = dO @ V.T
    delta = (P * dP).sum(axis=1, keepdims=True)
    dSc = P * (dP - delta)                 # masked entries have P = 0, so dSc = 0
    return scale * (dSc @ K), scale * (dSc.T @ Q), dV


# --------------------------------------------------------------------------- layer
def layer_fwd(X: np.ndarray, p: LayerParams, H: int, causal: bool, eps: float = 1e-5):
    """Forward of one layer on X[B, S, D] (float64). Returns (Y, cache)."""
    B, S, D = X.shape
    dh = D // H
    U, xhat1, rstd1 = layer_norm_fwd(X, p.ln1_g, p.ln1_b, eps)
    Q, K, V = U @ p.Wq, U @ p.Wk, U @ p.Wv
    O = np.empty_like(X)
    lse = np.empty((B, H, S))
    for b in range(B):
        for h in range(H):
            cols = slice(h * dh, (h + 1) * dh)
            O[b, :, cols], _, lse[b, h] = attention_head(Q[b, :, cols], K[b, :, cols],
                                                         V[b, :, cols], causal)
    # dropout on the two residual branches (factor 1 where the rate is 0)
    dm0 = dropout_factor(B * S, D, p.dropout_seed, 0, p.dropout).reshape(B, S, D)
    dm1 = dropout_factor(B * S, D, p.dropout_seed, 1, p.dropout).reshape(B, S, D)
    Hd = X + dm0 * (O @ p.Wo)
    Vn, xhat2, rstd2 = layer_norm_fwd(Hd, p.ln2_g, p.ln2_b, eps)
    Z = Vn @ p.W1
    if p.b1 is not None:
        Z = Z + p.b1
    G = act_fwd(p, Z)
    F2 = G @ p.W2
    if p.b2 is not None:
        F2 = F2 + p.b2
    Y = Hd + dm1 * F2
    cache = dict(X=X, U=U, xhat1=xhat1, rstd1=rstd1, Q=Q, K=K, V=V, O=O, lse=lse, Hd=Hd,
                 Vn=Vn, xhat2=xhat2, rstd2=rstd2, Z=Z, G=G, H=H, causal=causal, dm0=dm0, dm1=dm1)
    return Y, cache


def layer_bwd(cache: Dict, p: LayerParams, dY: np.ndarray) -> Dict[str, Optional[np.ndarray]]:
    """Backward of ``layer_fwd`` for upstream gradient dY[B, S, D].

    Returns a dict with dX and the gradient of every parameter (None for a
    parameter that is None). Weight gradients are summed over batch and tokens."""
    H, causal = cache["H"], cache["causal"]
    X, U, Q, K, V, O = (cache[k] for k in ("X", "U", "Q", "K", "V", "O"))
    B, S, D = X.shape
    dh = D // H
    flat = lambda a: a.reshape(-1, a.shape[-1])

    # FFN and residual 2 (the FFN branch sees dY through its dropout factor)
    dF2 = cache["dm1"] * dY
    dW2 = flat(cache["G"]).T @ flat(dF2)
    db2 = dF2.sum(axis=(0, 1)) if p.b2 is not None else None
    dG = dF2 @ p.W2.T
    dZ = dG * act_grad(p, cache["Z"])
    db1 = dZ.sum(axis=(0, 1)) if p.b1 is not None else None
    dW1 = flat(cache["Vn"]).T @ flat(dZ)
    dVn = dZ @ p.W1.T
    dz2, dg2, dbeta2 = layer_norm_bwd(dVn, cache["xhat2"], cache["rstd2"], p.ln2_g)
    dHd = dY + dz2

    # output projection (through its dropout factor) and attention
    dA = cache["dm0"] * dHd
    dWo = flat(O).T @ flat(dA)
    dO = dA @ p.Wo.T
    dQ, dK, dV = np.empty_like(Q), np.empty_like(K), np.empty_like(V)
    for b in range(B):
        for h in range(H):
            cols = slice(h * dh, (h + 1) * dh)
            q, k, v = Q[b, :, cols], K[b, :, cols], V[b, :, cols]
            _, P, _ = attention_head(q, k, v, causal)
            dQ[b, :, cols], dK[b, :, cols], dV[b, :, cols] = attention_head_bwd(
                q, k, v, P, dO[b, :, cols])

    # QKV projection and LN1, residual 1
    fU = flat(U)
    dWq, dWk, dWv = fU.T @ flat(dQ), fU.T @ flat(dK), fU.T @ flat(dV)
    dU = dQ @ p.Wq.T + dK @ p.Wk.T + dV @ p.Wv.T
    dz1, dg1, dbeta1 = layer_norm_bwd(dU, cache["xhat1"], cache["rstd1"], p.ln1_g)
    dX = dHd + dz1
    return dict(
        dX=dX, dWq=dWq, dWk=dWk, dWv=dWv, dWo=dWo, dW1=dW1, dW2=dW2, db1=db1, db2=db2,
        dln1_g=dg1 if p.ln1_g is not None else None,
        dln1_b=dbeta1 if p.ln1_b is not None else None,
        dln2_g=dg2 if p.ln2_g is not None else None,
        dln2_b=dbeta2 if p.ln2_b is not None else None,
        # intermediates, for kernel-level comparisons
        dO=dO, dQ=dQ, dK=dK, dV=dV, dHd=dHd,
    )
