"""A GPT training step, float64 — TEST INFRASTRUCTURE ONLY.

The experiments of the paper (section 5, Table 1 model shapes, Table 4 throughput)
train decoder-only GPT models built from the layer of ``oracle/layer.py``. The
paper fixes the layer; it does not spell out the rest of the model, so this
oracle takes the usual GPT reading (each choice is listed with the readings of the
paper in the design notes):

    X_0      = Wte[tokens] + Wpe[positions]      token [V, D] and position [S, D] tables;
                                                 a token outside [0, V) gives a NaN row
    X_{l+1}  = layer_l(X_l)                      l = 0 .. L-1, the pre-LN layer of eq. (1)/(2)
    h        = LN_f(X_L)                         final LayerNorm
    loss     = cross-entropy of h Wout            Wout [D, V] (untied), mean over B*S tokens

and the optimiser is AdamW (Adam with decoupled weight decay) with the paper's
weight decay of 0.1 and a learning rate supplied by the caller, who owns the
schedule (the paper decays it on a cosine):

    m  = b1 m + (1 - b1) g,     v = b2 v + (1 - b2) g^2
    p  = p - lr wd p - lr (m / (1 - b1^t)) / (sqrt(v / (1 - b2^t)) + eps)

Everything is the plain definition, unblocked: embedding gather and its
scatter-add, ``oracle.layer.layer_fwd/bwd`` per layer, ``oracle.layer`` LayerNorm,
``oracle.xent`` for the head.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional

import numpy as np

from .layer import LayerParams, layer_bwd, layer_fwd, layer_norm_bwd, layer_norm_fwd
from .xent import xent_bwd, xent_fwd


@dataclasses.dataclass
class GPTParams:
    """float64 parameters of an L-layer GPT; y = x @ W with W[D_in, D_out]."""
    Wte: np.ndarray                       # [V, D]
    Wpe: Optional[np.ndarray]             # [S, D] or None (no position table)
    layers: List[LayerParams]
    lnf_g: Optional[np.ndarray]           # [D]
    lnf_b: Optional[np.ndarray]           # [D]
    Wout: np.ndarray                      # [D, V]


# ------------------------------------------------------------------ embedding
def embed_fwd(tokens: np.ndarray, Wte: np.ndarray, Wpe: Optional[np.ndarray]) -> np.ndarray:
    """X[b, s] = Wte[tokens[b, s]] + Wpe[s]; NaN row for a token outside [0, V)."""
    tokens = np.asarray(tokens, dtype=np.int64)
    V, D = Wte.shape
    ok = (tokens >= 0) & (tokens < V)
    X = Wte[np.clip(tokens, 0, V - 1)].astype(np.float64)
    X[~ok] = np.nan
    if Wpe is not None:
        X = X + Wpe[None, : tokens.shape[1]]
    return X


def embed_bwd(tokens: np.ndarray, dX: np.ndarray, V: int, with_pe: bool):
    """dWte[v] = sum of dX over the tokens equal to v (tokens outside [0, V)
    contribute nothing); dWpe[s] = sum_b dX[b, s]."""
    tokens = np.asarray(tokens, dtype=np.int64)
    B, S, D = dX.shape
    dWte = np.zeros((V, D))
    ok = (tokens >= 0) & (tokens < V)
    np.add.at(dWte, tokens[ok], dX[ok])
    dWpe = dX.sum(axis=0) if with_pe else None
    return dWte, dWpe


# ------------------------------------------------------------------ optimiser
def adamw(p, g, m, v, step: int, lr: float, beta1: float = 0.9, beta2: float = 0.95,
          eps: float = 1e-8, weight_decay: float = 0.1):
    """One AdamW update at 1-based step ``step``; returns new (p, m, v)."""
    p = np.asarray(p, dtype=np.float64)
    g = np.asarray(g, dtype=np.float64)
    m = beta1 * np.asarray(m, dtype=np.float64) + (1.0 - beta1) * g
    v = beta2 * np.asarray(v, dtype=np.float64) + (1.0 - beta2) * g * g
    mhat = m / (1.0 - beta1 ** step)
    vhat = v / (1.0 - beta2 ** step)
    p = p - lr * weight_decay * p - lr * mhat / (np.sqrt(vhat) + eps)
    return p, m, v


# ------------------------------------------------------------------ model
def gpt_fwd_bwd(tokens: np.ndarray, targets: np.ndarray, P: GPTParams, H: int, causal: bool = True,
                eps: float = 1e-5, dloss: float = 1.0, backward: bool = True) -> Dict:
    """Loss of the model on tokens [B, S] with targets [B, S] and, if ``backward``,
    the gradient of dloss * loss for every parameter: keys Wte, Wpe, lnf_g, lnf_b,
    Wout, and ``layers`` (a list of ``oracle.layer.layer_bwd`` dicts)."""
    tokens = np.asarray(tokens)
    B, S = tokens.shape
    V, D = P.Wte.shape
    X = embed_fwd(tokens, P.Wte, P.Wpe)
    caches = []
    for lp in P.layers:
        X, c = layer_fwd(X, lp, H, causal, eps)
        caches.append(c)
    h, xhat, rstd = layer_norm_fwd(X, P.lnf_g, P.lnf_b, eps)
    hf = h.reshape(B * S, D)
    y = np.asarray(targets).reshape(B * S)
    fw = xent_fwd(hf, P.Wout, y, V)
    out = dict(loss=fw["loss"], token_loss=fw["token_loss"].reshape(B, S), X_L=X, h=h)
    if not backward:
        return out
    xb = xent_bwd(hf, P.Wout, y, V, g=dloss)
    dh = xb["dh"].reshape(B, S, D)
    dX, dgf, dbf = layer_norm_bwd(dh, xhat, rstd, P.lnf_g)
    grads_l = [None] * len(P.layers)
    for l in range(len(P.layers) - 1, -1, -1):
        grads_l[l] = layer_bwd(caches[l], P.layers[l], dX)
        dX = grads_l[l]["dX"]
    dWte, dWpe = embed_bwd(tokens, dX, V, P.Wpe is not None)
    out.update(Wte=dWte, Wpe=dWpe, Wout=xb["dW"],
               lnf_g=dgf if P.lnf_g is not None else None,
               lnf_b=dbf if P.lnf_b is not None else None,
               layers=grads_l, dX0=dX)
    return out
