"""Rounding model of a bf16 GPT training step — TEST INFRASTRUCTURE.

(See ``oracle/__init__.py``.) ``oracle/gpt.py`` (embedding, L layers, final LayerNorm,
LM-head cross-entropy) with bf16 rounding wherever a bf16 implementation of the step
stores a tensor in bf16 or hands it to a matrix product, and float64 everywhere else:

    X_0 = bf16(Wte[token] + Wpe[position])          the embedding sum, stored in bf16
    X_{l+1} = bf16(layer_l(X_l))                    each layer is ``bf16_model``'s, its
                                                    output stored in bf16
    h = bf16(LN_f(X_L))                             the head's input operand
    G = bf16((dloss / T) (softmax(h W) - onehot))   operand of dh = G W^T and dW = h^T G
    dh = bf16(G W^T)                                stored in bf16
    dX_L = bf16(LN_f^T(dh)),  dX_l = bf16(layer_l^T(dX_{l+1}))

so the parity gate of each gradient of the step can be set, as for one layer, by how
far any bf16-operand implementation lands from the float64 oracle on that input.
It shares no code with the HIP path.
"""
from __future__ import annotations

from typing import Dict

import numpy as np

from .bf16_model import bf16_layer_bwd, bf16_layer_fwd, to_bf16
from .gpt import GPTParams, embed_bwd, embed_fwd
from .layer import layer_norm_bwd, layer_norm_fwd


def bf16_gpt_fwd_bwd(tokens: np.ndarray, targets: np.ndarray, P: GPTParams, H: int, causal: bool = True,
                     eps: float = 1e-5, dloss: float = 1.0, round_operands: bool = True) -> Dict:
    """Loss and every gradient, keyed like ``oracle.gpt.gpt_fwd_bwd``; without rounding
    it is that definition."""
    to_bf16_ = to_bf16 if round_operands else (lambda a: a)
    tokens = np.asarray(tokens)
    B, S = tokens.shape
    V, D = P.Wte.shape
    T = B * S
    X = to_bf16_(embed_fwd(tokens, P.Wte, P.Wpe))
    caches = []
    for lp in P.layers:
        Y, c = bf16_layer_fwd(X, lp, H, causal, eps, round_operands)
        caches.append(c)
        X = to_bf16_(Y)
    h, xhat, rstd = layer_norm_fwd(X, P.lnf_g, P.lnf_b, eps)
    hr = to_bf16_(h).reshape(T, D)
    y = np.asarray(targets).reshape(T)
    z = hr @ P.Wout
    zmax = z.max(axis=1, keepdims=True)
    lse = zmax[:, 0] + np.log(np.exp(z - zmax).sum(axis=1))
    loss = float((lse - z[np.arange(T), y]).mean())
    G = np.exp(z - lse[:, None])
    G[np.arange(T), y] -= 1.0
    G = to_bf16_(G * (dloss / T))
    dh = to_bf16_(G @ P.Wout.T).reshape(B, S, D)
    out = dict(loss=loss, Wout=hr.T @ G)
    dX, dgf, dbf = layer_norm_bwd(dh, xhat, rstd, P.lnf_g)
    dX = to_bf16_(dX)
    grads_l = [None] * len(P.layers)
    for l in range(len(P.layers) - 1, -1, -1):
        grads_l[l] = bf16_layer_bwd(caches[l], P.layers[l], dX)
        dX = to_bf16_(grads_l[l]["dX"])
    dWte, dWpe = embed_bwd(tokens, dX, V, P.Wpe is not None)
    out.update(Wte=dWte, Wpe=dWpe, lnf_g=dgf if P.lnf_g is not None else None,
               lnf_b=dbf if P.lnf_b is not None else None, layers=grads_l, dX0=dX)
    return out
