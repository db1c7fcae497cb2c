"""Pins of the bf16 rounding model's rounding sites (``oracle/bf16_model.py``).

The model sets the floor of every bf16 parity gate, so where it rounds matters: an
extra rounding site loosens every gate that uses it, a missing one tightens them. Here
a scalar emulation, written with Python loops and ``math`` only and sharing no code with
the model, computes the layer (forward and backward) on tiny shapes with bf16 rounding
at exactly the matrix-multiply operands of the method (precision reading R12: every
operand of a matrix product that is not an input is rounded to bf16 from its fp32
value; accumulations, softmax and LayerNorm statistics stay exact):

    forward   LN1 out U; projections Q, K, V; the exponentiated scores exp(s - m)
              before they multiply V (Section 3's numerator, divided by the
              denominator at the end); the attention output O; LN2 out; GELU out
    backward  dY through the FFN dropout; dZ; the gradient into the output
              projection; dO; the probabilities rebuilt from the log-sum-exp (operand
              of dV); dS; dQ, dK, dV

The model must equal the emulation, and removing any one of its sites, or adding any
one candidate site that an fp32-accumulating implementation does not round, must make
it differ: so the comparison would catch a model with a site too many or too few.
"""
import math
import struct

import numpy as np
import pytest

import oracle
from oracle.bf16_model import EXTRA_SITES, SITES, bf16_layer_fwd_bwd
from oracle.dropout import dropout_factor

EPS = 1e-5


def bf(x: float) -> float:
    """x rounded to float32, then to the nearest bfloat16 (ties to even)."""
    u = struct.unpack("<I", struct.pack("<f", x))[0]
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return struct.unpack("<f", struct.pack("<I", u))[0]


def emulate(X, W, H, causal, dY, dm0, dm1):
    """The layer with bf16 rounding at the operand sites listed above, scalar loops.
    X, dY: [B][S][D] lists; W: dict of lists (biases / LayerNorm parameters present);
    dm0, dm1: the two residual branches' dropout factors [B][S][D]."""
    B, S, D = len(X), len(X[0]), len(X[0][0])
    F = len(W["b1"])
    dh = D // H
    sc = 1.0 / math.sqrt(dh)
    rng = range

    def ln(z, g, b):
        mu = sum(z) / len(z)
        var = sum((v - mu) ** 2 for v in z) / len(z)
        rs = 1.0 / math.sqrt(var + EPS)
        xh = [(v - mu) * rs for v in z]
        return [g[i] * xh[i] + b[i] for i in rng(len(z))], xh, rs

    def ln_bwd(dout, xh, rs, g):
        n = len(dout)
        gd = [dout[i] * g[i] for i in rng(n)]
        m1 = sum(gd) / n
        m2 = sum(gd[i] * xh[i] for i in rng(n)) / n
        return [rs * (gd[i] - m1 - xh[i] * m2) for i in rng(n)]

    def mm(a, w):          # [n][k] @ [k][m]
        return [[sum(a[i][k] * w[k][j] for k in rng(len(w))) for j in rng(len(w[0]))] for i in rng(len(a))]

    def mmT(a, w):         # [n][m] @ [k][m]^T
        return [[sum(a[i][j] * w[k][j] for j in rng(len(w[0]))) for k in rng(len(w))] for i in rng(len(a))]

    def gelu(z):
        return 0.5 * z * (1.0 + math.erf(z / math.sqrt(2.0)))

    def dgelu(z):
        return 0.5 * (1.0 + math.erf(z / math.sqrt(2.0))) + z * math.exp(-0.5 * z * z) / math.sqrt(2.0 * math.pi)

    vis = lambda q, k: (k <= q) if causal else True
    out = {k: [[0.0] * len(W[k][0]) for _ in W[k]] for k in ("Wq", "Wk", "Wv", "Wo", "W1", "W2")}
    for k in ("ln1_g", "ln1_b", "ln2_g", "ln2_b"):
        out[k] = [0.0] * D
    out["b1"], out["b2"] = [0.0] * F, [0.0] * D
    Y, dX, O_all, lse_all, dQ_all, dK_all, dV_all = [], [], [], [], [], [], []
    for b in rng(B):
        x = X[b]
        l1 = [ln(x[s], W["ln1_g"], W["ln1_b"]) for s in rng(S)]
        U = [[bf(v) for v in l1[s][0]] for s in rng(S)]
        Q = [[bf(v) for v in row] for row in mm(U, W["Wq"])]
        K = [[bf(v) for v in row] for row in mm(U, W["Wk"])]
        V = [[bf(v) for v in row] for row in mm(U, W["Wv"])]
        O = [[0.0] * D for _ in rng(S)]
        lse = [[0.0] * S for _ in rng(H)]
        for h in rng(H):
            cs = range(h * dh, (h + 1) * dh)
            for q in rng(S):
                ks = [k for k in rng(S) if vis(q, k)]
                t = {k: sum(Q[q][j] * K[k][j] for j in cs) for k in ks}
                m = max(t.values())
                e = {k: math.exp((t[k] - m) * sc) for k in ks}
                den = sum(e.values())
                for j in cs:
                    O[q][j] = bf(sum(bf(e[k]) * V[k][j] for k in ks) / den)
                lse[h][q] = m * sc + math.log(den)
        ow = mm(O, W["Wo"])
        Hd = [[x[s][i] + dm0[b][s][i] * ow[s][i] for i in rng(D)] for s in rng(S)]
        l2 = [ln(Hd[s], W["ln2_g"], W["ln2_b"]) for s in rng(S)]
        Vn = [[bf(v) for v in l2[s][0]] for s in rng(S)]
        Z = [[v + W["b1"][f] for f, v in enumerate(row)] for row in mm(Vn, W["W1"])]
        G = [[bf(gelu(v)) for v in row] for row in Z]
        f2 = mm(G, W["W2"])
        Y.append([[Hd[s][i] + dm1[b][s][i] * (f2[s][i] + W["b2"][i]) for i in rng(D)] for s in rng(S)])
        # backward
        dYm = [[bf(dm1[b][s][i] * dY[b][s][i]) for i in rng(D)] for s in rng(S)]
        dG = mmT(dYm, W["W2"])
        dZ = [[bf(dG[s][f] * dgelu(Z[s][f])) for f in rng(F)] for s in rng(S)]
        for f in rng(F):
            for i in rng(D):
                out["W2"][f][i] += sum(G[s][f] * dYm[s][i] for s in rng(S))
            out["b1"][f] += sum(dZ[s][f] for s in rng(S))
        for i in rng(D):
            for f in rng(F):
                out["W1"][i][f] += sum(Vn[s][i] * dZ[s][f] for s in rng(S))
            out["b2"][i] += sum(dYm[s][i] for s in rng(S))
        dVn = mmT(dZ, W["W1"])
        dHd = []
        for s in rng(S):
            for i in rng(D):
                out["ln2_g"][i] += dVn[s][i] * l2[s][1][i]
                out["ln2_b"][i] += dVn[s][i]
            dz = ln_bwd(dVn[s], l2[s][1], l2[s][2], W["ln2_g"])
            dHd.append([dY[b][s][i] + dz[i] for i in rng(D)])
        dHe = [[bf(dm0[b][s][i] * dHd[s][i]) for i in rng(D)] for s in rng(S)]
        dO = [[bf(v) for v in row] for row in mmT(dHe, W["Wo"])]
        for i in rng(D):
            for j in rng(D):
                out["Wo"][i][j] += sum(O[s][i] * dHe[s][j] for s in rng(S))
        dQ = [[0.0] * D for _ in rng(S)]
        dK = [[0.0] * D for _ in rng(S)]
        dV = [[0.0] * D for _ in rng(S)]
        for h in rng(H):
            cs = range(h * dh, (h + 1) * dh)
            P = [[math.exp(sc * sum(Q[q][j] * K[k][j] for j in cs) - lse[h][q]) if vis(q, k) else 0.0
                  for k in rng(S)] for q in rng(S)]
            delta = [sum(dO[q][j] * O[q][j] for j in cs) for q in rng(S)]
            dS = [[bf(P[q][k] * (sum(dO[q][j] * V[k][j] for j in cs) - delta[q])) if vis(q, k) else 0.0
                   for k in rng(S)] for q in rng(S)]
            for k in rng(S):
                for j in cs:
                    dV[k][j] = bf(sum(bf(P[q][k]) * dO[q][j] for q in rng(S)))
                    dK[k][j] = bf(sc * sum(dS[q][k] * Q[q][j] for q in rng(S)))
            for q in rng(S):
                for j in cs:
                    dQ[q][j] = bf(sc * sum(dS[q][k] * K[k][j] for k in rng(S)))
        for name, dt in (("Wq", dQ), ("Wk", dK), ("Wv", dV)):
            for i in rng(D):
                for j in rng(D):
                    out[name][i][j] += sum(U[s][i] * dt[s][j] for s in rng(S))
        dU = [[sum(dQ[s][j] * W["Wq"][i][j] + dK[s][j] * W["Wk"][i][j] + dV[s][j] * W["Wv"][i][j]
                   for j in rng(D)) for i in rng(D)] for s in rng(S)]
        dxb = []
        for s in rng(S):
            for i in rng(D):
                out["ln1_g"][i] += dU[s][i] * l1[s][1][i]
                out["ln1_b"][i] += dU[s][i]
            dz = ln_bwd(dU[s], l1[s][1], l1[s][2], W["ln1_g"])
            dxb.append([dHd[s][i] + dz[i] for i in rng(D)])
        dX.append(dxb)
        O_all.append(O)
        lse_all.append(lse)
        dQ_all.append(dQ)
        dK_all.append(dK)
        dV_all.append(dV)
    res = {"Y": Y, "dX": dX, "O": O_all, "lse": lse_all, "dQ": dQ_all, "dK": dK_all, "dV": dV_all}
    for k in ("Wq", "Wk", "Wv", "Wo", "W1", "W2", "b1", "b2"):
        res["d" + k] = out[k]
    for k in ("ln1_g", "ln1_b", "ln2_g", "ln2_b"):
        res["d" + k] = out[k]
    return {k: np.array(v, dtype=np.float64) for k, v in res.items()}


COMPARED = ("Y", "dX", "O", "lse", "dQ", "dK", "dV", "dWq", "dWk", "dWv", "dWo", "dW1", "dW2", "db1", "db2",
            "dln1_g", "dln1_b", "dln2_g", "dln2_b")


def _case(seed, causal, dropout):
    from oracle.bf16_model import to_bf16
    rng = np.random.default_rng(seed)
    B, S, D, H, F = 2, 5, 4, 2, 8
    bfv = lambda *shape, s=1.0: to_bf16(rng.normal(size=shape) * s)
    W = {"Wq": bfv(D, D, s=0.7), "Wk": bfv(D, D, s=0.7), "Wv": bfv(D, D, s=0.5), "Wo": bfv(D, D, s=0.5),
         "W1": bfv(D, F, s=0.5), "W2": bfv(F, D, s=0.4), "ln1_g": 1 + 0.1 * rng.normal(size=D),
         "ln1_b": 0.1 * rng.normal(size=D), "ln2_g": 1 + 0.1 * rng.normal(size=D), "ln2_b": 0.1 * rng.normal(size=D),
         "b1": 0.1 * rng.normal(size=F), "b2": 0.1 * rng.normal(size=D)}
    X, dY = bfv(B, S, D), bfv(B, S, D)
    p = oracle.LayerParams(**W)
    seed64 = 0x0123456789ABCDEF
    if dropout:
        p.dropout, p.dropout_seed = 0.3, seed64
    dm0 = dropout_factor(B * S, D, seed64, 0, p.dropout).reshape(B, S, D)
    dm1 = dropout_factor(B * S, D, seed64, 1, p.dropout).reshape(B, S, D)
    return X, dY, W, p, H, dm0, dm1


def _max_rel_dev(a, b):
    """Largest deviation over the compared tensors, each relative to the emulation's scale."""
    worst, where = 0.0, None
    for k in COMPARED:
        scale = max(float(np.abs(b[k]).max()), 1e-30)
        d = float(np.abs(np.asarray(a[k]) - b[k]).max()) / scale
        if d > worst:
            worst, where = d, k
    return worst, where


@pytest.mark.parametrize("causal,dropout,seed", [(True, False, 31), (False, False, 32), (True, True, 33)])
def test_model_equals_scalar_emulation(causal, dropout, seed):
    X, dY, W, p, H, dm0, dm1 = _case(seed, causal, dropout)
    em = emulate(X.tolist(), {k: v.tolist() for k, v in W.items()}, H, causal, dY.tolist(), dm0.tolist(),
                 dm1.tolist())
    m = bf16_layer_fwd_bwd(X, p, H, causal, dY, EPS)
    dev, where = _max_rel_dev(m, em)
    assert dev < 1e-12, (dev, where)


# sites whose rounding changes nothing without dropout (dY is bf16 already)
_NEEDS_DROPOUT = {"dYm"}


@pytest.mark.parametrize("site", SITES)
def test_removing_a_site_changes_the_result(site):
    dropout = site in _NEEDS_DROPOUT
    X, dY, W, p, H, dm0, dm1 = _case(34, True, dropout)
    em = emulate(X.tolist(), {k: v.tolist() for k, v in W.items()}, H, True, dY.tolist(), dm0.tolist(),
                 dm1.tolist())
    m = bf16_layer_fwd_bwd(X, p, H, True, dY, EPS, sites=[s for s in SITES if s != site])
    dev, where = _max_rel_dev(m, em)
    assert dev > 1e-6, f"model without site {site} still matches the emulation ({dev:.2e})"


@pytest.mark.parametrize("site", EXTRA_SITES)
def test_adding_a_site_changes_the_result(site):
    X, dY, W, p, H, dm0, dm1 = _case(35, True, False)
    em = emulate(X.tolist(), {k: v.tolist() for k, v in W.items()}, H, True, dY.tolist(), dm0.tolist(),
                 dm1.tolist())
    m = bf16_layer_fwd_bwd(X, p, H, True, dY, EPS, sites=list(SITES) + [site])
    dev, where = _max_rel_dev(m, em)
    assert dev > 1e-6, f"model with the extra site {site} still matches the emulation ({dev:.2e})"
