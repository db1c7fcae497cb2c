"""Pins for the LM-head cross-entropy oracle (oracle/xent.py), each independent of
its code: a hand-derived example (tests/golden/xent_closed_form.json), pure-Python
loops with math.exp, the closed form of zero weights, invariance to a vector added
to every vocabulary column and to a permutation of the vocabulary, and central
finite differences of the forward for both gradients."""
import json
import math
import os

import numpy as np

from oracle.xent import xent_bwd, xent_fwd


def test_xent_golden(golden_dir):
    g = json.load(open(os.path.join(golden_dir, "xent_closed_form.json")))
    h, W, y = np.array(g["h"]), np.array(g["W"]), np.array(g["targets"])
    f = xent_fwd(h, W, y, W.shape[1])
    assert abs(f["loss"] - g["loss"]) < 1e-15
    np.testing.assert_allclose(f["lse"], g["lse"], atol=1e-15)
    b = xent_bwd(h, W, y, W.shape[1])
    np.testing.assert_allclose(b["dh"], g["dh"], atol=1e-15)
    np.testing.assert_allclose(b["dW"], g["dW"], atol=1e-15)


def test_xent_brute_force_loops():
    rng = np.random.default_rng(0)
    T, D, V = 3, 2, 4
    h, W = rng.normal(size=(T, D)), rng.normal(size=(D, V + 2))   # two ignored columns
    y = np.array([0, 3, 1])
    tot = 0.0
    for t in range(T):
        z = [sum(h[t, d] * W[d, v] for d in range(D)) for v in range(V)]
        lse = math.log(sum(math.exp(zz) for zz in z))
        tot += lse - z[y[t]]
    assert abs(xent_fwd(h, W, y, V)["loss"] - tot / T) < 1e-14


def test_xent_zero_weights_closed_form():
    rng = np.random.default_rng(1)
    T, D, V = 5, 3, 7
    h, W = rng.normal(size=(T, D)), np.zeros((D, V))
    y = rng.integers(0, V, size=T)
    f = xent_fwd(h, W, y, V)
    assert abs(f["loss"] - math.log(V)) < 1e-14
    b = xent_bwd(h, W, y, V, g=2.0)
    assert np.abs(b["dh"]).max() == 0.0
    onehot = np.zeros((T, V))
    onehot[np.arange(T), y] = 1.0
    np.testing.assert_allclose(b["dW"], h.T @ (1.0 / V - onehot) * (2.0 / T), atol=1e-14)


def test_xent_column_shift_and_permutation_invariance():
    rng = np.random.default_rng(2)
    T, D, V = 6, 4, 9
    h, W = rng.normal(size=(T, D)), rng.normal(size=(D, V))
    y = rng.integers(0, V, size=T)
    u = rng.normal(size=(D, 1))
    a, b = xent_fwd(h, W, y, V), xent_fwd(h, W + u, y, V)
    assert abs(a["loss"] - b["loss"]) < 1e-12
    ga, gb = xent_bwd(h, W, y, V), xent_bwd(h, W + u, y, V)
    np.testing.assert_allclose(ga["dh"], gb["dh"], atol=1e-12)
    np.testing.assert_allclose(ga["dW"], gb["dW"], atol=1e-12)
    perm = rng.permutation(V)
    inv = np.argsort(perm)
    c = xent_fwd(h, W[:, perm], inv[y], V)
    assert abs(a["loss"] - c["loss"]) < 1e-12
    gc = xent_bwd(h, W[:, perm], inv[y], V)
    np.testing.assert_allclose(gc["dW"], ga["dW"][:, perm], atol=1e-12)


def test_xent_finite_differences():
    rng = np.random.default_rng(3)
    T, D, V = 4, 3, 5
    h, W = rng.normal(size=(T, D)), rng.normal(size=(D, V))
    y = rng.integers(0, V, size=T)
    g = 1.7
    b = xent_bwd(h, W, y, V, g=g)
    eps = 1e-6
    for X, dX in ((h, b["dh"]), (W, b["dW"])):
        num = np.zeros_like(X)
        for idx in np.ndindex(*X.shape):
            old = X[idx]
            X[idx] = old + eps
            fp = xent_fwd(h, W, y, V)["loss"]
            X[idx] = old - eps
            fm = xent_fwd(h, W, y, V)["loss"]
            X[idx] = old
            num[idx] = g * (fp - fm) / (2 * eps)
        np.testing.assert_allclose(dX, num, atol=1e-8)


def test_xent_bad_target_is_nan():
    h, W = np.ones((2, 1)), np.ones((1, 3))
    f = xent_fwd(h, W, np.array([0, 3]), 3)
    assert math.isnan(f["loss"]) and math.isfinite(f["token_loss"][0])
    b = xent_bwd(h, W, np.array([0, -1]), 3)
    np.testing.assert_allclose(b["G"][1], np.full(3, 1.0 / 3.0) / 2.0, atol=1e-15)


def test_xent_restricted_forms_match_the_full_definition():
    from oracle.bf16_model import to_bf16
    from oracle.xent import xent_dh_rows, xent_dW_cols, xent_lse_rows
    rng = np.random.default_rng(4)
    T, D, V = 37, 8, 23
    h, W = rng.normal(size=(T, D)), rng.normal(size=(D, V + 9))
    y = rng.integers(0, V, size=T)
    f, b = xent_fwd(h, W, y, V), xent_bwd(h, W, y, V, g=0.3)
    np.testing.assert_allclose(xent_lse_rows(h, W, V, chunk=5), f["lse"], atol=1e-13)
    rows = np.array([0, 5, 36])
    np.testing.assert_allclose(xent_dh_rows(h, W, y, V, rows, T, g=0.3), b["dh"][rows], atol=1e-13)
    cols = np.array([0, 7, V - 1])
    np.testing.assert_allclose(xent_dW_cols(h, W, y, f["lse"], cols, g=0.3), b["dW"][:, cols], atol=1e-13)
    br = xent_bwd(h, W, y, V, g=0.3, round_g=to_bf16)
    np.testing.assert_allclose(xent_dh_rows(h, W, y, V, rows, T, g=0.3, round_g=to_bf16), br["dh"][rows],
                               atol=1e-13)
    np.testing.assert_allclose(xent_dW_cols(h, W, y, f["lse"], cols, g=0.3, round_g=to_bf16),
                               br["dW"][:, cols], atol=1e-13)
