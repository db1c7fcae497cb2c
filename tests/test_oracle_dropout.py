"""Pins of the oracle's residual-branch dropout (``oracle/dropout.py`` and its use in
``oracle/layer.py``): the generator's published known-answer vectors, a scalar
brute-force layout check, the keep rate, the rate-0 special case and finite
differences of the layer with a fixed mask."""
import json
import os

import numpy as np
import pytest

from oracle.dropout import dropout_factor, keep_mask, philox4x32_10, threshold
from oracle.layer import LayerParams, layer_bwd, layer_fwd

HERE = os.path.dirname(os.path.abspath(__file__))


def test_philox_known_answers():
    kat = json.load(open(os.path.join(HERE, "golden", "philox4x32_10_kat.json")))
    for v in kat["vectors"]:
        c = [int(x, 16) for x in v["counter"]]
        k = [int(x, 16) for x in v["key"]]
        out = philox4x32_10(*[np.array([x]) for x in c], *k)
        assert [int(w[0]) for w in out] == [int(x, 16) for x in v["output"]]


def test_mask_layout_brute_force():
    """Element (t, n) is word n mod 4 of the counter (n div 4, t, site, 0), one scalar
    call per element."""
    T, D, seed, site, p = 3, 10, 0x1234567890ABCDEF, 1, 0.3
    m = keep_mask(T, D, seed, site, p)
    for t in range(T):
        for n in range(D):
            w = philox4x32_10(np.array([n // 4]), np.array([t]), np.array([site]), np.array([0]),
                              seed & 0xFFFFFFFF, seed >> 32)[n % 4][0]
            assert m[t, n] == (int(w) >= int(np.floor(np.float32(p) * 2.0 ** 32)))


def test_keep_rate_and_scale():
    p = 0.1
    m = keep_mask(512, 1024, 7, 0, p)
    n = m.size
    assert abs(m.mean() - (1 - p)) <= 5 * np.sqrt(p * (1 - p) / n)
    f = dropout_factor(4, 8, 7, 0, p)
    assert set(np.unique(f)) <= {0.0, 1.0 / (1.0 - float(np.float32(p)))}
    assert threshold(0.0) == 0 and threshold(0.5) == 2 ** 31
    assert not np.array_equal(keep_mask(64, 64, 7, 0, 0.5), keep_mask(64, 64, 7, 1, 0.5))
    assert not np.array_equal(keep_mask(64, 64, 7, 0, 0.5), keep_mask(64, 64, 8, 0, 0.5))


def _params(seed, D=16, F=32, p=0.0):
    r = np.random.default_rng(seed)
    n = lambda *s: r.normal(0, 0.4, s)
    return LayerParams(Wq=n(D, D), Wk=n(D, D), Wv=n(D, D), Wo=n(D, D), W1=n(D, F), W2=n(F, D),
                       ln1_g=1 + n(D), ln1_b=n(D), ln2_g=1 + n(D), ln2_b=n(D), b1=n(F), b2=n(D),
                       dropout=p, dropout_seed=99)


def test_rate_zero_is_no_dropout():
    X = np.random.default_rng(1).normal(size=(2, 9, 16))
    p0, p1 = _params(2), _params(2)
    p1.dropout_seed = 12345
    Y0, _ = layer_fwd(X, p0, 2, True)
    Y1, _ = layer_fwd(X, p1, 2, True)
    assert np.array_equal(Y0, Y1)


def test_dropped_branches_and_identity():
    """With rate p the output is X + f0 (O Wo) + f1 (FFN), f the factors: at a dropped
    element of both branches the layer passes X through unchanged."""
    X = np.random.default_rng(3).normal(size=(1, 12, 16))
    p = _params(4, p=0.5)
    Y, c = layer_fwd(X, p, 2, True)
    both = (c["dm0"] == 0) & (c["dm1"] == 0)
    assert both.any()
    np.testing.assert_array_equal(Y[both], X[both])


@pytest.mark.parametrize("name", ["Wo", "W1", "W2", "b2", "ln2_g", "Wq"])
def test_finite_differences_with_dropout(name):
    X = np.random.default_rng(5).normal(size=(2, 7, 16))
    p = _params(6, p=0.3)
    dY = np.random.default_rng(8).normal(size=X.shape)
    Y, c = layer_fwd(X, p, 2, True)
    g = layer_bwd(c, p, dY)
    d = np.random.default_rng(9).normal(size=getattr(p, name).shape)
    h = 1e-6
    arr = getattr(p, name)
    arr += h * d
    lp = (layer_fwd(X, p, 2, True)[0] * dY).sum()
    arr -= 2 * h * d
    lm = (layer_fwd(X, p, 2, True)[0] * dY).sum()
    arr += h * d
    fd = (lp - lm) / (2 * h)
    an = float((g["d" + name] * d).sum())
    assert abs(fd - an) <= 1e-6 * max(1.0, abs(fd)), (name, fd, an)
    # and through the input
    dX = np.random.default_rng(10).normal(size=X.shape)
    fd = ((layer_fwd(X + h * dX, p, 2, True)[0] - layer_fwd(X - h * dX, p, 2, True)[0]) * dY).sum() / (2 * h)
    assert abs(fd - float((g["dX"] * dX).sum())) <= 1e-6 * max(1.0, abs(fd))
