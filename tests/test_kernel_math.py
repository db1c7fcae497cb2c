"""Host-side checks of closed-form approximations the HIP kernels use (not the oracle).

The GEMM epilogue evaluates GELU(z) = z Phi(z) and GELU'(z) = Phi(z) + z phi(z) in fp32
with erf by Abramowitz & Stegun eq. 7.1.26 (|error| <= 1.5e-7) sharing exp(-z^2/2)
between the two. This re-evaluates the same formula in float32 with numpy and bounds
its error against the exact definition.
"""
import math

import numpy as np
from scipy.special import erf


def gelu_as7126(z):
    f = np.float32
    x = np.abs(z) * f(0.70710678118654752)
    t = f(1) / (f(0.3275911) * x + f(1))
    poly = t * (t * (t * (t * (t * f(1.061405429) + f(-1.453152027)) + f(1.421413741)) + f(-0.284496736))
                + f(0.254829592))
    e = np.exp2(-x * x * f(1.4426950408889634)).astype(np.float32)
    phi_cdf = f(0.5) + f(0.5) * np.copysign(f(1) - poly * e, z)
    return z * phi_cdf, z * f(0.39894228040143268) * e + phi_cdf


def test_gelu_formula_accuracy():
    z = np.linspace(-12, 12, 400001).astype(np.float32)
    g, gp = gelu_as7126(z)
    zd = z.astype(np.float64)
    cdf = 0.5 * (1 + erf(zd / math.sqrt(2)))
    g_ref = zd * cdf
    gp_ref = cdf + zd * np.exp(-zd * zd / 2) / math.sqrt(2 * math.pi)
    assert np.max(np.abs(g - g_ref) / np.maximum(1, np.abs(zd))) < 5e-7
    assert np.max(np.abs(gp - gp_ref)) < 5e-7
    # limits: GELU -> 0 and z, GELU' -> 0 and 1
    assert abs(g[0]) < 1e-6 and abs(g[-1] - 12) < 1e-5
    assert abs(gp[0]) < 1e-6 and abs(gp[-1] - 1) < 1e-6
