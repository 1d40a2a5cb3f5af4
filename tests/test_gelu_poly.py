"""The bf16 GEMM epilogue's GELU polynomial (gemm.hip, gelu_poly) against the exact GELU.

The coefficients are read from the kernel source and evaluated in float32 in the kernel's
operation order; the exact value is x * Phi(x) with Phi from the error function in float64.
Bounds: |error| <= 1.1e-5 for |x| <= 3 and <= 1.3e-4 everywhere (largest near |x| = 4, where
the fit is pinned to Phi = 1), far below the bf16 step the result is rounded to.
"""
import os
import re

import numpy as np
from scipy.special import erf

SRC = os.path.join(os.path.dirname(__file__), "..", "paper_2506_14107_amd", "csrc", "gemm.hip")


def _coefficients():
    src = open(SRC).read()
    body = src[src.index("float gelu_poly(float x)"):]
    body = body[:body.index("\n}\n")]
    lits = re.findall(r"([-+]?\d\.\d+e[-+]\d+)f", body)
    return [np.float32(v) for v in lits]   # highest degree first, as Horner consumes them


def _gelu_poly(x, coef):
    """The kernel's operation order in float32: y = clamp(x, -4, 4), p = P(y^2) by Horner,
    x * (y p + 1/2) (the last step one fused multiply-add, rounded once)."""
    x = np.asarray(x, dtype=np.float32)
    y = np.clip(x, np.float32(-4.0), np.float32(4.0))
    s = (y * y).astype(np.float32)
    p = np.full_like(x, coef[0])
    for c in coef[1:]:
        p = (p.astype(np.float64) * s + c).astype(np.float32)   # fused: one rounding
    u = (y.astype(np.float64) * p + 0.5).astype(np.float32)
    return (x * u).astype(np.float32)


def test_gelu_poly_error_bounds():
    coef = _coefficients()
    assert len(coef) == 9
    x = np.linspace(-12.0, 12.0, 480001)
    exact = x * 0.5 * (1.0 + erf(x / np.sqrt(2.0)))
    err = np.abs(_gelu_poly(x, coef).astype(np.float64) - exact)
    assert err[np.abs(x) <= 3.0].max() <= 1.1e-5
    assert err.max() <= 1.3e-4


def test_gelu_poly_special_values():
    coef = _coefficients()
    v = _gelu_poly(np.array([0.0, 1.0, -1.0, 8.0, -8.0], dtype=np.float32), coef)
    assert v[0] == 0.0
    assert abs(v[1] - 0.8413447460685429) < 1e-5 and abs(v[2] + 0.15865525393145707) < 1e-5
    assert abs(v[3] - 8.0) < 1e-5 and abs(v[4]) < 1e-5   # past |x| = 4: x and 0
