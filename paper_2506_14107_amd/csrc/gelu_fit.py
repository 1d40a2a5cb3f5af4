"""Fits the polynomial of the bf16 GELU epilogue (gemm.hip, gelu_poly).

Phi(x) - 1/2 = x * P(x^2) on [0, 4], P of degree 8, by least squares on Chebyshev nodes of
[0, 4] against the exact normal CDF (scipy's erf), in the scaled variable (x/4)^2 and then
unscaled, with 4 P(16) = 1/2 imposed (a heavily weighted row) so that the clamped evaluation
beyond |x| = 4 gives GELU(x) = x or 0.  Prints the coefficients c0 .. c8 of P in powers of x^2
and the largest error of the fp32 Horner evaluation over [0, 4].
"""
import numpy as np
from scipy.special import erf

X, DEG, NODES = 4.0, 8, 4000


def fit():
    t = np.cos(np.pi * (np.arange(NODES) + 0.5) / NODES)
    x = (t + 1) / 2 * X
    y = 0.5 * erf(x / np.sqrt(2))
    s = (x / X) ** 2
    A = np.stack([x * s ** k for k in range(DEG + 1)], 1)
    # the constraint 4 P(16) = 1/2, i.e. sum_k 4 * 1^k c_k = 1/2 in the scaled variable
    A = np.vstack([A, 1e4 * X * np.ones(DEG + 1)])
    y = np.append(y, 1e4 * 0.5)
    c, *_ = np.linalg.lstsq(A, y, rcond=None)
    return c / X ** (2 * np.arange(DEG + 1))   # coefficients in powers of x^2


def horner32(c, x):
    """The kernel's operation order in fp32: y = clamp(x, -4, 4), p = P(y^2) by Horner (fused
    multiply-adds), GELU(x) = x (y p + 1/2) with the inner multiply-add fused."""
    x = np.asarray(x, dtype=np.float32)
    y = np.clip(x, np.float32(-X), np.float32(X))
    s = (y * y).astype(np.float32)
    p = np.float32(c[-1])
    for k in range(len(c) - 2, -1, -1):
        p = np.float32(np.float64(p) * np.float64(s) + np.float64(np.float32(c[k])))
    inner = np.float32(np.float64(y) * np.float64(p) + 0.5)
    return (x * inner).astype(np.float32)


if __name__ == "__main__":
    c = fit()
    xs = np.linspace(-X - 1, X + 1, 400001)
    exact = xs * 0.5 * (1 + erf(xs / np.sqrt(2)))
    got = np.array([horner32(c, v) for v in xs[::50]], dtype=np.float64)
    print("max |GELU error| (fp32, kernel order):", np.max(np.abs(got - exact[::50])))
    for k, v in enumerate(c):
        print(f"c{k} = {np.float32(v)!r}")
