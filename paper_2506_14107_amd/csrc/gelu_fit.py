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
    """The kernel's operation order in fp32: m = min(|x|, 4), h = m P(m^2), 0.5 x + |x| h."""
    x = np.asarray(x, dtype=np.float32)
    m = np.minimum(np.abs(x), np.float32(X))
    s = m * m
    p = np.float32(c[-1])
    for k in range(len(c) - 2, -1, -1):
        p = (p * s + np.float32(c[k])).astype(np.float32)
    h = (m * p).astype(np.float32)
    return (np.float32(0.5) * x + np.abs(x) * h).astype(np.float32)


if __name__ == "__main__":
    c = fit()
    xs = np.linspace(0, X, 400001)
    cdf = 0.5 * erf(xs / np.sqrt(2))
    m = xs.astype(np.float32)
    p = np.float32(c[-1])
    for k in range(DEG - 1, -1, -1):
        p = (p * m * m + np.float32(c[k])).astype(np.float32)
    print("max |Phi error| (fp32):", np.max(np.abs(m * p - cdf)))
    for k, v in enumerate(c):
        print(f"c{k} = {np.float32(v)!r}")
