"""Constants of the GEMM epilogue's GELU (gelu_erf in gemm.hip).

GELU(x) = x Phi(x) = max(x, 0) - u Phi(-u) with u = |x|, for either sign of
x. The kernel evaluates Phi(-u) = 2^Q(min(u, U)) with U = 6 and Q a degree-7
polynomial in u fitted by least squares to log2 Phi(-u) on Chebyshev nodes
of [0, U] (log Phi(-u) is smooth and close to the parabola -u^2 / 2 there, so
a low degree fits it to a fractional error of a few 1e-6 once exponentiated).
Beyond U, where |GELU(x)| < |x| Phi(-6) < 1e-9 |x|, the clamped value keeps
the error below that bound.

Run: python3 gelu_fit.py  (prints U and the coefficients, highest power first).
"""
import numpy as np
from scipy.special import log_ndtr

DEGREE = 7
U = 6.0
NODES = 4000
LOG2E = 1.4426950408889634


def fit():
    """Coefficients of Q(u), highest power first, and the clamp U."""
    k = np.arange(NODES)
    u = 0.5 * U + 0.5 * U * np.cos((2 * k + 1) * np.pi / (2 * NODES))
    f = log_ndtr(-u) * LOG2E
    p = np.polynomial.chebyshev.Chebyshev.fit(u, f, DEGREE, domain=[0.0, U]).convert(
        kind=np.polynomial.Polynomial).coef
    return list(p[::-1]), U


if __name__ == "__main__":
    coef, clamp = fit()
    print(f"clamp {clamp!r}")
    for c in coef:
        print(repr(float(c)))
