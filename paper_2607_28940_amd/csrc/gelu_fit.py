"""Constants of the GEMM epilogue's GELU (gelu_erf in gemm.hip).

GELU(x) = x Phi(x) = max(x, 0) - |x| Phi(-|x|), and with z = |x| / sqrt 2,
Phi(-|x|) = erfc(z) / 2. erfc is written as t exp(-z^2 + P(t)) with
t = 1 / (1 + z / 2) (the form of Press et al., Numerical Recipes, erfcc);
P is fitted here by least squares on Chebyshev nodes of t over z in [0, 10]
(beyond, erfc(z) < 2e-45 is below fp32's range). The kernel evaluates
Phi(-|x|) = t 2^(P'(t) - (c |x|)^2) with P' = log2(e) P - 1 and
c^2 = log2(e) / 2, so this script prints P' and the two scale factors.

Run: python3 gelu_fit.py  (prints the constants in the kernel's order).
"""
import numpy as np
from scipy.special import erfc

DEGREE = 5
Z_MAX = 10.0
NODES = 400
LOG2E = 1.4426950408889634


def fit():
    """Coefficients of P'(t), highest power first, and the scales of t and of
    the exponent's square."""
    lo, hi = 1.0 / (1.0 + Z_MAX / 2.0), 1.0
    k = np.arange(NODES)
    t = 0.5 * (hi + lo) + 0.5 * (hi - lo) * np.cos((2 * k + 1) * np.pi / (2 * NODES))
    z = 2.0 * (1.0 / t - 1.0)
    f = np.log(erfc(z) / t) + z * z
    p = np.polynomial.chebyshev.Chebyshev.fit(t, f, DEGREE, domain=[lo, hi]).convert(
        kind=np.polynomial.Polynomial).coef
    p2 = p * LOG2E
    p2[0] -= 1.0
    return list(p2[::-1]), 1.0 / (2.0 * np.sqrt(2.0)), np.sqrt(LOG2E / 2.0)


if __name__ == "__main__":
    coef, t_scale, w_scale = fit()
    print(f"t scale {float(t_scale)!r}")
    for c in coef:
        print(repr(float(c)))
    print(f"exponent scale {float(w_scale)!r}")
