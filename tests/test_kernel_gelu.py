"""The GEMM epilogue's GELU formula, checked on the CPU (no GPU needed).

The FFN's activation is the exact erf GELU, x Phi(x) (Sec. 4.1.2). The HIP
epilogue evaluates Phi(-|x|) = erfc(|x| / sqrt 2) / 2 from the Chebyshev fit
of Press et al. (Numerical Recipes, erfcc) with the change to base 2 and the
halving folded into its coefficients. This test reads the constants out of
`gelu_erf` in the kernel source, evaluates the same formula in fp64 and
compares it with scipy's erfc: a mistyped or wrongly rescaled coefficient, or
a wrong sign in the final combination, shows up as an error far above the
fit's 1.2e-7.
"""
import os
import re

import numpy as np
from scipy.special import erfc

SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "paper_2607_28940_amd", "csrc",
                   "gemm.hip")


def _constants():
    text = open(SRC).read()
    body = text[text.index("float gelu_erf(float x)"):]
    body = body[:body.index("\n}\n")]
    return [float(v) for v in re.findall(r"(-?\d+\.\d+(?:e-?\d+)?)f", body)]


def _formula(x):
    c = _constants()
    # order in the source: t scale, 1.0, ten polynomial coefficients from the
    # highest power down, the scale of the exponent's square
    assert len(c) == 13, c
    t_scale, one, poly, w_scale = c[0], c[1], c[2:12], c[12]
    assert one == 1.0
    u = np.abs(x)
    t = 1.0 / (u * t_scale + one)
    p = np.full_like(x, poly[0])
    for k in poly[1:]:
        p = p * t + k
    w = u * w_scale
    q = t * np.exp2(p - w * w)
    return np.maximum(x, 0.0) - u * q, q


def test_phi_tail_relative_error():
    x = np.linspace(-14.0, 14.0, 400001)
    _, q = _formula(x)
    phi = 0.5 * erfc(np.abs(x) / np.sqrt(2.0))  # Phi(-|x|)
    assert np.max(np.abs(q / phi - 1.0)) < 2e-7


def test_gelu_relative_error():
    x = np.concatenate([np.linspace(-14.0, 14.0, 400001), [-1e-30, 1e-30, 0.0]])
    g, _ = _formula(x)
    ref = 0.5 * x * erfc(-x / np.sqrt(2.0))
    nz = ref != 0
    assert np.max(np.abs(g[nz] / ref[nz] - 1.0)) < 2e-7
    assert np.all(g[~nz] == 0.0)
