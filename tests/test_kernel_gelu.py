"""The GEMM epilogue's GELU formula, checked on the CPU (no GPU needed).

The FFN's activation is the exact erf GELU, x Phi(x) (Sec. 4.1.2). The HIP
epilogue evaluates Phi(-|x|) = erfc(|x| / sqrt 2) / 2 in the form of Press et
al. (erfc(z) = t exp(-z^2 + P(t)), t = 1 / (1 + z / 2)) with P a degree-5 fit
made by csrc/gelu_fit.py, the change to base 2 and the halving folded into
its coefficients. This test reads the constants out of `gelu_erf` in the
kernel source, checks that they are the fit script's, evaluates the formula
in fp64 and compares it with scipy's erfc: a mistyped or wrongly rescaled
coefficient, or a wrong sign in the final combination, shows up as an error
far above the fit's 8.2e-6. (The kernel's fp32 constants and arithmetic add
rounding of order 1e-6, up to ~1e-5 in the far negative tail |x| > 8 where
the squared exponent is large; the bf16 output resolves 4e-3.)
"""
import importlib.util
import os
import re

import numpy as np
from scipy.special import erfc

CSRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "paper_2607_28940_amd", "csrc")
SRC = os.path.join(CSRC, "gemm.hip")
BOUND = 1e-5


def _constants():
    text = open(SRC).read()
    body = text[text.index("float gelu_erf(float x)"):]
    body = body[:body.index("\n}\n")]
    return [float(v) for v in re.findall(r"(-?\d+\.\d+(?:e-?\d+)?)f", body)]


def _formula(x):
    c = _constants()
    # order in the source: t scale, 1.0, six polynomial coefficients from
    # the highest power down, the scale of the exponent's square
    assert len(c) == 9, c
    t_scale, one, poly, w_scale = c[0], c[1], c[2:8], c[8]
    assert one == 1.0
    u = np.abs(x)
    t = 1.0 / (u * t_scale + one)
    p = np.full_like(x, poly[0])
    for k in poly[1:]:
        p = p * t + k
    w = u * w_scale
    q = t * np.exp2(p - w * w)
    return np.maximum(x, 0.0) - u * q, q


def test_constants_are_the_fit():
    spec = importlib.util.spec_from_file_location("gelu_fit", os.path.join(CSRC, "gelu_fit.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    coef, t_scale, w_scale = mod.fit()
    c = _constants()
    want = [t_scale, 1.0] + list(coef) + [w_scale]
    assert np.allclose(c, want, rtol=1e-12, atol=0), (c, want)


def test_phi_tail_relative_error():
    x = np.linspace(-14.0, 14.0, 400001)
    _, q = _formula(x)
    phi = 0.5 * erfc(np.abs(x) / np.sqrt(2.0))  # Phi(-|x|)
    assert np.max(np.abs(q / phi - 1.0)) < BOUND


def test_gelu_relative_error():
    x = np.concatenate([np.linspace(-14.0, 14.0, 400001), [-1e-30, 1e-30, 0.0]])
    g, _ = _formula(x)
    ref = 0.5 * x * erfc(-x / np.sqrt(2.0))
    nz = ref != 0
    assert np.max(np.abs(g[nz] / ref[nz] - 1.0)) < BOUND
    assert np.all(g[~nz] == 0.0)
