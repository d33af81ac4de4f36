"""The GEMM epilogue's GELU formula, checked on the CPU (no GPU needed).

The FFN's activation is the exact erf GELU, x Phi(x) (Sec. 4.1.2). The HIP
epilogue evaluates it as max(x, 0) - |x| Phi(-|x|) with Phi(-u) = 2^Q(min(u, 6))
and Q a degree-7 polynomial fitted to log2 Phi(-u) by csrc/gelu_fit.py. This
test reads the constants out of `gelu_erf` in the kernel source, checks that
they are the fit script's, evaluates the formula with the kernel's fp32
arithmetic (Horner steps rounded to fp32) and compares it with scipy's erfc:
a mistyped coefficient, a wrong clamp or a wrong sign in the final
combination shows up as an error far above the fit's 5.5e-6. Beyond the
clamp |GELU(x)| < |x| Phi(-6) < 1e-9 |x|, and that is the bound there (the
bf16 output resolves 4e-3 of a value).
"""
import importlib.util
import os
import re

import numpy as np
from scipy.special import erfc

CSRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "paper_2607_28940_amd", "csrc")
SRC = os.path.join(CSRC, "gemm.hip")
BOUND = 1e-5       # fractional error, |x| <= 6
TAIL_BOUND = 1e-9  # absolute error over |x|, |x| > 6


def _constants():
    text = open(SRC).read()
    body = text[text.index("float gelu_erf(float x)"):]
    body = body[:body.index("\n}\n")]
    return [float(v) for v in re.findall(r"(-?\d+\.\d+(?:e-?\d+)?)f", body)]


def _formula(x):
    c = _constants()
    # order in the source: the clamp, eight coefficients from the highest
    # power down
    assert len(c) == 9, c
    clamp, poly = np.float32(c[0]), [np.float32(v) for v in c[1:]]
    xf = x.astype(np.float32)
    u = np.minimum(np.abs(xf), clamp)
    q = np.full_like(u, poly[0])
    for k in poly[1:]:
        q = (q * u + k).astype(np.float32)
    phi = np.exp2(q.astype(np.float64))
    return np.maximum(x, 0.0) - np.abs(x) * phi, phi


def test_constants_are_the_fit():
    spec = importlib.util.spec_from_file_location("gelu_fit", os.path.join(CSRC, "gelu_fit.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    coef, clamp = mod.fit()
    c = _constants()
    want = [clamp] + list(coef)
    assert np.allclose(c, want, rtol=1e-12, atol=0), (c, want)


def test_phi_relative_error():
    x = np.linspace(-6.0, 6.0, 400001)
    _, q = _formula(x)
    phi = 0.5 * erfc(np.abs(x) / np.sqrt(2.0))  # Phi(-|x|)
    assert np.max(np.abs(q / phi - 1.0)) < BOUND


def test_gelu_error():
    x = np.concatenate([np.linspace(-14.0, 14.0, 400001), [-1e-30, 1e-30, 0.0, -1e4, 1e4]])
    g, _ = _formula(x)
    ref = 0.5 * x * erfc(-x / np.sqrt(2.0))
    inner = np.abs(x) <= 6.0
    nz = inner & (ref != 0)
    assert np.max(np.abs(g[nz] / ref[nz] - 1.0)) < BOUND
    assert np.all(g[inner & (ref == 0)] == 0.0)
    out = ~inner
    assert np.max(np.abs(g[out] - ref[out]) / np.abs(x[out])) < TAIL_BOUND
