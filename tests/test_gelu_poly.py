"""The bf16 GEMM epilogue evaluates GELU's erf as x Q(x^2) with the
coefficients of paper_2607_21291_amd/csrc/gelu_poly.h. Checked here against
scipy's erf, with the polynomial evaluated in float32 by Horner's rule as the
kernel does: the erf error stays within 2.5e-5 over the real line, which
keeps GELU within 2e-5 of its exact value relative to |x|/2 (a small fraction
of a bf16 ulp)."""
import importlib.util
import math
import os

import numpy as np
from scipy.special import erf

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SCRIPT = os.path.join(ROOT, "paper_2607_21291_amd", "csrc", "erf_poly_fit.py")


def _fit_module():
    spec = importlib.util.spec_from_file_location("erf_poly_fit", SCRIPT)
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_header_polynomial_within_bound():
    F = _fit_module()
    c = F.header_coeffs()[::-1]  # lowest degree first
    assert len(c) == F.DEG + 1
    assert F.max_error(c) < 2.5e-5
    # Q(0) = erf'(0) / sqrt 2 = sqrt(2 / pi)
    assert abs(c[0] - math.sqrt(2.0 / math.pi)) < 1e-4


def test_gelu_from_header_against_exact():
    F = _fit_module()
    c = F.header_coeffs()  # highest degree first, as the kernel's Horner loop
    x = np.linspace(-12.0, 12.0, 240001).astype(np.float32)
    xc = np.clip(x, -np.float32(F.XMAX), np.float32(F.XMAX))
    u = (xc * xc).astype(np.float32)
    q = np.full_like(u, np.float32(c[0]))
    for v in c[1:]:
        q = (q * u + np.float32(v)).astype(np.float32)
    h = (np.float32(0.5) * x).astype(np.float32)
    g = (h * (xc * q) + h).astype(np.float64)
    exact = 0.5 * x.astype(np.float64) * (1.0 + erf(x.astype(np.float64) / math.sqrt(2.0)))
    assert np.all(np.abs(g - exact) <= 2e-5 * 0.5 * np.abs(x.astype(np.float64)) + 1e-30)
