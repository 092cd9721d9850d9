"""The GEMM epilogue's GELU approximation (csrc/device_common.h) on the CPU.

The kernels evaluate the exact-erf GELU z * Phi(z) as
max(z, 0) - |z| * 2^P(min(|z|, 6)), P a degree-7 polynomial fit to
log2 Phi(-u).  These tests read the coefficients out of the header, check them
against a fresh fit (csrc/gelu_fit.py), and bound the error of the fp32
evaluation against the exact GELU (scipy's normal CDF in fp64).
"""
import os
import re
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2506_12035_amd", "csrc")
sys.path.insert(0, CSRC)

import gelu_fit  # noqa: E402


def header_coeffs():
    src = open(os.path.join(CSRC, "device_common.h")).read()
    body = src[src.index("float gelu_erf(float z)"):]
    body = body[:body.index("\n}\n")]
    vals = dict(re.findall(r"\b(c\d) = ([-+0-9.e]+)f", body))
    return np.array([float(vals[f"c{k}"]) for k in range(len(vals))], np.float32)


def test_header_matches_fit():
    c = header_coeffs()
    assert len(c) == gelu_fit.DEGREE + 1
    np.testing.assert_allclose(c, gelu_fit.fit(), rtol=2e-6, atol=0)


def test_tail_relative_error():
    c = header_coeffs()
    assert gelu_fit.error_report(c)["max_rel_err_phi_0_6"] < 1e-5


def test_gelu_error_bound_and_special_values():
    c = header_coeffs()
    assert gelu_fit.error_report(c)["max_abs_err_gelu_over_max1z"] < 1e-6
    g = gelu_fit.gelu_fp32(c, np.array([0.0, -0.0, 1e-30, -1e-30, 50.0, -50.0], np.float32))
    assert g[0] == 0.0 and g[1] == 0.0
    # near zero gelu(z) = z / 2 to the tail's relative error
    assert abs(g[2] / 5e-31 - 1) < 1e-5 and abs(g[3] / -5e-31 - 1) < 1e-5
    assert g[4] == np.float32(50.0) and abs(g[5]) < 1e-7
    # odd part: gelu(z) - gelu(-z) = z, to the fp32 rounding of the terms
    z = np.linspace(0.0, 8.0, 4001).astype(np.float32)
    d = gelu_fit.gelu_fp32(c, z).astype(np.float64) - gelu_fit.gelu_fp32(c, -z)
    np.testing.assert_allclose(d, z, rtol=0, atol=2e-6 * 8)


@pytest.mark.parametrize("z", [-3.0, -1.0, -0.25, 0.5, 2.0])
def test_gelu_points(z):
    c = header_coeffs()
    got = float(gelu_fit.gelu_fp32(c, np.array([z], np.float32))[0])
    assert abs(got - float(gelu_fit.gelu_exact(np.float32(z)))) < 1e-6
