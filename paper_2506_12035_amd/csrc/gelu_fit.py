"""Coefficients of the GELU epilogue's normal-tail polynomial (device_common.h).

The exact-erf GELU is z * Phi(z) = max(z, 0) - |z| * Phi(-|z|).  The kernels
evaluate Phi(-a) as 2^P(min(a, 6)), where P is a degree-7 polynomial close to
log2 Phi(-u) on [0, 6]: one exp2 and seven FMAs per element.

P is fitted here by Lawson-type iteratively reweighted least squares (each
pass raises the weights where the error is largest, moving the least-squares
fit toward the equal-ripple minimax polynomial), and its error is measured
with every step rounded to fp32 as the kernel evaluates it (Horner with
fused multiply-adds).  Run it to print the coefficients and the error bounds:

    python paper_2506_12035_amd/csrc/gelu_fit.py
"""
from __future__ import annotations

import numpy as np
from scipy.special import log_ndtr, ndtr

U_MAX = 6.0   # the polynomial's argument is clamped to [0, U_MAX]
DEGREE = 7


def fit(degree: int = DEGREE, u_max: float = U_MAX, passes: int = 60) -> np.ndarray:
    """Monomial coefficients c[0..degree] of P(u) ~ log2 Phi(-u) on [0, u_max]."""
    u = np.linspace(0.0, u_max, 40001)
    target = log_ndtr(-u) / np.log(2.0)
    v = np.vander(u, degree + 1, increasing=True)
    w = np.ones_like(u)
    c = None
    for _ in range(passes):
        c, *_ = np.linalg.lstsq(v * w[:, None], target * w, rcond=None)
        err = np.abs(v @ c - target)
        w = w * (1.0 + 3.0 * err / err.max())
    return c.astype(np.float32)


def p_fp32(c: np.ndarray, u: np.ndarray) -> np.ndarray:
    """P(u) evaluated as the kernel does: Horner, one fp32 rounding per FMA."""
    u = u.astype(np.float32)
    acc = np.full(u.shape, c[-1], np.float32)
    for k in range(len(c) - 2, -1, -1):
        acc = (acc.astype(np.float64) * u + np.float64(c[k])).astype(np.float32)
    return acc


def gelu_fp32(c: np.ndarray, z: np.ndarray) -> np.ndarray:
    """The kernel's GELU on fp32 inputs (exp2 and the final FMA rounded once each)."""
    z = z.astype(np.float32)
    a = np.abs(z)
    e = np.exp2(p_fp32(c, np.minimum(a, np.float32(U_MAX))).astype(np.float64)).astype(np.float32)
    return (np.maximum(z, 0).astype(np.float64) - a.astype(np.float64) * e).astype(np.float32)


def gelu_exact(z: np.ndarray) -> np.ndarray:
    z = np.asarray(z, np.float64)
    return z * ndtr(z)


def error_report(c: np.ndarray) -> dict:
    u = np.linspace(0.0, U_MAX, 60001)
    rel_phi = np.abs(np.exp2(p_fp32(c, u).astype(np.float64) - log_ndtr(-u) / np.log(2.0)) - 1.0)
    z = np.linspace(-40.0, 40.0, 400001)
    dz = np.abs(gelu_fp32(c, z).astype(np.float64) - gelu_exact(z.astype(np.float32)))
    return {"max_rel_err_phi_0_6": float(rel_phi.max()),
            "max_abs_err_gelu_over_max1z": float((dz / np.maximum(1.0, np.abs(z))).max())}


if __name__ == "__main__":
    coeffs = fit()
    for k, v in enumerate(coeffs):
        print(f"c{k} = {float(v):.9g}f")
    print(error_report(coeffs))
