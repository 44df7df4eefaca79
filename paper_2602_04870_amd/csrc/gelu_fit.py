"""Constants of the forward GELU in ``device_common.hpp`` (``gelu_logistic``).

    python paper_2602_04870_amd/csrc/gelu_fit.py

The standard normal CDF is written as a logistic function of an odd
polynomial, Phi(z) ~ sigma(g(z)) with g(z) = z P(z^2) and P of degree 4, so
gelu(z) = z Phi(z) costs one exponential and one reciprocal plus a short
Horner chain.  P is fitted on [0, 6] by weighted minimax in the logit domain:
an error d in g moves sigma(g) by about Phi(1 - Phi) d, so minimising
max |Phi(1 - Phi) (g(z) - logit Phi(z))| over a grid is a linear programme in
P's coefficients.  Oddness makes the fit hold on [-6, 0] too; beyond |z| = 6
the fitted g keeps growing (checked to |z| = 60; past that the positive
leading coefficient dominates), so sigma(g) stays within fp32 rounding of 0
or 1 there.

Prints the coefficients pre-multiplied by -log2(e) (the kernel evaluates
exp2(z P'(z^2)) directly), rounded to fp32, and the largest |Phi error| of
the rounded constants evaluated in fp32.
"""
from __future__ import annotations

import numpy as np
from scipy.optimize import linprog
from scipy.special import log_ndtr, ndtr

DEGREE = 4
LOG2E = 1.4426950408889634


def fit(degree: int = DEGREE, zmax: float = 6.0, n: int = 4000) -> np.ndarray:
    z = np.linspace(1e-3, zmax, n)
    logit = log_ndtr(z) - log_ndtr(-z)
    w = ndtr(z) * ndtr(-z)
    basis = np.stack([z ** (2 * i + 1) for i in range(degree + 1)], axis=1)
    m = degree + 1
    # Variables: P's coefficients and the bound t; minimise t subject to
    # +-w (basis c - logit) <= t.
    a_ub = np.vstack([np.hstack([w[:, None] * basis, -np.ones((n, 1))]),
                      np.hstack([-w[:, None] * basis, -np.ones((n, 1))])])
    b_ub = np.concatenate([w * logit, -w * logit])
    res = linprog(np.r_[np.zeros(m), 1.0], A_ub=a_ub, b_ub=b_ub,
                  bounds=[(None, None)] * m + [(0, None)], method="highs")
    if not res.success:
        raise RuntimeError(res.message)
    return res.x[:m]


def kernel_constants(c: np.ndarray) -> np.ndarray:
    """P's coefficients (lowest degree first) times -log2(e), as fp32."""
    return (-LOG2E * c).astype(np.float32)


def phi_error_fp32(k: np.ndarray, zmax: float = 8.0, n: int = 400001) -> float:
    """max |Phi(z) - 1 / (1 + 2^(z P'(z^2)))| with every step in fp32."""
    z = np.linspace(-zmax, zmax, n).astype(np.float32)
    z2 = z * z
    p = np.full_like(z, k[-1])
    for c in k[-2::-1]:
        p = (p * z2 + c).astype(np.float32)
    with np.errstate(over="ignore"):
        r = (np.float32(1) / (np.float32(1) + np.exp2(z * p))).astype(np.float32)
    return float(np.abs(r.astype(np.float64) - ndtr(z.astype(np.float64))).max())


def main() -> None:
    c = fit()
    zz = np.linspace(0.0, 60.0, 600001)
    g = zz * np.polyval(c[::-1], zz * zz)
    if not np.all(np.diff(g) > 0):
        raise RuntimeError("fitted g is not increasing on [0, 60]")
    k = kernel_constants(c)
    print("coefficients (x -log2 e, fp32, z^0 first):")
    for v in k:
        print(f"  {float(v):.9e}f")
    print(f"max |Phi error| in fp32 on [-8, 8]: {phi_error_fp32(k):.3e}")


if __name__ == "__main__":
    main()
