"""Host-side checks of constants compiled into the kernels.

The forward GELU of the expert FFN (``gelu_logistic`` in device_common.hpp)
writes the normal CDF as 1 / (1 + 2^(z P(z^2))) with P's coefficients fitted
by ``csrc/gelu_fit.py``.  These tests read the constants out of the source and
check them against scipy's normal CDF, evaluating every step in fp32 as the
kernel does: the error bound the header states, the limits at large |z| and
monotonicity (so gelu keeps its shape outside the fitted interval).
"""
from __future__ import annotations

import importlib.util
import os
import re

import numpy as np
import pytest
from scipy.special import ndtr

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2602_04870_amd", "csrc")


def _gelu_constants() -> np.ndarray:
    src = open(os.path.join(CSRC, "device_common.hpp")).read()
    body = src[src.index("float gelu_logistic(float z)"):]
    body = body[:body.index("}")]
    nums = [float(v) for v in re.findall(r"([-+]?\d\.\d+e[-+]\d+)f", body)]
    # Horner from the top: fmaf(c4, z2, c3), then c2, c1, c0.
    assert len(nums) == 5, nums
    return np.array([nums[4], nums[3], nums[2], nums[1], nums[0]], dtype=np.float32)


def _phi_fp32(k: np.ndarray, z: np.ndarray) -> np.ndarray:
    z = z.astype(np.float32)
    with np.errstate(over="ignore", invalid="ignore"):
        z2 = z * z
        p = np.full_like(z, k[-1])
        for c in k[-2::-1]:
            p = (p * z2 + c).astype(np.float32)
        return (np.float32(1) / (np.float32(1) + np.exp2(z * p))).astype(np.float32)


def test_gelu_constants_meet_the_stated_bound():
    k = _gelu_constants()
    z = np.linspace(-8.0, 8.0, 800001).astype(np.float32).astype(np.float64)
    err = np.abs(_phi_fp32(k, z).astype(np.float64) - ndtr(z))
    assert err.max() <= 1.6e-6, err.max()
    # gelu = z Phi(z): absolute error below 1.6e-6 |z| everywhere on the grid.
    g = (z.astype(np.float32) * _phi_fp32(k, z)).astype(np.float64)
    assert np.all(np.abs(g - z * ndtr(z)) <= 1.6e-6 * np.abs(z) + 2.0 ** -24 * np.abs(g))


def test_gelu_constants_limits_and_monotonicity():
    k = _gelu_constants()
    z = np.linspace(0.0, 60.0, 600001)
    phi = _phi_fp32(k, z)
    assert np.all(np.diff(phi.astype(np.float64)) >= 0)
    big = np.array([6.0, 10.0, 60.0, 1e3, 1e5, 1e30, np.inf], dtype=np.float32)
    assert np.all(_phi_fp32(k, big) == 1.0)
    # The bound is absolute: Phi(-6) ~ 1e-9 is within it, not resolved
    # relatively; further out the result is exactly 0.
    assert abs(float(_phi_fp32(k, -big[:1])[0]) - ndtr(-6.0)) <= 1.6e-6
    assert np.all(_phi_fp32(k, -big[1:]) == 0.0)
    # gelu(-inf) is -0, not NaN: the reciprocal of +inf is 0 and -inf * 0 would
    # be NaN, so the kernel only meets -inf through z * 0 with z finite.
    assert np.isfinite(np.float32(-1e30) * _phi_fp32(k, np.array([-1e30], np.float32)))
    assert _phi_fp32(k, np.array([0.0], np.float32))[0] == 0.5


def test_gelu_fit_script_reproduces_the_constants():
    spec = importlib.util.spec_from_file_location("gelu_fit", os.path.join(CSRC, "gelu_fit.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    k = mod.kernel_constants(mod.fit())
    np.testing.assert_allclose(k, _gelu_constants(), rtol=1e-5)
    # The fitted g (not just its fp32 evaluation) increases on [0, 60].
    c = mod.fit()
    zz = np.linspace(0.0, 60.0, 600001)
    assert np.all(np.diff(zz * np.polyval(c[::-1], zz * zz)) > 0)


@pytest.mark.parametrize("z0", [-3.0, -1.0, 0.5, 2.0])
def test_gelu_constants_match_the_erf_form_pointwise(z0):
    k = _gelu_constants()
    z = np.array([z0], dtype=np.float32)
    ref = z0 * 0.5 * (1.0 + __import__("math").erf(z0 / 2 ** 0.5))
    assert abs(float(z[0] * _phi_fp32(k, z)[0]) - ref) <= 1.6e-6 * abs(z0) + 1e-7


def test_slot_division_by_magic_multiply_is_exact():
    """The backward's floor(slot / k) as (slot * m) >> S with S = 31 +
    ceil(log2 k), m = ceil(2^S / k) (``div_magic`` / ``div_by_magic`` in
    device_common.hpp) equals integer division for every k the library
    accepts (1..32) over the slot range [0, 2^31), and the product stays
    below 2^64: at both ends, around multiples of k near the top and in the
    middle, and on random values."""
    rng = np.random.default_rng(7)
    top = (1 << 31) - 1
    for k in range(1, 33):
        c = max(0, (k - 1).bit_length())
        S = 31 + c
        m = ((1 << S) + k - 1) // k
        assert m <= (1 << 32) and top * m < (1 << 64), k
        q_hi = top // k
        edges = [0, 1, k - 1, k, k + 1, top, top - 1]
        for q in (q_hi, q_hi - 1, q_hi - 2, 1 << 20, (1 << 26) + 3):
            edges += [q * k - 1, q * k, q * k + k - 1]
        n = np.array([e for e in edges if 0 <= e <= top], dtype=np.uint64)
        n = np.concatenate([n, rng.integers(0, top + 1, 200000, dtype=np.uint64)])
        got = (n * np.uint64(m)) >> np.uint64(S)   # < 2^63: exact in uint64
        assert np.array_equal(got, n // np.uint64(k)), k
