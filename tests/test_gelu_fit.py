"""The GELU epilogue's erfc approximation (host side, no GPU): the
coefficients compiled into the kernels are the ones the committed fit
script produces, and evaluated in float32 the way the kernels evaluate
them they keep erfc within 1e-6 relative error over the whole range the
epilogue uses (erfc(10) is below float32).  The kernels' GELU itself is
checked on the GPU against the oracle over every bf16 input in a range
(tests/test_gpu_ops.py)."""

import os
import re
import sys

import numpy as np
import pytest
from scipy.special import erfc

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2105_03215_amd", "csrc")
sys.path.insert(0, CSRC)
import gelu_erfc_fit  # noqa: E402


def _kernel_coefficients():
    src = open(os.path.join(CSRC, "device_common.h")).read()
    m = re.search(r"kErfcP\[9\]\s*=\s*\{([^}]*)\}", src)
    assert m, "kErfcP table not found"
    return np.array([float(v.strip().rstrip("f")) for v in m.group(1).split(",")], dtype=np.float32)


def test_kernel_table_is_the_fit():
    np.testing.assert_array_equal(_kernel_coefficients(), gelu_erfc_fit.coefficients())


@pytest.mark.parametrize("lo,hi", [(0.0, 1.0), (1.0, 4.0), (4.0, 9.2)])
def test_erfc_relative_error_in_float32(lo, hi):
    a = np.linspace(lo, hi, 100001).astype(np.float32)
    got = gelu_erfc_fit.erfc_f32(a, _kernel_coefficients()).astype(np.float64)
    ref = erfc(a.astype(np.float64))
    assert np.max(np.abs(got - ref) / ref) < 1e-6


def test_gelu_from_the_fit_matches_the_exact_form():
    """x * Phi(x) assembled as the kernel does (Phi = erfc(a) / 2 below
    zero, 1 - erfc(a) / 2 above, a = |x| / sqrt 2 capped at 10) against
    x * erfc(-x / sqrt 2) / 2 in float64."""
    x = np.linspace(-14.0, 14.0, 200001).astype(np.float32)
    a = np.minimum(np.abs(x) * np.float32(0.70710678118654752440), np.float32(10.0)).astype(np.float32)
    ec = gelu_erfc_fit.erfc_f32(a, _kernel_coefficients())
    phi = np.where(x < 0, np.float32(0.5) * ec, np.float32(1.0) - np.float32(0.5) * ec).astype(np.float32)
    got = (x * phi).astype(np.float64)
    x64 = x.astype(np.float64)
    ref = x64 * 0.5 * erfc(-x64 / np.sqrt(2.0))
    # the float32 rounding of a = |x| / sqrt 2 alone moves erfc(a) by up to
    # about 2 a^2 2^-24 relative (exp(-a^2) is that sensitive to a), on top of
    # the approximation's 1e-6; float32 steps are absolute (2^-149) in the
    # denormal range that erfc(a) / 2 enters below x of about -13
    bound = (2e-6 + 2.5e-7 * a.astype(np.float64) ** 2) * np.abs(ref) + 2.0 ** -140
    assert np.all(np.abs(got - ref) <= bound)
