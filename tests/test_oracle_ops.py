"""Pins of the oracle's operator definitions.

Each operator is checked against something other than itself: pure-Python
brute force on tiny shapes, library routines (torch CPU float64 conv2d,
scipy.signal.correlate2d, math.erf), closed forms (1x1 conv = matrix
product, identity kernel, border tap counts, stride subsampling, linearity)
and invariants (ReLU non-negative and idempotent, GELU odd part, max-pool
membership).
"""

import json
import math
import os

import numpy as np
import pytest
import scipy.signal
import torch
import torch.nn.functional as F

from oracle import brute, ops

RNG = np.random.default_rng(1234)


def _rand(*shape):
    return RNG.standard_normal(shape)


CONV_CASES = [
    # n, c, h, w, k, r, s, stride, pad(t,l,b,r), groups
    (1, 3, 5, 5, 4, 3, 3, (1, 1), (1, 1, 1, 1), 1),
    (2, 4, 7, 6, 2, 3, 3, (2, 2), (1, 1, 1, 1), 1),
    (1, 2, 6, 7, 3, 1, 1, (1, 1), (0, 0, 0, 0), 1),
    (1, 4, 7, 7, 4, 3, 3, (2, 1), (0, 1, 2, 0), 1),
    (2, 4, 5, 5, 4, 3, 3, (1, 1), (1, 1, 1, 1), 4),
    (1, 4, 6, 6, 6, 3, 3, (2, 2), (1, 1, 1, 1), 2),
    (1, 3, 9, 9, 2, 5, 5, (2, 2), (2, 2, 2, 2), 1),
    (1, 2, 4, 4, 3, 2, 3, (1, 2), (0, 1, 1, 1), 1),
]


@pytest.mark.parametrize("case", CONV_CASES)
def test_conv2d_matches_brute_force(case):
    n, c, h, w, k, r, s, stride, pad, groups = case
    x = _rand(n, c, h, w)
    wt = _rand(k, c // groups, r, s)
    got = ops.conv2d(x, wt, stride, pad, groups)
    ref = np.array(brute.conv2d(x.tolist(), wt.tolist(), stride, pad, groups))
    assert got.shape == ref.shape
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-12)


@pytest.mark.parametrize("case", CONV_CASES)
def test_conv2d_matches_torch_library(case):
    n, c, h, w, k, r, s, stride, pad, groups = case
    x = _rand(n, c, h, w)
    wt = _rand(k, c // groups, r, s)
    xt = F.pad(torch.from_numpy(x), (pad[1], pad[3], pad[0], pad[2]))
    ref = F.conv2d(xt, torch.from_numpy(wt), stride=stride, groups=groups).numpy()
    got = ops.conv2d(x, wt, stride, pad, groups)
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-12)


def test_conv2d_resnet_shapes_match_torch():
    # larger shapes of the kind the workloads use (7x7/2 stem, 1x1/2, 3x3)
    for (c, h, k, r, st, p) in [(3, 32, 8, 7, 2, 3), (16, 14, 32, 1, 2, 0), (32, 9, 16, 3, 1, 1)]:
        x = _rand(2, c, h, h)
        wt = _rand(k, c, r, r)
        ref = F.conv2d(torch.from_numpy(x), torch.from_numpy(wt), stride=st, padding=p).numpy()
        got = ops.conv2d(x, wt, (st, st), (p, p, p, p))
        np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-11)


def test_conv1x1_is_channel_matmul():
    x = _rand(2, 5, 4, 3)
    wt = _rand(6, 5, 1, 1)
    got = ops.conv2d(x, wt)
    ref = np.matmul(wt[:, :, 0, 0], x.reshape(2, 5, 12)).reshape(2, 6, 4, 3)
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-12)


def test_identity_kernel_returns_input():
    x = _rand(2, 4, 6, 5)
    wt = np.zeros((4, 4, 3, 3))
    for c in range(4):
        wt[c, c, 1, 1] = 1.0
    assert np.array_equal(ops.conv2d(x, wt, (1, 1), (1, 1, 1, 1)), x)


def test_border_tap_counts(golden_dir):
    with open(os.path.join(golden_dir, "conv_ones_border.json")) as f:
        g = json.load(f)
    c, h, w = g["C"], g["H"], g["W"]
    y = ops.conv2d(np.ones((1, c, h, w)), np.ones((3, c, 3, 3)), (1, 1), (1, 1, 1, 1))
    for k in range(3):
        assert np.array_equal(y[0, k], np.array(g["expected_per_channel_out"], dtype=float))


def test_stride2_is_subsampled_stride1():
    x = _rand(1, 3, 9, 8)
    wt = _rand(2, 3, 3, 3)
    y1 = ops.conv2d(x, wt, (1, 1), (1, 1, 1, 1))
    y2 = ops.conv2d(x, wt, (2, 2), (1, 1, 1, 1))
    np.testing.assert_allclose(y2, y1[:, :, ::2, ::2], rtol=0, atol=1e-12)


def test_conv_linearity():
    x1, x2 = _rand(1, 3, 6, 6), _rand(1, 3, 6, 6)
    wt = _rand(4, 3, 3, 3)
    a, b = 0.7, -1.3
    lhs = ops.conv2d(a * x1 + b * x2, wt, (1, 1), (1, 1, 1, 1))
    rhs = a * ops.conv2d(x1, wt, (1, 1), (1, 1, 1, 1)) + b * ops.conv2d(x2, wt, (1, 1), (1, 1, 1, 1))
    np.testing.assert_allclose(lhs, rhs, rtol=0, atol=1e-12)


def test_depthwise_matches_scipy_correlate2d():
    c = 6
    x = _rand(2, c, 9, 7)
    wt = _rand(c, 1, 3, 3)
    got = ops.conv2d(x, wt, (1, 1), (1, 1, 1, 1), groups=c)
    for n in range(2):
        for ch in range(c):
            ref = scipy.signal.correlate2d(x[n, ch], wt[ch, 0], mode="same", boundary="fill")
            np.testing.assert_allclose(got[n, ch], ref, rtol=0, atol=1e-12)


def test_dense_matches_brute_force():
    x = _rand(5, 7)
    wt = _rand(3, 7)
    np.testing.assert_allclose(ops.dense(x, wt), np.array(brute.dense(x.tolist(), wt.tolist())),
                               rtol=0, atol=1e-12)


def test_dense_equals_conv1x1_on_1x1_image():
    x = _rand(4, 6)
    wt = _rand(5, 6)
    y = ops.conv2d(x.reshape(4, 6, 1, 1), wt.reshape(5, 6, 1, 1)).reshape(4, 5)
    np.testing.assert_allclose(ops.dense(x, wt), y, rtol=0, atol=1e-12)


def test_bias_add_axis():
    y = np.zeros((2, 3, 2, 2))
    b = np.array([1.0, 2.0, 3.0])
    out = ops.bias_add(y, b)
    for k in range(3):
        assert np.all(out[:, k] == b[k])
    assert np.array_equal(ops.bias_add(np.zeros((4, 3)), b), np.tile(b, (4, 1)))


def test_relu_family_invariants():
    x = _rand(1000) * 5
    r = ops.relu(x)
    assert np.all(r >= 0)
    assert np.array_equal(ops.relu(r), r)
    np.testing.assert_allclose(ops.relu(x) - ops.relu(-x), x, rtol=0, atol=0)
    r6 = ops.relu6(x)
    assert np.all((r6 >= 0) & (r6 <= 6))
    inside = (x > 0) & (x < 6)
    assert np.array_equal(r6[inside], x[inside])


def test_leaky_relu_piecewise_and_closed_forms():
    x = _rand(1000) * 5
    for a in (0.1, 0.0, 0.25):
        y = ops.leaky_relu(x, a)
        ref = np.array([v if v >= 0 else a * v for v in x])  # the scalar definition
        assert np.array_equal(y, ref)
        # relu(x) - a relu(-x) is the same function
        np.testing.assert_allclose(y, ops.relu(x) - a * ops.relu(-x), rtol=0, atol=1e-15)
    assert np.array_equal(ops.leaky_relu(x, 0.0), ops.relu(x))


def test_gelu_against_math_erf_and_odd_part():
    x = np.linspace(-8, 8, 2001)
    g = ops.gelu(x)
    ref = np.array([brute.gelu(float(v)) for v in x])
    np.testing.assert_allclose(g, ref, rtol=1e-15, atol=1e-15)
    np.testing.assert_allclose(g - ops.gelu(-x), x, rtol=0, atol=1e-12)
    assert ops.gelu(np.array([0.0]))[0] == 0.0


def test_gelu_far_left_tail_against_ndtr():
    """y * Phi(y) for y << 0, against SciPy's normal CDF routine (ndtr, not
    the erfc the oracle calls): relative accuracy down to y = -37, where
    Phi(y) is about 6e-300; the form (1 + erf(y / sqrt 2)) / 2 cancels to
    nothing there (already about 20% off at y = -8)."""
    from scipy.special import ndtr
    y = -np.geomspace(1.0, 37.0, 500)
    np.testing.assert_allclose(ops.gelu(y), y * ndtr(y), rtol=1e-12, atol=0)
    assert np.all(ops.gelu(y) < 0)


def test_gelu_against_normal_table(golden_dir):
    with open(os.path.join(golden_dir, "normal_cdf_table.json")) as f:
        t = json.load(f)
    z = np.array(t["z"])
    phi = np.array(t["Phi"])
    np.testing.assert_allclose(ops.gelu(z), z * phi, rtol=0, atol=t["abs_tol"] * 4)
    np.testing.assert_allclose(ops.gelu(-z), -z * (1 - phi), rtol=0, atol=t["abs_tol"] * 4)


@pytest.mark.parametrize("pool,stride,pad,shape", [
    ((3, 3), (2, 2), (1, 1, 1, 1), (2, 3, 7, 8)),
    ((3, 3), (1, 1), (1, 1, 1, 1), (1, 2, 5, 5)),
    ((2, 2), (2, 2), (0, 0, 0, 0), (1, 2, 6, 6)),
    ((3, 3), (2, 2), (0, 1, 1, 0), (1, 1, 6, 7)),
])
def test_max_pool_brute_and_membership(pool, stride, pad, shape):
    x = _rand(*shape)
    y = ops.max_pool2d(x, pool, stride, pad)
    ref = np.array(brute.max_pool2d(x.tolist(), pool, stride, pad))
    assert np.array_equal(y, ref)
    # every output is one of its window's elements and bounds them all
    n, c, h, w = shape
    for (ni, ci, p, q), v in np.ndenumerate(y):
        h0, w0 = p * stride[0] - pad[0], q * stride[1] - pad[1]
        win = x[ni, ci, max(h0, 0):h0 + pool[0], max(w0, 0):w0 + pool[1]]
        assert v in win and np.all(win <= v)


def test_max_pool_padding_moot_for_nonnegative_input():
    x = np.abs(_rand(1, 3, 8, 8))
    y = ops.max_pool2d(x, (3, 3), (2, 2), (1, 1, 1, 1))
    xp = np.pad(x, ((0, 0), (0, 0), (1, 1), (1, 1)))
    y0 = ops.max_pool2d(xp, (3, 3), (2, 2), (0, 0, 0, 0))
    assert np.array_equal(y, y0)


def test_global_avg_pool():
    x = _rand(2, 3, 4, 5)
    np.testing.assert_allclose(ops.global_avg_pool2d(x), np.array(brute.global_avg_pool2d(x.tolist())),
                               rtol=0, atol=1e-14)
    np.testing.assert_allclose(ops.global_avg_pool2d(x), x.mean(axis=(2, 3)), rtol=0, atol=1e-14)
    assert np.all(ops.global_avg_pool2d(np.full((1, 2, 7, 7), 3.25)) == 3.25)


def test_conv_output_size():
    assert ops.conv_output_size(224, 7, 2, 3, 3) == 112
    assert ops.conv_output_size(112, 3, 2, 1, 1) == 56
    assert ops.conv_output_size(56, 1, 2, 0, 0) == 28
    assert ops.conv_output_size(7, 3, 1, 1, 1) == 7
    assert math.floor((5 + 0 - 3) / 2) + 1 == ops.conv_output_size(5, 3, 2, 0, 0)


@pytest.mark.parametrize("pool,strides,padding,incl", [((3, 3), (1, 1), (1, 1, 1, 1), False),
                                                       ((3, 3), (1, 1), (1, 1, 1, 1), True),
                                                       ((3, 2), (2, 1), (1, 0, 0, 1), False),
                                                       ((2, 2), (2, 2), (0, 0, 0, 0), False)])
def test_avg_pool_against_brute_force(pool, strides, padding, incl):
    x = _rand(2 * 3 * 7 * 6).reshape(2, 3, 7, 6)
    got = ops.avg_pool2d(x, pool, strides, padding, incl)
    want = np.array(brute.avg_pool2d(x.tolist(), pool, strides, padding, incl))
    np.testing.assert_allclose(got, want, rtol=1e-14, atol=1e-14)


def test_avg_pool_closed_forms():
    # a constant image averages to itself when padding is not counted, and
    # to the constant times the inside fraction of the window when it is
    x = np.full((1, 2, 5, 5), 3.0)
    assert np.allclose(ops.avg_pool2d(x, (3, 3), (1, 1), (1, 1, 1, 1), False), 3.0)
    y = ops.avg_pool2d(x, (3, 3), (1, 1), (1, 1, 1, 1), True)
    assert y[0, 0, 0, 0] == 3.0 * 4 / 9 and y[0, 0, 0, 2] == 3.0 * 6 / 9 and y[0, 0, 2, 2] == 3.0
    # without padding, a window covering the image is the global mean
    z = _rand(2 * 3 * 4 * 4).reshape(2, 3, 4, 4)
    np.testing.assert_allclose(ops.avg_pool2d(z, (4, 4), (1, 1), (0, 0, 0, 0))[:, :, 0, 0],
                               ops.global_avg_pool2d(z), rtol=1e-13)  # same 16 terms, summed in another order


def test_concatenate_slices_back():
    a, b = _rand(2 * 3 * 4 * 5).reshape(2, 3, 4, 5), _rand(2 * 5 * 4 * 5).reshape(2, 5, 4, 5)
    y = ops.concatenate([a, b])
    assert y.shape == (2, 8, 4, 5)
    assert np.array_equal(y[:, :3], a) and np.array_equal(y[:, 3:], b)


@pytest.mark.parametrize("incl", [False, True])
def test_avg_pool_against_torch(incl):
    x = _rand(2 * 4 * 9 * 8).reshape(2, 4, 9, 8)
    want = F.avg_pool2d(torch.from_numpy(x), 3, stride=1, padding=1, count_include_pad=incl).numpy()
    np.testing.assert_allclose(ops.avg_pool2d(x, (3, 3), (1, 1), (1, 1, 1, 1), incl), want, rtol=1e-14, atol=1e-14)
