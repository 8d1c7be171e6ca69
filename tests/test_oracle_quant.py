"""Pins of the int8 oracle (partial quantization, Sec. 3.2 / Fig. 4a).

Each test checks a definition of ``oracle.quant`` against something other
than itself: exact rational arithmetic (fractions) and an error bound for
the float32 rescaling, round trips of every
code, brute-force integer loops on tiny shapes, and the float64 operator
definitions in the cases where quantization is exact (dyadic scales and
weights that are integer multiples of their scale, so every multiplier is a
power of two and the integer path must equal the rounded float result).  A
dropped zero point, a padding filled with the wrong code, a sign error in the
border correction, a mis-scaled bias or residual, or a wrong rounding fails
one of them.
"""

from fractions import Fraction

import numpy as np
import pytest

from oracle import brute, ops
from oracle import quant as Q


def _round_half_even(fr):
    """Fraction -> nearest integer, ties to even."""
    f = fr.numerator // fr.denominator  # floor
    rem = fr - f
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and f % 2 == 1):
        f += 1
    return f


def test_rescale_is_exact_for_power_of_two_factors():
    """With m = 2^-j and |a| < 2^24 the float32 product is exact, so the
    result is a * m rounded to nearest, ties to even (exact rationals)."""
    rng = np.random.default_rng(0)
    for _ in range(3000):
        a = int(rng.integers(-(2 ** 24) + 1, 2 ** 24))
        j = int(rng.integers(0, 40))
        want = _round_half_even(Fraction(a, 2 ** j))
        want = max(-(2 ** 20), min(2 ** 20, want))
        assert int(Q.rescale(a, 2.0 ** -j)) == want, (a, j)
    assert int(Q.rescale(3, 0.5)) == 2 and int(Q.rescale(5, 0.5)) == 2  # ties to even
    assert int(Q.rescale(-3, 0.5)) == -2 and int(Q.rescale(-1, 0.5)) == 0


def test_rescale_error_bound():
    """For any factor the result is within half a unit plus the float32
    rounding of a and of the product (2^-23 relative each) of a * m."""
    rng = np.random.default_rng(1)
    a = rng.integers(-(2 ** 31) + 1, 2 ** 31, size=5000)
    m = 10.0 ** rng.uniform(-9, 0, size=5000)
    for ai, mi in zip(a, m):
        exact = int(ai) * float(np.float32(mi))
        got = int(Q.rescale(int(ai), mi))
        assert abs(got - max(-2.0 ** 20, min(2.0 ** 20, exact))) <= 0.5 + abs(exact) * 2.0 ** -22 + 1e-9
    with pytest.raises(ValueError):
        Q.multiplier(2.0 ** 20)
    with pytest.raises(ValueError):
        Q.multiplier(0.0)
    assert int(Q.rescale(2 ** 30, 0.5)) == 2 ** 20  # saturation


@pytest.mark.parametrize("scale,zp", [(0.02, 0), (0.0371, -128), (1.7, 45), (2.0 ** -6, 127)])
def test_quantize_dequantize_round_trips(scale, zp):
    codes = np.arange(-128, 128)
    back = Q.quantize(Q.dequantize(codes, scale, zp), scale, zp)
    assert np.array_equal(back, codes)
    rng = np.random.default_rng(2)
    lo, hi = scale * (-128 - zp), scale * (127 - zp)
    x = rng.uniform(lo, hi, 5000).astype(np.float32)
    err = np.abs(Q.dequantize(Q.quantize(x, scale, zp), scale, zp).astype(np.float64) - x)
    assert err.max() <= scale * (0.5 + 1e-5)
    # saturation outside the range
    assert Q.quantize(np.float32(hi + 10 * scale), scale, zp) == 127
    assert Q.quantize(np.float32(lo - 10 * scale), scale, zp) == -128
    # float32 product, ties to even: x = 2.5 S lands on code Z + 2
    assert Q.quantize(np.float32(2.5 * 2.0 ** -6), 2.0 ** -6, 0) == 2


def test_weights_quantize_per_channel_symmetric():
    rng = np.random.default_rng(3)
    j = rng.integers(-127, 128, size=(5, 3, 2, 2))
    j[:, 0, 0, 0] = 127  # channel maximum
    w = j * 2.0 ** -7
    wq, s_w = Q.quantize_weights(w)
    assert np.array_equal(wq, j) and np.all(s_w == 2.0 ** -7)
    w2 = rng.normal(size=(4, 7))
    wq2, s2 = Q.quantize_weights(w2)
    assert np.all(np.abs(wq2).max(axis=1) == 127)
    assert np.all(np.abs(wq2 * s2[:, None] - w2) <= s2[:, None] / 2 + 1e-15)
    wq0, s0 = Q.quantize_weights(np.zeros((2, 3)))
    assert np.all(wq0 == 0) and np.all(s0 == 1.0)


def test_relu6_bound_in_code_space():
    assert Q.act_bounds("relu6", 0.05, -100) == (-100, 20)
    assert Q.act_bounds("relu", 0.05, -100) == (-100, 127)
    assert Q.act_bounds(None, 0.05, 3) == (-128, 127)
    with pytest.raises(ValueError):
        Q.act_bounds("gelu", 0.1, 0)
    assert Q.act_bounds("leaky", 0.05, -100) == (-128, 127)


def test_leaky_codes_scale_negative_offsets():
    """Leaky ReLU on codes is the float leaky ReLU of the dequantized value,
    re-rounded: exact when alpha * offset is an integer, ties to even."""
    v = np.arange(-128, 128)
    z = -20
    out = Q.leaky_codes(v, z, 0.25)
    t = v - z
    assert np.array_equal(out[t >= 0], v[t >= 0])
    want = z + np.array([_round_half_even(Fraction(int(x), 4)) for x in t[t < 0]])
    assert np.array_equal(out[t < 0], want)
    assert Q.leaky_codes(np.array([z - 2]), z, 0.25)[0] == z - 0   # -0.5 -> 0 (even)
    assert Q.leaky_codes(np.array([z - 6]), z, 0.25)[0] == z - 2   # -1.5 -> -2 (even)


@pytest.mark.parametrize("shape,wshape,strides,padding", [
    ((1, 2, 5, 4), (3, 2, 3, 3), (1, 1), (1, 1, 1, 1)),
    ((2, 3, 6, 7), (2, 3, 3, 2), (2, 1), (2, 0, 1, 1)),
    ((1, 1, 4, 4), (2, 1, 1, 1), (1, 1), (0, 0, 0, 0)),
])
def test_integer_conv_against_brute_force(shape, wshape, strides, padding):
    rng = np.random.default_rng(4)
    xq = rng.integers(-128, 128, size=shape)
    wq = rng.integers(-127, 128, size=wshape)
    zx = 37
    got = Q.conv_accumulate(xq, zx, wq, strides, padding)
    # taps outside the image contribute nothing: brute force over (x - Z)
    want = np.array(brute.conv2d((xq - zx).tolist(), wq.tolist(), strides, padding))
    assert np.array_equal(got, want.astype(np.int64))


def _dyadic_case(seed, zx, zy, act, residual):
    """Codes and constants for which int8 execution is exact: S_x = 2^-5,
    S_w = 2^-7 (weights integer multiples of it, channel maximum 127),
    S_y = 2^-3, so the accumulator multiplier is 2^-9; the bias is an
    integer multiple of S_x S_w; a residual shares S_y (multiplier 1)."""
    rng = np.random.default_rng(seed)
    sx, sw, sy = 2.0 ** -5, 2.0 ** -7, 2.0 ** -3
    xq = rng.integers(-128, 128, size=(2, 3, 6, 5))
    j = rng.integers(-127, 128, size=(4, 3, 3, 3))
    j[:, 0, 0, 0] = 127
    w = j * sw
    b = rng.integers(-3000, 3000, size=4) * (sx * sw)
    rq = rng.integers(-128, 128, size=(2, 4, 3, 3)) if residual else None
    return sx, sy, xq, w, b, rq


@pytest.mark.parametrize("zx,zy,act,residual", [(0, 0, None, False), (37, -20, None, False),
                                                 (-90, -128, "relu", True), (11, 5, "relu6", True)])
def test_quantized_conv_equals_rounded_float_conv(zx, zy, act, residual):
    sx, sy, xq, w, b, rq = _dyadic_case(5, zx, zy, act, residual)
    attrs = {"strides": (2, 2), "padding": (1, 1, 1, 1)}
    qr = (sy, 13) if residual else None
    got = Q.qconv(xq, (sx, zx), w, b, attrs, (sy, zy), act, rq, qr)
    # float definition on the dequantized input (zero padding = code Z_x)
    yf = ops.bias_add(ops.conv2d(sx * (xq - zx), w, (2, 2), (1, 1, 1, 1)), b)
    if residual:
        yf = yf + sy * (rq - 13)
    t = yf / sy  # exact: dyadic values far below 2^24 (float32 products exact)
    want = zy + np.rint(t)
    lo, hi = Q.act_bounds(act, sy, zy)
    want = np.clip(np.clip(want, lo, hi), -128, 127)
    assert np.array_equal(got, want.astype(np.int64))


def test_quantized_dense_equals_rounded_float_dense():
    rng = np.random.default_rng(6)
    sx, sw, sy, zx, zy = 2.0 ** -4, 2.0 ** -7, 2.0 ** -2, -50, 9
    xq = rng.integers(-128, 128, size=(5, 40))
    j = rng.integers(-127, 128, size=(6, 40))
    j[:, 0] = -127
    b = rng.integers(-500, 500, size=6) * (sx * sw)
    got = Q.qdense(xq, (sx, zx), j * sw, b, (sy, zy), "relu")
    t = ops.bias_add(ops.dense(sx * (xq - zx), j * sw), b) / sy
    want = np.clip(np.maximum(zy + np.rint(t), zy), -128, 127)
    assert np.array_equal(got, want.astype(np.int64))


def test_max_pool_commutes_with_dequantize():
    rng = np.random.default_rng(7)
    xq = rng.integers(-128, 128, size=(2, 3, 7, 6))
    attrs = {"pool_size": (3, 3), "strides": (2, 2), "padding": (1, 1, 1, 1)}
    got = Q.qmax_pool2d(xq, attrs)
    want = brute.max_pool2d(xq.tolist(), (3, 3), (2, 2), (1, 1, 1, 1))
    assert np.array_equal(got, np.array(want, dtype=np.int64))
    s, z = 0.07, -30
    assert np.array_equal(Q.dequantize(got, s, z),
                          ops.max_pool2d(Q.dequantize(xq, s, z), (3, 3), (2, 2), (1, 1, 1, 1)).astype(np.float32))


def test_global_avg_pool_rounds_the_mean():
    rng = np.random.default_rng(8)
    xq = rng.integers(-128, 128, size=(3, 5, 4, 4))
    s, zx, zy = 0.1, 17, -3
    got = Q.qglobal_avg_pool2d(xq, (s, zx), (s, zy))  # multiplier 1/16: exact
    want = [[zy + _round_half_even(Fraction(int((xq[n, c] - zx).sum()), 16)) for c in range(5)]
            for n in range(3)]
    assert np.array_equal(got, np.clip(np.array(want), -128, 127))


def test_add_with_shared_scale_is_integer_sum():
    rng = np.random.default_rng(9)
    a = rng.integers(-128, 128, size=(2, 8))
    b = rng.integers(-128, 128, size=(2, 8))
    s = 0.25
    got = Q.qadd(a, (s, 10), b, (s, -4), (s, 2), "relu")
    want = np.clip(np.maximum((a - 10) + (b + 4) + 2, 2), -128, 127)
    assert np.array_equal(got, want)


def _tiny_int8_graph():
    rng = np.random.default_rng(10)
    w1 = rng.normal(0, 0.3, size=(8, 3, 3, 3)).astype(np.float32)
    b1 = rng.normal(0, 0.1, size=8).astype(np.float32)
    w2 = rng.normal(0, 0.2, size=(8, 8, 1, 1)).astype(np.float32)
    wd = rng.normal(0, 0.2, size=(5, 8)).astype(np.float32)

    def q(s, z):
        return {"scale": s, "zero_point": z}

    g = {"format": "byoc-subgraph", "version": 1,
         "inputs": [{"name": "x", "shape": [2, 3, 9, 9], "dtype": "f32", "quant": q(1 / 255, -128)}],
         "constants": [{"name": "w1", "index": 0, "shape": [8, 3, 3, 3], "dtype": "f32"},
                       {"name": "b1", "index": 1, "shape": [8], "dtype": "f32"},
                       {"name": "w2", "index": 2, "shape": [8, 8, 1, 1], "dtype": "f32"},
                       {"name": "wd", "index": 3, "shape": [5, 8], "dtype": "f32"}],
         "nodes": [
             {"name": "c1", "composite": "conv2d_bias_relu", "inputs": ["x", "w1", "b1"], "out_dtype": "int8",
              "attrs": {"strides": [1, 1], "padding": [1, 1, 1, 1]}, "quant": q(0.02, -128)},
             {"name": "c2", "composite": "conv2d_add_relu", "inputs": ["c1", "w2", "c1"], "out_dtype": "int8",
              "quant": q(0.03, -128)},
             {"name": "p", "composite": "max_pool2d", "inputs": ["c2"], "out_dtype": "int8",
              "attrs": {"pool_size": [3, 3], "strides": [2, 2], "padding": [1, 1, 1, 1]}, "quant": q(0.03, -128)},
             {"name": "g", "composite": "global_avg_pool2d", "inputs": ["p"], "out_dtype": "int8",
              "quant": q(0.02, -128)},
             {"name": "d", "composite": "dense", "inputs": ["g", "wd"], "out_dtype": "int8", "quant": q(0.01, 0)}],
         "outputs": [{"name": "d", "dtype": "f32"}]}
    return g, [w1, b1, w2, wd]


def test_int8_graph_tracks_the_float_graph():
    """The int8 executor reproduces the float graph within the quantization
    error (a sanity bound, not an exact pin), and its codes chain through
    the per-op definitions above."""
    from oracle.graph import run_graph
    g, consts = _tiny_int8_graph()
    x = np.random.default_rng(11).random((2, 3, 9, 9)).astype(np.float32)
    got, codes = Q.run_quantized_graph(g, consts, [x], keep=True)
    gf = {**g, "nodes": [{**n, "out_dtype": "f32"} for n in g["nodes"]]}
    ref = run_graph(gf, consts, [x], mode="exact")[0]
    assert np.max(np.abs(got[0] - ref)) < 0.06
    c1 = Q.qconv(Q.quantize(x, 1 / 255, -128), (1 / 255, -128), consts[0], consts[1],
                 {"strides": [1, 1], "padding": [1, 1, 1, 1]}, (0.02, -128), "relu")
    assert np.array_equal(codes["c1"], c1)
    assert np.array_equal(got[0], Q.dequantize(codes["d"], 0.01, 0))


def test_int8_graph_rejects_pool_rescaling():
    g, consts = _tiny_int8_graph()
    g["nodes"][2]["quant"] = {"scale": 0.05, "zero_point": -128}
    with pytest.raises(ValueError):
        Q.run_quantized_graph(g, consts, [np.zeros((2, 3, 9, 9), np.float32)])


def test_quantized_depthwise_equals_rounded_float_depthwise():
    """Depthwise (one input channel per output channel): the dyadic case
    against the float64 grouped conv on dequantized codes."""
    rng = np.random.default_rng(14)
    sx, sw, sy, zx, zy = 2.0 ** -5, 2.0 ** -7, 2.0 ** -3, 23, -7
    xq = rng.integers(-128, 128, size=(2, 6, 7, 5))
    j = rng.integers(-127, 128, size=(6, 1, 3, 3))
    j[:, 0, 0, 0] = 127
    b = rng.integers(-900, 900, size=6) * (sx * sw)
    attrs = {"strides": (2, 1), "padding": (1, 1, 1, 1), "groups": 6}
    got = Q.qconv(xq, (sx, zx), j * sw, b, attrs, (sy, zy), "relu6")
    t = ops.bias_add(ops.conv2d(sx * (xq - zx), j * sw, (2, 1), (1, 1, 1, 1), groups=6), b) / sy
    lo, hi = Q.act_bounds("relu6", sy, zy)
    want = np.clip(np.clip(zy + np.rint(t), lo, hi), -128, 127)
    assert np.array_equal(got, want.astype(np.int64))


def test_int8_graph_wiring_dyadic_hand_derived():
    """A five-node int8 graph whose scales make every rescaling an exact
    integer operation, checked code by code against the arithmetic written
    out here with plain integers (not the oracle's helpers): a 1x1 conv with
    two output channels of different weight scales, bias and a residual of
    another scale; a max pool keeping its input's (S, Z); an add of the pool
    and an input of a third scale; a global average pool; a dense layer.  A
    residual, pool or add operand wired to the wrong tensor's scale or zero
    point, or a pool over the wrong window count, changes the codes.

    Scales: x (1/4, 0), r (1/2, -3), conv (1/4, 5), add (1/4, -10),
    pool of the add (1/16, 0), dense (1/16, 0).  Weights [1, -2] quantize to
    codes [127, -127] with scales [1/127, 2/127], biases [1/2, -1/2] to
    [254, -127], so the conv terms are x_q + 2 and -2 (x_q + 1) exactly."""
    q = lambda s, z: {"scale": s, "zero_point": z}
    rng = np.random.default_rng(5)
    xq = rng.integers(-8, 12, size=(1, 1, 4, 4))
    rq = rng.integers(-6, 7, size=(1, 2, 4, 4))
    zq = rng.integers(-3, 4, size=(1, 2, 2, 2))
    x = (xq * 0.25).astype(np.float32)
    r = ((rq + 3) * 0.5).astype(np.float32)
    z = zq.astype(np.float32)
    w = np.array([1.0, -2.0], np.float32).reshape(2, 1, 1, 1)
    b = np.array([0.5, -0.5], np.float32)
    wd = np.array([[1.0, 0.0], [0.0, 1.0], [1.0, -1.0]], np.float32)
    g = {"format": "byoc-subgraph", "version": 1,
         "inputs": [{"name": "x", "shape": [1, 1, 4, 4], "dtype": "f32", "quant": q(0.25, 0)},
                    {"name": "r", "shape": [1, 2, 4, 4], "dtype": "f32", "quant": q(0.5, -3)},
                    {"name": "z", "shape": [1, 2, 2, 2], "dtype": "f32", "quant": q(1.0, 0)}],
         "constants": [{"name": "w", "index": 0, "shape": [2, 1, 1, 1], "dtype": "f32"},
                       {"name": "b", "index": 1, "shape": [2], "dtype": "f32"},
                       {"name": "wd", "index": 2, "shape": [3, 2], "dtype": "f32"}],
         "nodes": [
             {"name": "c", "composite": "conv2d_bias_add_relu", "inputs": ["x", "w", "b", "r"], "out_dtype": "int8",
              "attrs": {"strides": [1, 1], "padding": [0, 0, 0, 0]}, "quant": q(0.25, 5)},
             {"name": "p", "composite": "max_pool2d", "inputs": ["c"], "out_dtype": "int8",
              "attrs": {"pool_size": [2, 2], "strides": [2, 2], "padding": [0, 0, 0, 0]}, "quant": q(0.25, 5)},
             {"name": "s", "composite": "add_relu", "inputs": ["p", "z"], "out_dtype": "int8", "quant": q(0.25, -10)},
             {"name": "gp", "composite": "global_avg_pool2d", "inputs": ["s"], "out_dtype": "int8",
              "quant": q(1.0 / 16, 0)},
             {"name": "d", "composite": "dense", "inputs": ["gp", "wd"], "out_dtype": "int8", "quant": q(1.0 / 16, 0)}],
         "outputs": [{"name": "d", "dtype": "f32"}, {"name": "p", "dtype": "f32"}, {"name": "s", "dtype": "f32"}]}
    got = Q.run_quantized_graph(g, [w, b, wd], [x, r, z])

    clip = lambda v: max(-128, min(127, v))
    c = np.zeros((2, 4, 4), dtype=np.int64)
    for i in range(4):
        for j in range(4):
            t0 = (int(xq[0, 0, i, j]) + 2) + 2 * (int(rq[0, 0, i, j]) + 3)
            t1 = -2 * (int(xq[0, 0, i, j]) + 1) + 2 * (int(rq[0, 1, i, j]) + 3)
            c[0, i, j] = clip(max(5 + t0, 5))
            c[1, i, j] = clip(max(5 + t1, 5))
    p = np.zeros((2, 2, 2), dtype=np.int64)
    for k in range(2):
        for i in range(2):
            for j in range(2):
                p[k, i, j] = max(c[k, 2 * i + a, 2 * j + e] for a in range(2) for e in range(2))
    s = np.zeros((2, 2, 2), dtype=np.int64)
    for k in range(2):
        for i in range(2):
            for j in range(2):
                s[k, i, j] = clip(max(-10 + (p[k, i, j] - 5) + 4 * int(zq[0, k, i, j]), -10))
    gp = [clip(sum(int(s[k, i, j]) + 10 for i in range(2) for j in range(2))) for k in range(2)]
    d = [clip(gp[0]), clip(gp[1]), clip(gp[0] - gp[1])]
    assert np.array_equal(got[1][0], 0.25 * (p - 5)), (got[1][0], p)
    assert np.array_equal(got[2][0], 0.25 * (s + 10)), (got[2][0], s)
    assert np.array_equal(got[0][0], np.array(d, dtype=np.float64) / 16.0), (got[0][0], d)
