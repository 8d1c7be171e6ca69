"""Partial quantization: affine int8 execution of an offloaded subgraph.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Sec. 3.2 (Fig. 4a) lets an accelerator backend insert quantize and
dequantize nodes into a partitioned function, converting between floating
tensors T and fixed-point tensors T_q through a scale S and a zero point Z,
T = S (T_q - Z), with S and Z fixed at compile time from calibration data
or at run time.  The paper fixes neither the integer width nor the rounding
of the fixed-point arithmetic.  This module writes out the definitions the
int8 variant of the executor follows (each is a reading, listed with the
others in the design notes):

* codes are int8 in [-128, 127]; every activation tensor of the function
  carries its own (S, Z) with S > 0 and Z an int8 code;
* boundary quantize Q of a float input x (float32 arithmetic):
  q = clip(rint(fl32(x * fl32(1 / S))) + Z, -128, 127), rint ties to even;
* boundary dequantize DQ of codes q: y = fl32(fl32(S) * (q - Z));
* weights are quantized per output channel, symmetric (zero point 0):
  S_w[k] = max |W[k]| / 127 in float64 (1 for an all-zero channel),
  W_q = clip(rint(W / S_w[k]), -127, 127); a bias becomes the int32
  b_q[k] = rint(b[k] / (S_x S_w[k])) (saturated);
* a real rescaling factor m is applied in float32: rescale(a, m) =
  rint(fl32(fl32(a) * fl32(m))), ties to even, saturated to +-2^20 before the
  conversion back to an integer (one rounding of the product; the factor
  must be finite, positive and below 2^20);
* conv / dense (and depthwise conv, one input channel per output channel):
  acc = sum over taps inside the image and input channels of
  (x_q - Z_x) W_q, plus b_q (exact integers; padding contributes nothing,
  which is zero padding of the float tensor), then
  v = Z_y + rescale(acc, S_x S_w[k] / S_y) [+ rescale(r_q - Z_r, S_r / S_y)],
  the activation in code space (ReLU: v >= Z_y; ReLU6 also
  v <= Z_y + rint(6 / S_y); leaky ReLU: a negative offset t = v - Z_y
  becomes rint(fl32(t * alpha))), and a final clip to [-128, 127];
* max pooling takes the largest code of the window (monotone, so the output
  keeps the input's S and Z; padding never wins);
* global average pooling: v = Z_y + rescale(sum_hw (x_q - Z_x), S_x / (S_y H W));
* add: v = Z_y + rescale(a_q - Z_a, S_a / S_y) + rescale(b_q - Z_b, S_b / S_y),
  then the activation clamp and the clip.

The conv sum runs through ``ops.conv2d`` in float64 on integer-valued
arrays: every partial sum is an integer far below 2^53, so the result is
the exact integer whatever the summation order.
"""

import numpy as np

from . import ops
from .graph import load_graph, parse_composite

QMIN, QMAX = -128, 127


def _as_f32(v):
    return np.asarray(v, dtype=np.float32)


RESCALE_LIMIT = 2.0 ** 20


def multiplier(m):
    """The float32 form of a real rescaling factor (finite, 0 < m < 2^20)."""
    m32 = np.float32(float(m))
    if not (np.isfinite(m32) and 0.0 < float(m32) < RESCALE_LIMIT):
        raise ValueError("rescaling factor %r outside (0, 2^20)" % m)
    return m32


def rescale(a, m):
    """rint(fl32(fl32(a) * fl32(m))) as int64, saturated to +-2^20."""
    t = np.rint(np.asarray(a, dtype=np.int64).astype(np.float32) * multiplier(m))
    return np.clip(t, -RESCALE_LIMIT, RESCALE_LIMIT).astype(np.int64)


def quantize(x, scale, zero_point):
    """Boundary Q: float tensor -> int8 codes (float32 arithmetic)."""
    inv = np.float32(1.0 / float(scale))
    t = np.rint(_as_f32(x) * inv)  # float32 product, rounded to an integer value
    t = np.clip(t, -512.0, 512.0).astype(np.int64)
    return np.clip(t + int(zero_point), QMIN, QMAX).astype(np.int64)


def dequantize(q, scale, zero_point):
    """Boundary DQ: int8 codes -> float32 values."""
    d = (np.asarray(q, dtype=np.int64) - int(zero_point)).astype(np.float32)
    return np.float32(scale) * d


def quantize_weights(w):
    """Per-output-channel symmetric int8 weights: (W_q, S_w)."""
    w = np.asarray(w, dtype=np.float64)
    k = w.shape[0]
    amax = np.abs(w.reshape(k, -1)).max(axis=1)
    s_w = np.where(amax > 0, amax / 127.0, 1.0)
    wq = np.rint(w / s_w.reshape((k,) + (1,) * (w.ndim - 1)))
    return np.clip(wq, -127, 127).astype(np.int64), s_w


def quantize_bias(b, s_x, s_w):
    """int32 bias in the accumulator's scale S_x S_w[k]."""
    q = np.rint(np.asarray(b, dtype=np.float64) / (float(s_x) * s_w))
    return np.clip(q, -2.0 ** 31, 2.0 ** 31 - 1).astype(np.int64)


def act_bounds(act, s_y, z_y):
    """Code-space clamp [lo, hi] of an activation on a tensor (S_y, Z_y)."""
    lo, hi = QMIN, QMAX
    if act in ("relu", "relu6"):
        lo = int(z_y)
    if act == "relu6":
        hi = int(z_y) + int(np.rint(6.0 / float(s_y)))
    if act not in (None, "relu", "relu6", "leaky"):
        raise ValueError("activation %r has no int8 form" % act)
    return lo, hi


def leaky_codes(v, z_y, alpha):
    """Leaky ReLU on codes: the offset t = v - Z_y is kept where t >= 0 and
    becomes rint(fl32(fl32(t) * fl32(alpha))) below (float32, ties to even)."""
    t = np.asarray(v, dtype=np.int64) - int(z_y)
    neg = np.rint(t.astype(np.float32) * np.float32(alpha)).astype(np.int64)
    return int(z_y) + np.where(t < 0, neg, t)


def _requant_out(v, act, s_y, z_y, alpha=0.1):
    if act == "leaky":
        v = leaky_codes(v, z_y, alpha)
    lo, hi = act_bounds(act, s_y, z_y)
    v = np.maximum(v, lo)
    v = np.minimum(v, hi)
    return np.clip(v, QMIN, QMAX)


def conv_accumulate(xq, zx, wq, strides, padding, groups=1):
    """Exact integer sum of (x_q - Z_x) W_q over the taps inside the image."""
    d = np.asarray(xq, dtype=np.int64) - int(zx)
    acc = ops.conv2d(d.astype(np.float64), np.asarray(wq, dtype=np.float64), strides, padding, groups)
    return np.rint(acc).astype(np.int64)


def qconv(xq, qx, w, b, attrs, qy, act=None, res=None, qr=None, alpha=0.1):
    """Quantized conv2d composite on NCHW codes.  qx, qy, qr are (S, Z)."""
    wq, s_w = quantize_weights(w)
    acc = conv_accumulate(xq, qx[1], wq, tuple(attrs.get("strides", (1, 1))),
                          tuple(attrs.get("padding", (0, 0, 0, 0))), int(attrs.get("groups", 1)))
    return _qepilogue(acc, s_w, b, qx, qy, act, res, qr, axis_shape=(1, -1, 1, 1), alpha=alpha)


def qdense(xq, qx, w, b, qy, act=None, res=None, qr=None, alpha=0.1):
    """Quantized dense composite on [M, K] codes."""
    wq, s_w = quantize_weights(w)
    d = (np.asarray(xq, dtype=np.int64) - int(qx[1])).astype(np.float64)
    acc = np.rint(ops.dense(d, wq.astype(np.float64))).astype(np.int64)
    return _qepilogue(acc, s_w, b, qx, qy, act, res, qr, axis_shape=(1, -1), alpha=alpha)


def _qepilogue(acc, s_w, b, qx, qy, act, res, qr, axis_shape, alpha=0.1):
    s_x, _ = qx
    s_y, z_y = qy
    if b is not None:
        acc = acc + quantize_bias(b, s_x, s_w).reshape(axis_shape)
    v = np.empty_like(acc)
    for k in range(acc.shape[1]):
        v[:, k] = rescale(acc[:, k], (float(s_x) * s_w[k]) / float(s_y))
    v = v + int(z_y)
    if res is not None:
        v = v + rescale(np.asarray(res, dtype=np.int64) - int(qr[1]), float(qr[0]) / float(s_y))
    return _requant_out(v, act, s_y, z_y, alpha)


def qmax_pool2d(xq, attrs):
    """Max pooling of codes (padding never wins)."""
    y = ops.max_pool2d(np.asarray(xq, dtype=np.float64), tuple(attrs.get("pool_size", (3, 3))),
                       tuple(attrs.get("strides", (2, 2))), tuple(attrs.get("padding", (1, 1, 1, 1))))
    return y.astype(np.int64)


def qglobal_avg_pool2d(xq, qx, qy):
    """Global average pooling of codes: [N, C, H, W] -> [N, C]."""
    xq = np.asarray(xq, dtype=np.int64)
    n, c, h, w = xq.shape
    tot = (xq - int(qx[1])).sum(axis=(2, 3))
    return np.clip(int(qy[1]) + rescale(tot, float(qx[0]) / (float(qy[0]) * h * w)), QMIN, QMAX)


def qadd(aq, qa, bq, qb, qy, act=None, alpha=0.1):
    """Quantized elementwise add with activation."""
    v = (int(qy[1]) + rescale(np.asarray(aq, dtype=np.int64) - int(qa[1]), float(qa[0]) / float(qy[0]))
         + rescale(np.asarray(bq, dtype=np.int64) - int(qb[1]), float(qb[0]) / float(qy[0])))
    return _requant_out(v, act, qy[0], qy[1], alpha)


def _qp(desc, where):
    q = desc.get("quant")
    if not q:
        raise ValueError("%s: int8 graph needs quant {scale, zero_point}" % where)
    return float(q["scale"]), int(q["zero_point"])


def run_quantized_graph(graph, consts, inputs, keep=False):
    """Execute an int8 subgraph: Q at the inputs, integer composites, DQ at
    the outputs.  Returns float32 outputs (bf16-declared outputs are the
    float32 values; rounding them is the caller's business) and, with
    ``keep=True``, the dict of codes of every value."""
    g = load_graph(graph)
    codes, qps = {}, {}
    for desc, arr in zip(g["inputs"], inputs):
        qp = _qp(desc, "input " + desc["name"])
        a = np.asarray(arr)
        if list(a.shape) != list(desc["shape"]):
            raise ValueError("input %s: shape %s != %s" % (desc["name"], a.shape, desc["shape"]))
        codes[desc["name"]] = quantize(a.astype(np.float32), *qp)
        qps[desc["name"]] = qp
    cvals = {c["name"]: np.asarray(consts[c["index"]], dtype=np.float64) for c in g.get("constants", [])}
    for node in g["nodes"]:
        if node.get("out_dtype") != "int8":
            raise ValueError("node %s: not an int8 node" % node["name"])
        op, has_bias, has_add, act = parse_composite(node["composite"])
        attrs = node.get("attrs", {})
        alpha = float(attrs.get("alpha", 0.1))
        ins = node["inputs"]
        if op == "max_pool2d" and not node.get("quant"):
            qy = qps[ins[0]]  # a max pool keeps its input's scale and zero point
        else:
            qy = _qp(node, "node " + node["name"])
        if op in ("conv2d", "dense"):
            x, w = ins[0], cvals[ins[1]]
            i = 2
            b = None
            if has_bias:
                b = cvals[ins[i]]
                i += 1
            r = qr = None
            if has_add:
                r, qr = codes[ins[i]], qps[ins[i]]
            if op == "conv2d":
                groups = int(attrs.get("groups", 1))
                if groups != 1 and not (groups == w.shape[0] and w.shape[1] == 1):
                    raise ValueError("node %s: grouped conv other than depthwise has no int8 form" % node["name"])
                y = qconv(codes[x], qps[x], w, b, attrs, qy, act, r, qr, alpha)
            else:
                y = qdense(codes[x], qps[x], w, b, qy, act, r, qr, alpha)
        elif op == "max_pool2d":
            if qps[ins[0]] != qy:
                raise ValueError("node %s: max pool keeps its input's scale and zero point" % node["name"])
            y = qmax_pool2d(codes[ins[0]], attrs)
        elif op == "global_avg_pool2d":
            y = qglobal_avg_pool2d(codes[ins[0]], qps[ins[0]], qy)
        else:
            y = qadd(codes[ins[0]], qps[ins[0]], codes[ins[1]], qps[ins[1]], qy, act, alpha)
        codes[node["name"]] = y
        qps[node["name"]] = qy
    outs = [dequantize(codes[o["name"]], *qps[o["name"]]) for o in g["outputs"]]
    if keep:
        return outs, codes
    return outs
