"""Operator definitions in float64, op by op, unfused.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper's composite functions are built from Relay operators that it names
but does not define (nn.conv2d, nn.bias_add, nn.relu in the pattern of
Sec. 3.1.1; Dense is the other MAC operator of the TensorRT case study,
Sec. 4.1).  The definitions below are the standard ones:

conv2d     y[n,k,p,q] = sum_{c<C/G, r<R, s<S} xpad[n, g*C/G + c, p*sh + r, q*sw + s] * w[k,c,r,s]
           with g = k // (K/G), xpad = x zero-padded by (top, left, bottom, right),
           P = (H + top + bottom - R) // sh + 1, Q likewise; cross-correlation (no flip).
dense      y[m,n] = sum_k x[m,k] * W[n,k]
bias_add   y[:, k, ...] += b[k]
add        y = a + b (same shape)
relu       max(y, 0);  relu6 = min(max(y, 0), 6);  gelu = y * Phi(y) = y * erfc(-y / sqrt 2) / 2
max_pool2d max over the in-bounds part of each window (padding acts as -inf)
global_avg_pool2d   y[n,c] = mean over h, w of x[n,c,h,w]

Layouts are the external ones: activations NCHW (or [M, K] row-major for
dense), conv weights OIHW, dense weights [out, in].
"""

import numpy as np
from scipy.special import erfc


def _f64(a):
    return np.asarray(a, dtype=np.float64)


def conv_output_size(h, r, stride, pad_before, pad_after):
    """Output extent of a convolution or pooling window along one axis."""
    return (h + pad_before + pad_after - r) // stride + 1


def conv2d(x, w, strides=(1, 1), padding=(0, 0, 0, 0), groups=1):
    """Grouped 2-D cross-correlation, NCHW input, OIHW weights.

    The sum over the R*S taps is an explicit loop; the sum over input
    channels of a group at one tap is a matrix product.
    """
    x = _f64(x)
    w = _f64(w)
    n, c, h, wd = x.shape
    k, cg, r, s = w.shape
    if c % groups or k % groups or cg != c // groups:
        raise ValueError("conv2d: channel counts do not match groups")
    sh, sw = strides
    pt, pl, pb, pr = padding
    p = conv_output_size(h, r, sh, pt, pb)
    q = conv_output_size(wd, s, sw, pl, pr)
    xp = np.zeros((n, c, h + pt + pb, wd + pl + pr), dtype=np.float64)
    xp[:, :, pt:pt + h, pl:pl + wd] = x
    y = np.zeros((n, k, p, q), dtype=np.float64)
    kg = k // groups
    for ri in range(r):
        for si in range(s):
            # window of input pixels seen by tap (ri, si): [n, c, p, q]
            win = xp[:, :, ri:ri + sh * (p - 1) + 1:sh, si:si + sw * (q - 1) + 1:sw]
            if cg == 1 and kg == 1:
                # depthwise: one input channel per output channel
                y += win * w[:, 0, ri, si].reshape(1, k, 1, 1)
                continue
            for g in range(groups):
                # sum over the group's input channels: [n, p, q, kg] -> [n, kg, p, q]
                t = np.tensordot(win[:, g * cg:(g + 1) * cg], w[g * kg:(g + 1) * kg, :, ri, si],
                                 axes=([1], [1]))
                y[:, g * kg:(g + 1) * kg] += t.transpose(0, 3, 1, 2)
    return y


def dense(x, w):
    """y = x W^T for x [M, K] and W [N, K]."""
    return _f64(x) @ _f64(w).T


def bias_add(y, b):
    """Add b[k] along axis 1 (the channel / feature axis)."""
    y = _f64(y)
    b = _f64(b)
    shape = [1] * y.ndim
    shape[1] = b.shape[0]
    return y + b.reshape(shape)


def add(a, b):
    a = _f64(a)
    b = _f64(b)
    if a.shape != b.shape:
        raise ValueError("add: shapes differ")
    return a + b


def relu(y):
    return np.maximum(_f64(y), 0.0)


def relu6(y):
    return np.minimum(np.maximum(_f64(y), 0.0), 6.0)


def gelu(y):
    """Exact GELU: y * Phi(y) with Phi the standard normal CDF, Phi(y) =
    erfc(-y / sqrt 2) / 2 (the same function as (1 + erf(y / sqrt 2)) / 2
    without its cancellation for y << 0, where 1 + erf loses every digit)."""
    y = _f64(y)
    return y * 0.5 * erfc(-y / np.sqrt(2.0))


def leaky_relu(y, alpha=0.1):
    """y for y >= 0, alpha * y below (0 <= alpha < 1)."""
    y = _f64(y)
    return np.where(y >= 0.0, y, float(alpha) * y)


ACTIVATIONS = {"relu": relu, "relu6": relu6, "gelu": gelu, "leaky": leaky_relu}


def max_pool2d(x, pool_size=(3, 3), strides=(2, 2), padding=(1, 1, 1, 1)):
    """Max over each window; padded positions never win (they are -inf)."""
    x = _f64(x)
    n, c, h, wd = x.shape
    r, s = pool_size
    sh, sw = strides
    pt, pl, pb, pr = padding
    p = conv_output_size(h, r, sh, pt, pb)
    q = conv_output_size(wd, s, sw, pl, pr)
    xp = np.full((n, c, h + pt + pb, wd + pl + pr), -np.inf, dtype=np.float64)
    xp[:, :, pt:pt + h, pl:pl + wd] = x
    y = np.full((n, c, p, q), -np.inf, dtype=np.float64)
    for ri in range(r):
        for si in range(s):
            y = np.maximum(y, xp[:, :, ri:ri + sh * (p - 1) + 1:sh, si:si + sw * (q - 1) + 1:sw])
    return y


def avg_pool2d(x, pool_size=(3, 3), strides=(1, 1), padding=(1, 1, 1, 1), count_include_pad=False):
    """Mean over each window.  Without count_include_pad the divisor is the
    number of window positions inside the image; with it, the full window."""
    x = _f64(x)
    n, c, h, wd = x.shape
    r, s = pool_size
    sh, sw = strides
    pt, pl, pb, pr = padding
    p = conv_output_size(h, r, sh, pt, pb)
    q = conv_output_size(wd, s, sw, pl, pr)
    xp = np.zeros((n, c, h + pt + pb, wd + pl + pr), dtype=np.float64)
    xp[:, :, pt:pt + h, pl:pl + wd] = x
    inside = np.zeros((h + pt + pb, wd + pl + pr), dtype=np.float64)
    inside[pt:pt + h, pl:pl + wd] = 1.0
    tot = np.zeros((n, c, p, q), dtype=np.float64)
    cnt = np.zeros((p, q), dtype=np.float64)
    for ri in range(r):
        for si in range(s):
            tot += xp[:, :, ri:ri + sh * (p - 1) + 1:sh, si:si + sw * (q - 1) + 1:sw]
            cnt += inside[ri:ri + sh * (p - 1) + 1:sh, si:si + sw * (q - 1) + 1:sw]
    return tot / (float(r * s) if count_include_pad else cnt)


def concatenate(xs, axis=1):
    """Join tensors along an axis (the channel axis of NCHW)."""
    return np.concatenate([_f64(x) for x in xs], axis=axis)


def global_avg_pool2d(x):
    """Mean over the spatial axes; output [N, C]."""
    x = _f64(x)
    return x.sum(axis=(2, 3)) / (x.shape[2] * x.shape[3])
