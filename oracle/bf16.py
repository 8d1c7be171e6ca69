"""bfloat16 round-to-nearest-even, computed on float64 values.

TEST INFRASTRUCTURE ONLY (see the package docstring).

A bfloat16 number has the float32 exponent range (8 exponent bits, bias 127)
and 8 significant bits (1 implicit + 7 stored).  Rounding a float64 value to
the nearest bfloat16, ties to an even last significand bit, is done here in
one step on the significand returned by ``frexp``:

    x = m * 2**e with 0.5 <= |m| < 1   ->   t = m * 2**8 in [128, 256)
    t is rounded half-to-even to an integer (NumPy's ``round``), result t * 2**(e-8).

Below the smallest normal (2**-126) the spacing is fixed at 2**-133, so the
value is rounded on that grid instead.  Results whose magnitude reaches 2**128
overflow to infinity.  NaN and infinities pass through.

This is the "partial quantization" cast at the subgraph boundary (the
fp32 -> reduced-precision cast of the TensorRT case study, Sec. 4.1) and the
storage rounding of every bf16 tensor in the declared graph.
"""

import numpy as np

_MIN_NORMAL = 2.0 ** -126
_SUB_QUANTUM = 2.0 ** -133
_OVERFLOW = 2.0 ** 128


def round_bf16(x):
    """Round float64 values to the nearest bfloat16 value (ties to even).

    Accepts any array-like; returns a float64 array whose every element is
    exactly representable in bfloat16.
    """
    x = np.asarray(x, dtype=np.float64)
    out = np.empty_like(x)
    finite = np.isfinite(x)
    out[~finite] = x[~finite]
    xf = x[finite]
    ax = np.abs(xf)
    normal = ax >= _MIN_NORMAL
    res = np.empty_like(xf)
    m, e = np.frexp(xf[normal])
    t = np.round(m * 256.0)  # half-to-even on the integer grid [128, 256]
    res[normal] = np.ldexp(t, e - 8)
    sub = ~normal
    res[sub] = np.round(xf[sub] / _SUB_QUANTUM) * _SUB_QUANTUM
    over = np.abs(res) >= _OVERFLOW
    res[over] = np.copysign(np.inf, res[over])
    out[finite] = res
    return out


def bf16_bits(x):
    """The 16-bit bfloat16 patterns of values already representable in bf16.

    Used by tests to compare bit patterns with device output.  Raises if an
    element is not exactly representable.
    """
    x = np.asarray(x, dtype=np.float64)
    f32 = x.astype(np.float32)
    if not np.array_equal(f32.astype(np.float64), x, equal_nan=True):
        raise ValueError("value not representable in float32")
    bits = f32.view(np.uint32)
    if np.any(bits & 0xFFFF):
        raise ValueError("value not representable in bfloat16")
    return (bits >> 16).astype(np.uint16)


def from_bf16_bits(bits):
    """float64 values of 16-bit bfloat16 patterns."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return b.view(np.float32).astype(np.float64)
