"""Pins of the oracle's bfloat16 rounding (round to nearest, ties to even).

Against two independent references: torch's CPU float32 -> bfloat16
conversion (a library routine), and exact rational arithmetic choosing the
nearest of the two neighbouring bfloat16 values by brute force.
"""

from fractions import Fraction

import numpy as np
import pytest
import torch

from oracle.bf16 import bf16_bits, from_bf16_bits, round_bf16


def _torch_bf16(x32):
    t = torch.from_numpy(np.ascontiguousarray(x32, dtype=np.float32))
    return t.to(torch.bfloat16).to(torch.float64).numpy()


def _nearest_bf16_exact(v):
    """Nearest bfloat16 to the float64 v by exact rational comparison."""
    if v == 0.0:
        return v
    # neighbours: truncate the float32 nearest below/above to bf16 grid
    f = Fraction(v)
    a = abs(v)
    e = int(np.floor(np.log2(a)))
    e = max(e, -126)
    quantum = Fraction(2) ** (e - 7)
    lo = (abs(f) // quantum) * quantum
    hi = lo + quantum
    dlo = abs(f) - lo
    dhi = hi - abs(f)
    if dlo < dhi:
        r = lo
    elif dhi < dlo:
        r = hi
    else:
        r = lo if (lo / quantum) % 2 == 0 else hi
    r = float(r)
    if r >= 2.0 ** 128:
        r = np.inf
    return r if v > 0 else -r


def test_matches_torch_on_random_float32():
    rng = np.random.default_rng(0)
    bits = rng.integers(0, 2 ** 32, size=1_000_000, dtype=np.uint64).astype(np.uint32)
    x = bits.view(np.float32)
    x = x[np.isfinite(x)]
    ours = round_bf16(x.astype(np.float64))
    ref = _torch_bf16(x)
    assert np.array_equal(ours, ref)


def test_ties_go_to_even():
    # bf16 values 1 + k/128; midpoints 1 + (2k+1)/256 are exact float32 ties
    k = np.arange(0, 128)
    mid = 1.0 + (2 * k + 1) / 256.0
    got = round_bf16(mid)
    even = np.where(k % 2 == 0, 1.0 + k / 128.0, 1.0 + (k + 1) / 128.0)
    assert np.array_equal(got, even)
    assert np.array_equal(got, _torch_bf16(mid.astype(np.float32)))


def test_special_values():
    maxf = float(np.frombuffer(np.uint32(0x7F7FFFFF).tobytes(), np.float32)[0])
    max_bf16 = float(from_bf16_bits(0x7F7F))
    vals = np.array([0.0, -0.0, np.inf, -np.inf, maxf, -maxf, max_bf16, 2.0 ** -126,
                     2.0 ** -133, 2.0 ** -134, 3 * 2.0 ** -135, 1e-45, 5e-39])
    got = round_bf16(vals)
    ref = _torch_bf16(vals.astype(np.float32))
    assert np.array_equal(got, ref)
    assert np.isnan(round_bf16(np.array([np.nan]))[0])


def test_no_double_rounding_from_float64():
    # just above a bf16 tie by less than half a float32 ulp: a float32 detour
    # would land on the tie and round to even (down); the direct rounding
    # must go up.
    k = np.arange(0, 128, 2)
    tie = 1.0 + (2 * k + 1) / 256.0
    x = tie + 2.0 ** -30
    assert np.all(x.astype(np.float32).astype(np.float64) == tie)
    got = round_bf16(x)
    assert np.array_equal(got, 1.0 + (k + 1) / 128.0)


def test_brute_force_rationals():
    rng = np.random.default_rng(1)
    x = rng.standard_normal(3000) * np.exp(rng.uniform(-40, 40, size=3000))
    x = np.concatenate([x, rng.uniform(-1, 1, 500) * 2.0 ** -128])
    got = round_bf16(x)
    ref = np.array([_nearest_bf16_exact(v) for v in x])
    assert np.array_equal(got, ref)


def test_bits_roundtrip():
    v = round_bf16(np.array([1.0, -2.5, 3.140625, 65280.0]))
    b = bf16_bits(v)
    assert list(b) == [0x3F80, 0xC020, 0x4049, 0x477F]
    assert np.array_equal(from_bf16_bits(b), v)
    with pytest.raises(ValueError):
        bf16_bits(np.array([1.0 + 2.0 ** -10]))
