"""Pins of the oracle's bf16 decoding and single RNE rounding: PyTorch's
binary32 -> bf16 conversion on exact binary32 inputs (midpoints included),
exact rational rounding on fp64 inputs, and exhaustive decoding."""
from fractions import Fraction

import numpy as np
import torch

from oracle import bf16_to_f64, f64_to_bf16_rne, bf16_ulp


def _torch_bits(x_f32):
    t = torch.from_numpy(np.asarray(x_f32, dtype=np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def test_decode_all_patterns():
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    via_torch = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()
    got = bf16_to_f64(bits)
    same = (got == via_torch) | (np.isnan(got) & np.isnan(via_torch))
    assert same.all()


def test_round_trip_all_finite_patterns():
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    x = bf16_to_f64(bits)
    fin = np.isfinite(x)
    np.testing.assert_array_equal(f64_to_bf16_rne(x[fin]), bits[fin])


def test_matches_torch_on_binary32_inputs():
    rng = np.random.default_rng(0)
    x = np.concatenate([
        rng.standard_normal(200000).astype(np.float32) * np.float32(0.02),
        rng.standard_normal(50000).astype(np.float32) * np.float32(1e30),
        rng.standard_normal(50000).astype(np.float32) * np.float32(1e-39),   # subnormals
        rng.integers(0, 1 << 32, size=100000, dtype=np.uint64).astype(np.uint32).view(np.float32),
    ])
    x = x[np.isfinite(x)]
    np.testing.assert_array_equal(f64_to_bf16_rne(x.astype(np.float64)), _torch_bits(x))


def test_midpoints_round_to_even():
    bits = np.arange(0, 0x7F7F, dtype=np.uint32)          # positive finite, below max
    lo = bits << np.uint32(16)
    mid = (lo | np.uint32(0x8000)).view(np.float32)          # exact midpoint in binary32
    got = f64_to_bf16_rne(mid.astype(np.float64))
    np.testing.assert_array_equal(got, _torch_bits(mid))
    even = (bits & 1) == 0
    np.testing.assert_array_equal(got[even], bits[even].astype(np.uint16))
    np.testing.assert_array_equal(got[~even], (bits[~even] + 1).astype(np.uint16))
    got_neg = f64_to_bf16_rne(-mid.astype(np.float64))
    np.testing.assert_array_equal(got_neg, got | np.uint16(0x8000))


def _exact_round(x):
    """Round a fp64 value to the bf16 grid with exact rational arithmetic."""
    f = Fraction(x)
    if f == 0:
        return 0.0
    a = abs(f)
    e = 0
    while a >= 2:
        a /= 2
        e += 1
    while a < 1:
        a *= 2
        e -= 1
    e = max(e, -126)
    q = Fraction(2) ** (e - 7)
    n = abs(f) / q
    fl = n.numerator // n.denominator
    rem = n - fl
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and fl % 2 == 1):
        fl += 1
    v = float(fl * q)
    return v if f > 0 else -v


def test_single_rounding_of_fp64_inputs():
    rng = np.random.default_rng(1)
    x = rng.standard_normal(3000) * 0.02
    # values just off a binary32 midpoint, where a binary32 step first would
    # round the wrong way (double rounding)
    base = bf16_to_f64(rng.integers(0x3A00, 0x3D00, size=1000).astype(np.uint16))
    near = base + bf16_ulp(base) * (0.5 - 2.0 ** -30)
    x = np.concatenate([x, near, -near])
    got = bf16_to_f64(f64_to_bf16_rne(x))
    expect = np.array([_exact_round(float(v)) for v in x])
    np.testing.assert_array_equal(got, expect)
    # and those near-midpoint values do differ from binary32-then-bf16
    two_step = bf16_to_f64(_torch_bits(near.astype(np.float32)))
    assert np.any(two_step != bf16_to_f64(f64_to_bf16_rne(near)))


def test_specials_and_ulp():
    assert f64_to_bf16_rne(np.inf)[0] == 0x7F80
    assert f64_to_bf16_rne(-np.inf)[0] == 0xFF80
    assert f64_to_bf16_rne(np.nan)[0] == 0x7FC0
    assert f64_to_bf16_rne(3.5e38)[0] == 0x7F80              # rounds past max finite
    assert f64_to_bf16_rne(-0.0)[0] == 0x8000
    assert f64_to_bf16_rne(-1e-50)[0] == 0x8000
    assert bf16_ulp(1.0) == 2.0 ** -7
    assert bf16_ulp(0.02) == 2.0 ** -13
    assert bf16_ulp(0.0) == 2.0 ** -133
