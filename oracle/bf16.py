"""bfloat16 decoding and single round-to-nearest-even encoding (oracle; test-only).

The paper never states the parameter dtype; its memory figures (8.41 GB for a
4B model, 51.75 GB for 27B, Table of Sudoku results and Section 4) imply 16-bit
weights, and this library stores them as bfloat16.  A bf16 value is the top 16
bits of a binary32: 1 sign bit, 8 exponent bits (bias 127), 7 fraction bits.

f64_to_bf16_rne rounds an fp64 value straight to the bf16 grid, once, ties to
even, with no intermediate binary32 rounding: the spacing of bf16 values in the
binade [2^e, 2^(e+1)) is 2^(e-7), floored at the subnormal spacing 2^-133, and
values that round to 2^128 or beyond become infinity.

f64_to_bf16_sr is the optional stochastic rounding of the update (the paper
does not state how its updates are rounded; this mode exists because small
reward-weighted steps fall below half a bf16 spacing and round-to-nearest
drops them).  The value is first rounded to binary32 (ties to even), the
precision in which the kernels form theta + increment, so that both sides take
the rounding decision on the same binary32 number.  With lo that number
truncated toward zero onto the bf16 grid, q the bf16 spacing at lo and
f = (|x32| - |lo|) / q (a multiple of 2^-16 in [0, 1)), a 16-bit draw r moves
the result one step away from zero exactly when r / 2^16 >= 1 - f.  Over the
65536 draws the step is taken f * 2^16 times, so the expected result is x32.
A step past the largest finite bf16 gives infinity; infinities stay; NaN
becomes 0x7FC0.

Pins (tests/test_oracle_bf16.py, tests/test_oracle_rounding.py): agreement
with PyTorch's binary32 -> bf16 conversion (itself round-to-nearest-even) on
inputs that are exact binary32 values, including every bf16 midpoint; exact
rational rounding (Python fractions) on fp64 inputs that are not binary32
values; exhaustive decoding of all 65536 bit patterns; for stochastic
rounding, exhaustive enumeration of all 65536 draws (the mean is x32 exactly,
results only take the two bracketing values, truncation at r = 0) against
bit-level truncation of the binary32 pattern.
"""

import numpy as np


def bf16_to_f64(bits):
    """Decode bf16 bit patterns (uint16 array) to fp64, exactly."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    with np.errstate(invalid="ignore"):
        return b.view(np.float32).astype(np.float64)


def f64_to_bf16_rne(x):
    """Round fp64 values to bf16 (ties to even) once; returns uint16 bits."""
    x = np.atleast_1d(np.asarray(x, dtype=np.float64))
    out = np.empty(x.shape, dtype=np.uint16)
    nan = np.isnan(x)
    finite = np.isfinite(x)
    ax = np.abs(np.where(finite, x, 0.0))
    # exponent of the leading bit: ax = m 2^e with m in [0.5, 1)
    _, e = np.frexp(ax)
    lead = np.where(ax == 0, -126, np.maximum(e.astype(np.int64) - 1, -126))
    quantum = np.ldexp(1.0, (lead - 7).astype(np.int32))
    # x / quantum is exact (power-of-two scaling); np.round is half-to-even
    r = np.round(np.where(finite, x, 0.0) / quantum) * quantum
    with np.errstate(over="ignore"):
        r32 = np.where(np.abs(r) >= 2.0 ** 128, np.copysign(np.inf, r), r
                       ).astype(np.float32)
    bits = (r32.view(np.uint32) >> np.uint32(16)).astype(np.uint16)
    out[:] = bits
    inf_in = ~finite & ~nan
    out[inf_in] = np.where(x[inf_in] > 0, 0x7F80, 0xFF80).astype(np.uint16)
    out[nan] = 0x7FC0
    return out


def bf16_ulp(x):
    """Spacing of the bf16 grid at |x| (fp64): 2^(e-7) for |x| in [2^e, 2^(e+1)),
    floored at the subnormal spacing 2^-133."""
    ax = np.abs(np.asarray(x, dtype=np.float64))
    _, e = np.frexp(ax)
    lead = np.where(ax == 0, -126, np.maximum(e.astype(np.int64) - 1, -126))
    return np.ldexp(1.0, (lead - 7).astype(np.int32))


def f64_to_bf16_sr(x, r16):
    """Stochastically round fp64 values to bf16 via binary32, one 16-bit draw
    per value (r16, integers in [0, 65535]); returns uint16 bits."""
    x = np.atleast_1d(np.asarray(x, dtype=np.float64))
    r = np.broadcast_to(np.asarray(r16, dtype=np.int64), x.shape)
    if np.any((r < 0) | (r > 0xFFFF)):
        raise ValueError("draws must be 16-bit integers")
    with np.errstate(over="ignore", invalid="ignore"):
        x32 = x.astype(np.float32).astype(np.float64)
    finite = np.isfinite(x32)
    a = np.abs(np.where(finite, x32, 0.0))
    _, e = np.frexp(a)
    lead = np.where(a == 0, -126, np.maximum(e.astype(np.int64) - 1, -126))
    q = np.ldexp(1.0, (lead - 7).astype(np.int32))
    lo = np.floor(a / q) * q                  # exact: a / q has at most 24 bits
    f = (a - lo) / q                          # exact multiple of 2^-16
    away = r.astype(np.float64) / 65536.0 >= 1.0 - f
    mag = np.where(away, lo + q, lo)          # lo + q may be 2^128: infinity below
    res = np.where(finite, np.copysign(mag, x32), x32)
    return f64_to_bf16_rne(res)
