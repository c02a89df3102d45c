"""bfloat16 decoding and single round-to-nearest-even encoding (oracle; test-only).

The paper never states the parameter dtype; its memory figures (8.41 GB for a
4B model, 51.75 GB for 27B, Table of Sudoku results and Section 4) imply 16-bit
weights, and this library stores them as bfloat16.  A bf16 value is the top 16
bits of a binary32: 1 sign bit, 8 exponent bits (bias 127), 7 fraction bits.

f64_to_bf16_rne rounds an fp64 value straight to the bf16 grid, once, ties to
even, with no intermediate binary32 rounding: the spacing of bf16 values in the
binade [2^e, 2^(e+1)) is 2^(e-7), floored at the subnormal spacing 2^-133, and
values that round to 2^128 or beyond become infinity.

Pins (tests/test_oracle_bf16.py): agreement with PyTorch's binary32 -> bf16
conversion (itself round-to-nearest-even) on inputs that are exact binary32
values, including every bf16 midpoint; exact rational rounding (Python
fractions) on fp64 inputs that are not binary32 values; exhaustive decoding of
all 65536 bit patterns.
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
