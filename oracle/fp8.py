"""ES on fp8 (OCP E4M3) parameters with per-row scales (oracle; test-only).

The paper leaves quantized ES to future work (Appendix A.2, the paragraph on
quantized ES optimization): noise that knows the quantization scale,
numerically stable updates, and perturbations that seed replay can undo.
This is the library's reading for 8-bit floating-point codes, next to the
int8 one in quant.py:

  theta_j = s_r(j) * v(c_j),  c_j an E4M3 code,  r(j) = j div row
  (row = 0: one scale for the whole tensor), s_r binary32.

E4M3 (the OCP 8-bit floating-point format with 4 exponent and 3 mantissa
bits, bias 7, no infinities): code bits s eeee mmm;
  e = 0:           v = (-1)^s * m/8 * 2^-6          (zero and subnormals)
  1 <= e <= 15:    v = (-1)^s * (1 + m/8) * 2^(e-7)
  e = 15, m = 7:   not a number (codes 0x7F and 0xFF)
so the finite values are a grid G, symmetric about zero, uniform with spacing
2^-9 on [-2^-5, 2^-5] and with spacing 2^(k-3) on each binade [2^k, 2^(k+1)),
up to the largest value 448.

A pass forms x, the code's value in scale units plus a step, rounds x to
binary32 (the precision the kernels compute in), and rounds it onto G:

  lo = the largest point of G <= x,  h = the distance to the next point,
  f  = (x - lo) / h in [0, 1)
  result = lo + h * [step],  then clamped to [-448, 448]

(x >= 448 gives 448 and x <= -448 gives -448.)  The step condition is the
int8 path's integer rounding moved onto G:

  perturb:  x = v(c) + d,  d = sign sigma eps_j / s,  step iff f >= 1 - u
  restore:  y = v(c) - d,                             step iff f >  u
  update:   x = v(c) + sum_d w_d eps_j(seed_d) / s,   step iff f >= 1 - r 2^-16

with u = (2 r9 + 1) 2^-10 from the spare top 9 bits r9 of element j's own
noise word (as the int8 perturbation; no extra generator call) and r the
16-bit update draw of domain 1 under the rounding seed.  E[result] = x to
within 2^-10 h for a perturbation and to the 2^-16 h grid for an update: the
noise and the update are unbiased at any scale, and an update far smaller
than the local spacing still moves the codes in expectation.

Restore undoes perturb exactly wherever x, the perturbed value and y lie in
one uniform stretch of G (the same binade, or the band around zero): there
lo = n h with n an integer, f = frac(n + d/h) and the restore's fraction is
1 - f, so the two conditions are complementary; the binary32 rounding of x
and y is at the same position with round-to-nearest-even, which is
symmetric, so it keeps them complementary.  A perturbation that carries a
value into a coarser binade maps two codes onto one, which no in-place revert
can undo; such a revert (and one whose perturbation clamped at 448) is off by
at most one step of the coarser grid it touched, measured and reported
rather than hidden (about 5 % of N(0, 0.02) weights per perturb-restore
cycle at sigma = 1e-3, most of them near zero, where the perturbation spans
many binades).

Codes that are not a number, and elements whose row scale is not a normal
positive finite binary32 value, are left unchanged.  A zero result is +0
(code 0x00), so -0 (0x80) becomes +0 once a pass moves through it.

Pins (tests/test_oracle_fp8.py): the decoder against a separately written
enumeration of the format with exact fractions and against PyTorch's
float8_e4m3fn conversion; the grid floor against a brute-force scan;
enumeration of all 512 perturbation draws and all 65536 update draws (mean
within 2^-10 h of x, and exactly x on the 2^-16 h grid); exact revert inside
every binade and the band around zero for every code; an element-by-element
pure-Python rendering (big-integer Philox, math functions, explicit grid
search) equal to the vectorised one; unbiased updates and a 70-update
trajectory that tracks the unrounded sum; identities (sigma = 0, equal
rewards, non-finite rewards, invalid scales, not-a-number codes, clamping).
"""

import numpy as np

from .noise import normals, rounding_draws, spare_draws, DOMAIN_ROUNDING
from .es import zscore, update_coefficient, member_weights, ES_REWARDS_ARE_WEIGHTS
from .quant import row_scales

E4M3_MAX = 448.0
NAN_CODES = (0x7F, 0xFF)


def e4m3_decode(codes):
    """Values of E4M3 codes (fp64; NaN for the not-a-number codes)."""
    b = np.asarray(codes).astype(np.int64) & 0xFF
    s = np.where(b >> 7, -1.0, 1.0)
    e = (b >> 3) & 0xF
    m = (b & 7).astype(np.float64)
    sub = m / 8.0 * 2.0 ** -6
    norm = (1.0 + m / 8.0) * np.exp2(e.astype(np.float64) - 7.0)
    v = s * np.where(e == 0, sub, norm)
    return np.where((e == 15) & ((b & 7) == 7), np.nan, v)


def _grid():
    v = e4m3_decode(np.arange(256))
    return np.unique(v[np.isfinite(v)])       # 253 values, -448 .. 448


GRID = _grid()


def grid_floor(x):
    """(lo, h): the largest grid value <= x and the distance to the next one,
    for x in [-448, 448) (fp64 arrays)."""
    x = np.asarray(x, dtype=np.float64)
    i = np.searchsorted(GRID, x, side="right") - 1
    if np.any((i < 0) | (i >= GRID.size - 1)):
        raise ValueError("grid_floor needs -448 <= x < 448")
    return GRID[i], GRID[i + 1] - GRID[i]


def _grid_codes():
    """The code of each GRID value (the +0 code for zero)."""
    vals = e4m3_decode(np.arange(256))
    out = np.empty(GRID.size, dtype=np.uint8)
    for i, g in enumerate(GRID):
        hits = [c for c in range(256) if vals[c] == g and (g != 0.0 or c == 0)]
        out[i] = hits[0]
    return out


GRID_CODES = _grid_codes()


def e4m3_encode(v):
    """Codes of grid values (exact; zero encodes as +0).  Raises for a value
    that is not on the grid."""
    v = np.asarray(v, dtype=np.float64)
    i = np.clip(np.searchsorted(GRID, v), 0, GRID.size - 1)
    if not np.all(GRID[i] == v):
        raise ValueError("e4m3_encode: value not on the E4M3 grid")
    return GRID_CODES[i]


def _f32(x):
    return np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64)


def round_onto_grid(x32, rule, draw):
    """Round binary32 values x32 (given as fp64) onto the grid with `rule`:
    'perturb' steps iff f >= 1 - u (u = draw, the offset (2 r + 1) 2^-10),
    'restore' iff f > u, 'update' iff f >= 1 - u (u = r 2^-16); clamped to
    [-448, 448].  Returns fp64 grid values."""
    x = np.asarray(x32, dtype=np.float64)
    u = np.asarray(draw, dtype=np.float64)
    top = x >= E4M3_MAX
    bottom = x <= -E4M3_MAX
    xc = np.clip(x, -E4M3_MAX, np.nextafter(E4M3_MAX, 0.0))
    lo, h = grid_floor(xc)
    f = (xc - lo) / h
    step = (f > u) if rule == "restore" else (f >= 1.0 - u)
    out = lo + np.where(step, h, 0.0)
    out = np.where(top, E4M3_MAX, np.where(bottom, -E4M3_MAX, out))
    return out + 0.0                          # -0.0 -> +0.0


def perturb_values(codes, scales, row, seed, tensor_id, sign, sigma, elems):
    """(v, d, u, ok): code values, steps d_j = sign sigma eps_j / s (fp64),
    the perturbation offsets u_j = (2 r9 + 1) 2^-10, and which elements may
    change (finite code, valid scale)."""
    el = np.asarray(elems, dtype=np.uint64)
    v = e4m3_decode(codes)
    s = row_scales(scales, row, el)
    ok = np.isfinite(s) & (s >= 2.0 ** -126) & np.isfinite(v)
    d = sign * float(np.float32(sigma)) * normals(seed, tensor_id, el) / np.where(ok, s, 1.0)
    u = (2 * spare_draws(seed, tensor_id, el).astype(np.float64) + 1) * 2.0 ** -10
    return np.where(ok, v, 0.0), np.where(ok, d, 0.0), u, ok


def _pass(codes, values, ok):
    c = np.asarray(codes, dtype=np.uint8).ravel()
    return np.where(ok, e4m3_encode(np.where(ok, values, 0.0)), c).astype(np.uint8)


def f8perturb(codes, scales, row, seed, tensor_id, sign, sigma, elems=None):
    """c' = E4M3 code of round_onto_grid(f32(v(c) + sign sigma eps / s), 'perturb', u)."""
    if sign not in (1, -1):
        raise ValueError("sign must be +1 or -1")
    c = np.asarray(codes, dtype=np.uint8).ravel()
    if float(np.float32(sigma)) == 0.0:
        return c.copy()
    el = np.arange(c.size, dtype=np.uint64) if elems is None else np.asarray(elems, np.uint64)
    v, d, u, ok = perturb_values(c, scales, row, seed, tensor_id, sign, sigma, el)
    return _pass(c, round_onto_grid(_f32(v + d), "perturb", u), ok)


def f8restore(codes, scales, row, seed, tensor_id, sign, sigma, elems=None):
    """c' = E4M3 code of round_onto_grid(f32(v(c) - sign sigma eps / s), 'restore', u)."""
    if sign not in (1, -1):
        raise ValueError("sign must be +1 or -1")
    c = np.asarray(codes, dtype=np.uint8).ravel()
    if float(np.float32(sigma)) == 0.0:
        return c.copy()
    el = np.arange(c.size, dtype=np.uint64) if elems is None else np.asarray(elems, np.uint64)
    v, d, u, ok = perturb_values(c, scales, row, seed, tensor_id, sign, sigma, el)
    return _pass(c, round_onto_grid(_f32(v - d), "restore", u), ok)


def f8update_values(codes, scales, row, tensor_id, seeds, signs, rewards, alpha, sigma,
                    flags=0, zscore_eps=1e-8, elems=None, round_seed=0):
    """(v, delta, u, ok, live, status): code values, the update's step in scale
    units delta_j = sum_d w_d eps_j(seed_d) / s (fp64), the draws as offsets
    u = r 2^-16, the elements that may change, the live (seed, weight) pairs
    and the status."""
    if flags & ES_REWARDS_ARE_WEIGHTS:
        z = np.asarray(rewards, dtype=np.float32).astype(np.float64)
        status = 0 if np.all(np.isfinite(z)) else 1
    else:
        z, status = zscore(rewards, zscore_eps)
    c = np.asarray(codes, dtype=np.uint8).ravel()
    el = np.arange(c.size, dtype=np.uint64) if elems is None else np.asarray(elems, np.uint64)
    if status:
        return None, None, None, None, [], status
    coef = update_coefficient(alpha, sigma, len(seeds), flags)
    distinct, w = member_weights([int(x) for x in seeds], [int(x) for x in signs], z, coef)
    live = [(sd, wd) for sd, wd in zip(distinct, w) if wd != 0.0]
    v = e4m3_decode(c)
    s = row_scales(scales, row, el)
    ok = np.isfinite(s) & (s >= 2.0 ** -126) & np.isfinite(v)
    delta = np.zeros(el.size)
    for sd, wd in live:
        delta += wd * normals(sd, tensor_id, el)
    delta = np.where(ok, delta / np.where(ok, s, 1.0), 0.0)
    u = rounding_draws(round_seed, tensor_id, el, DOMAIN_ROUNDING).astype(np.float64) * 2.0 ** -16
    return np.where(ok, v, 0.0), delta, u, ok, live, 0


def f8update(codes, scales, row, tensor_id, seeds, signs, rewards, alpha, sigma, flags=0,
             zscore_eps=1e-8, elems=None, round_seed=0):
    """c' = E4M3 code of round_onto_grid(f32(v(c) + sum_d w_d eps_d / s),
    'update', r 2^-16).  Returns (codes, status); a non-finite reward or no
    nonzero weight leaves the codes unchanged."""
    if len(seeds) == 0 or len(seeds) != len(signs) or len(seeds) != len(rewards):
        raise ValueError("seeds, signs and rewards must have the same nonzero length")
    if any(int(x) not in (1, -1) for x in signs):
        raise ValueError("signs must be +1 or -1")
    c = np.asarray(codes, dtype=np.uint8).ravel()
    v, delta, u, ok, live, status = f8update_values(c, scales, row, tensor_id, seeds, signs,
                                                    rewards, alpha, sigma, flags, zscore_eps,
                                                    elems, round_seed)
    if status or not live:
        return c.copy(), status
    return _pass(c, round_onto_grid(_f32(v + delta), "update", u), ok), 0
