"""ES on int8 parameters with per-row scales (oracle; test-only).

The paper leaves quantized ES to future work (Appendix A.2, the paragraph on
quantized ES optimization): perturbing quantized weights needs noise that knows the
quantization scale, numerically stable updates, and perturbations that can
still be replayed from a seed.  This is the library's reading of that
direction, for symmetric int8 codes:

  theta_j = s_r(j) * q_j,  q_j in [-127, 127],  r(j) = j div row
  (row = 0: one scale for the whole tensor), s_r binary32.

Perturbation in quantum units.  The real perturbation sign * sigma * eps_j is
expressed in units of its row's quantum, d_j = sign * sigma * eps_j / s_r(j),
and rounded stochastically to an integer offset with a 9-bit draw r_j:

  k_j = floor(d_j + (2 r_j + 1) * 2^-10),   |E[k_j] - d_j| <= 2^-10
  q_j <- clamp(q_j + k_j, -127, 127)

eps_j is the perturbation noise of the bf16 path (domain 0 under the member
seed) and r_j the spare top 9 bits of element j's own noise word (see the
noise module), so the rounding costs no generator calls.  Because k_j is
regenerated bit-for-bit from the seed, the revert q_j <- clamp(q_j - k_j)
returns the exact code wherever the perturbation was not clamped: seed replay
is exact in integers, with no drift.

Update in quantum units: delta_j = sum_d w_d eps_j(seed_d) / s_r(j) with the
merged weights of the bf16 update, k_j = floor(delta_j + r_j * 2^-16) with a
16-bit r_j from domain 1 under the update's rounding seed (E[k_j] = delta_j to
the 2^-16 grid), q_j <- clamp(q_j + k_j).  The
rounding is always stochastic: the paper's update steps are a fraction of a
quantum, and rounding to nearest would drop nearly all of them.

Elements whose row scale is not a normal positive finite binary32 value
(2^-126 <= s < infinity) are left unchanged.

Pins (tests/test_oracle_quant.py): the mean of k over all 65536 16-bit draws
equals d exactly for d on the 2^-16 grid, and over all 512 9-bit draws lies
within 2^-10 of d; every revert of an unclamped perturbation is
exact; the variance of the offsets against the closed form
(sigma/s)^2 + 1/6; a per-element pure-Python rendering (big-integer Philox,
math.log / math.cos, explicit row lookup) agrees with the vectorised one; the
update's mean step against delta within its standard error; identities.
"""

import numpy as np

from .noise import normals, rounding_draws, spare_draws, DOMAIN_ROUNDING
from .es import zscore, update_coefficient, member_weights, ES_REWARDS_ARE_WEIGHTS

QMAX = 127


def _f32(x):
    return float(np.float32(x))


def row_scales(scales, row, elems):
    """The scale of each listed element (fp64): scales[j div row], or
    scales[0] for every element when row == 0."""
    scales = np.asarray(scales, dtype=np.float32).astype(np.float64)
    elems = np.asarray(elems, dtype=np.uint64)
    if row == 0:
        return np.full(elems.shape, scales[0])
    return scales[(elems // np.uint64(row)).astype(np.int64)]


def offset_values(scales, row, seed, tensor_id, sign, sigma, elems):
    """d_j = sign sigma eps_j / s_r(j) (fp64), the 9-bit draws r_j and the
    validity of each element's scale; the offset is round_offset9(d, r)."""
    el = np.asarray(elems, dtype=np.uint64)
    s = row_scales(scales, row, el)
    ok = np.isfinite(s) & (s >= 2.0 ** -126)
    d = sign * _f32(sigma) * normals(seed, tensor_id, el) / np.where(ok, s, 1.0)
    return np.where(ok, d, 0.0), spare_draws(seed, tensor_id, el), ok


def round_offset9(d, r9):
    """k = floor(d + (2 r + 1) 2^-10): d rounded to an integer stochastically
    with the 9-bit draw r (fp64 d, integer r in [0, 511])."""
    r = np.asarray(r9, dtype=np.int64)
    if np.any((r < 0) | (r > 511)):
        raise ValueError("draws must be 9-bit integers")
    return np.floor(np.asarray(d, dtype=np.float64) + (2 * r + 1) * 2.0 ** -10).astype(np.int64)


def round_offset(d, r16):
    """k = floor(d + r 2^-16): d rounded to an integer stochastically with
    the 16-bit draw r (fp64 d, integer r in [0, 65535])."""
    r = np.asarray(r16, dtype=np.int64)
    if np.any((r < 0) | (r > 0xFFFF)):
        raise ValueError("draws must be 16-bit integers")
    return np.floor(np.asarray(d, dtype=np.float64) + r * 2.0 ** -16).astype(np.int64)


def _apply(q, k, ok):
    q = np.asarray(q, dtype=np.int8).astype(np.int64)
    out = np.where(ok, np.clip(q + k, -QMAX, QMAX), q)
    return out.astype(np.int8)


def qperturb(q, scales, row, seed, tensor_id, sign, sigma, elems=None):
    """q' = clamp(q + floor(sign sigma eps / s + (2 r + 1) 2^-10), -127, 127)."""
    if sign not in (1, -1):
        raise ValueError("sign must be +1 or -1")
    q = np.asarray(q, dtype=np.int8).ravel()
    if _f32(sigma) == 0.0:
        return q.copy()
    el = np.arange(q.size, dtype=np.uint64) if elems is None else np.asarray(elems, np.uint64)
    d, r, ok = offset_values(scales, row, seed, tensor_id, sign, sigma, el)
    return _apply(q, round_offset9(d, r), ok)


def qrestore(q, scales, row, seed, tensor_id, sign, sigma, elems=None):
    """Subtract the offsets qperturb added: q' = clamp(q - k, -127, 127)."""
    if sign not in (1, -1):
        raise ValueError("sign must be +1 or -1")
    q = np.asarray(q, dtype=np.int8).ravel()
    if _f32(sigma) == 0.0:
        return q.copy()
    el = np.arange(q.size, dtype=np.uint64) if elems is None else np.asarray(elems, np.uint64)
    d, r, ok = offset_values(scales, row, seed, tensor_id, sign, sigma, el)
    return _apply(q, -round_offset9(d, r), ok)


def update_values(scales, row, tensor_id, seeds, signs, rewards, alpha, sigma, flags=0,
                  zscore_eps=1e-8, elems=None, round_seed=0, n=None):
    """delta_j = sum_d w_d eps_j(seed_d) / s_r(j) (fp64), the draws r_j, the
    validity of each scale, the live (seed, weight) pairs and the status."""
    if flags & ES_REWARDS_ARE_WEIGHTS:
        z = np.asarray(rewards, dtype=np.float32).astype(np.float64)
        status = 0 if np.all(np.isfinite(z)) else 1
    else:
        z, status = zscore(rewards, zscore_eps)
    el = np.arange(n, dtype=np.uint64) if elems is None else np.asarray(elems, np.uint64)
    if status:
        return None, None, None, [], status
    c = update_coefficient(alpha, sigma, len(seeds), flags)
    distinct, w = member_weights([int(x) for x in seeds], [int(x) for x in signs], z, c)
    live = [(sd, wd) for sd, wd in zip(distinct, w) if wd != 0.0]
    s = row_scales(scales, row, el)
    ok = np.isfinite(s) & (s >= 2.0 ** -126)
    delta = np.zeros(el.size)
    for sd, wd in live:
        delta += wd * normals(sd, tensor_id, el)
    d = np.where(ok, delta / np.where(ok, s, 1.0), 0.0)
    return d, rounding_draws(round_seed, tensor_id, el, DOMAIN_ROUNDING), ok, live, 0


def qupdate(q, scales, row, tensor_id, seeds, signs, rewards, alpha, sigma, flags=0,
            zscore_eps=1e-8, elems=None, round_seed=0):
    """q' = clamp(q + floor(sum_d w_d eps_d / s + r 2^-16), -127, 127), the
    draws r from domain 1 under round_seed.  Returns (codes, status); a
    non-finite reward or no nonzero weight leaves q unchanged."""
    if len(seeds) == 0 or len(seeds) != len(signs) or len(seeds) != len(rewards):
        raise ValueError("seeds, signs and rewards must have the same nonzero length")
    if any(int(x) not in (1, -1) for x in signs):
        raise ValueError("signs must be +1 or -1")
    q = np.asarray(q, dtype=np.int8).ravel()
    d, r, ok, live, status = update_values(scales, row, tensor_id, seeds, signs, rewards, alpha,
                                           sigma, flags, zscore_eps, elems, round_seed, n=q.size)
    if status or not live:
        return q.copy(), status
    return _apply(q, round_offset(d, r), ok), 0
