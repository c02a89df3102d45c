"""Perturb, restore, reward z-score, reward-weighted update and the sigma
schedule, in fp64 with one bf16 rounding (oracle; test-only).

Paper references (arXiv 2608.17310):
  * perturb / restore: Section 3 -- each perturbed agent is obtained by an
    in-place addition of sigma * eps_i and reverted by the matching
    subtraction, eps_i regenerated from its seed; Appendix D.6 states the
    same order: apply theta + sigma_t eps_i, evaluate, revert.
  * z-score: Section 3, zhat_i = (R_i - mu_R) / (s_R + varepsilon) with the
    population (1/G) variance.
  * update: Section 3, theta <- theta + (alpha / G) sum_i zhat_i eps_i, with
    no 1/sigma factor (alpha is the effective step); Appendix C.1 gives the
    canonical estimator with the factor 1/(G sigma), selectable here.
  * sigma schedule: Section 3.1,
    sigma_t = sigma_T + (sigma_0 - sigma_T) (1 + cos(pi t / T)) / 2.

Readings where the paper is silent (each also listed in the design notes):
  * Scalars cross the library boundary as binary32 (sigma, alpha, the z-score
    epsilon, rewards); the oracle takes those binary32 values and does all
    arithmetic on them in fp64.
  * Every result is rounded to bf16 once, round-to-nearest-even.  The update
    optionally rounds stochastically instead (ES_UPDATE_STOCHASTIC_ROUND,
    with a 64-bit rounding seed; the draws and the rounding are defined in
    the noise and bf16 modules).
  * sigma = 0 leaves the parameters bit-for-bit unchanged (no -0.0 -> +0.0).
  * A per-member sign s_i in {+1, -1} multiplies eps_i (antithetic pairs);
    s_i = +1 for every member is the paper's one-sided sampling.
  * Members that share a seed share eps; their weights c s_i zhat_i are summed
    into one weight per distinct seed (distinct seeds in order of first
    appearance).  Members whose merged weight is exactly zero contribute
    nothing, and when no weight is nonzero the parameters are left
    bit-for-bit unchanged (a zero update is no update, also for -0.0).
  * When all rewards are equal every zhat_i is exactly 0 (the mathematical
    value; computing mu in floating point could leave ~1e-17 residues).
  * A non-finite reward makes the update a no-op and raises a status flag
    (the paper maps invalid candidates to finite penalties before
    normalisation and skips all-invalid batches, Appendix D.6; the caller
    owns that mapping, the library only refuses non-finite input).
  * Update step t uses sigma_t, t = 0 .. T-1; sigma_T is reached after the
    last update.

Pins (tests/test_oracle_es.py): exact restore of the unrounded accumulation;
sigma = 0 and alpha = 0 identities; restore(sign) == perturb(-sign); the
z-score against scipy.stats.zscore and its closed forms (sum zero, mean
square, G = 2); single-member update == perturb; linearity; the direction of
the update; the schedule's endpoints and midpoint; and the distribution of
70-step update magnitudes against the paper's table for Qwen3.5-27B on
WebArena (Appendix A.1, Limitations).
"""

import numpy as np

from .bf16 import bf16_to_f64, f64_to_bf16_rne, f64_to_bf16_sr
from .noise import normals, rounding_draws

ES_UPDATE_DIV_SIGMA = 1
ES_REWARDS_ARE_WEIGHTS = 2
ES_UPDATE_STOCHASTIC_ROUND = 4
ES_UPDATE_MASTER = 8


def _f32(x):
    """The binary32 value a scalar takes at the library boundary, as fp64."""
    return float(np.float32(x))


def _elems(theta_bits, elems):
    if elems is None:
        return np.arange(np.asarray(theta_bits).size, dtype=np.uint64)
    return np.asarray(elems, dtype=np.uint64)


def perturb(theta_bits, seed, tensor_id, sign, sigma, elems=None):
    """theta' = RNE_bf16(theta + sign * sigma * eps(seed)) for the listed
    elements (all elements when elems is None).  theta_bits holds the bf16
    bits of exactly those elements, in the same order."""
    if sign not in (1, -1):
        raise ValueError("sign must be +1 or -1")
    if _f32(sigma) == 0.0:
        return np.asarray(theta_bits, dtype=np.uint16).ravel().copy()
    theta = bf16_to_f64(theta_bits).ravel()
    eps = normals(seed, tensor_id, _elems(theta_bits, elems))
    return f64_to_bf16_rne(theta + sign * _f32(sigma) * eps)


def restore(theta_bits, seed, tensor_id, sign, sigma, elems=None):
    """theta' = RNE_bf16(theta - sign * sigma * eps(seed))."""
    return perturb(theta_bits, seed, tensor_id, -sign, sigma, elems)


def swap(theta_bits, tensor_id, seed_from, sign_from, sigma_from, seed_to, sign_to,
         sigma_to, elems=None):
    """Move the perturbation from member a to member b: the revert of a
    followed by the apply of b (Section 3; Appendix D.6), each rounded to
    bf16 as the separate calls would be,
    theta' = RNE_bf16(RNE_bf16(theta - s_a sigma_a eps_a) + s_b sigma_b eps_b).

    Rounding the intermediate is what lets a walk over many members come
    back to its starting parameters: where a perturbation stays in the
    parameter's binade, the revert lands exactly on the starting bf16 value,
    so rounding errors do not accumulate from member to member (a single
    rounding of theta - a + b would carry each member's error into the next).
    """
    mid = restore(theta_bits, seed_from, tensor_id, sign_from, sigma_from, elems=elems)
    return perturb(mid, seed_to, tensor_id, sign_to, sigma_to, elems=elems)


def zscore(rewards, eps=1e-8):
    """Population z-score of a reward vector.

    Returns (z, status): z in fp64; status 1 (and z = 0) if any reward is not
    finite, else 0.  The rewards and eps are binary32 at the boundary.
    """
    r = np.asarray(rewards, dtype=np.float32).astype(np.float64)
    if r.size == 0:
        raise ValueError("empty reward vector")
    if not np.all(np.isfinite(r)):
        return np.zeros(r.size), 1
    if np.all(r == r[0]):
        return np.zeros(r.size), 0
    g = r.size
    mu = np.sum(r) / g
    s = np.sqrt(np.sum((r - mu) ** 2) / g)
    return (r - mu) / (s + _f32(eps)), 0


def update_coefficient(alpha, sigma, n_members, flags=0):
    """c = alpha / G (the paper's implemented update), or alpha / (G sigma)
    with ES_UPDATE_DIV_SIGMA (the canonical estimator of Appendix C.1)."""
    c = _f32(alpha) / n_members
    if flags & ES_UPDATE_DIV_SIGMA:
        c /= _f32(sigma)
    return c


def member_weights(seeds, signs, z, c):
    """Merge per-member weights c * s_i * zhat_i by seed.

    Returns (distinct_seeds, weights) with distinct seeds in order of first
    appearance and each weight the fp64 sum over the members with that seed.
    """
    order = []
    acc = {}
    for seed, s, zi in zip(seeds, signs, z):
        seed = int(seed)
        if seed not in acc:
            order.append(seed)
            acc[seed] = 0.0
        acc[seed] += c * int(s) * float(zi)
    return order, np.array([acc[k] for k in order], dtype=np.float64)


def update(theta_bits, tensor_id, seeds, signs, rewards, alpha, sigma,
           flags=0, zscore_eps=1e-8, elems=None, round_seed=0):
    """theta' = RNE_bf16(theta + sum_d w_d eps_d) over distinct seeds d.

    rewards are z-scored first unless ES_REWARDS_ARE_WEIGHTS is set, in which
    case they are used as zhat directly.  With ES_UPDATE_STOCHASTIC_ROUND the
    sum is rounded stochastically with the draws of round_seed instead.
    Returns (bits, status).
    """
    seeds = [int(s) for s in seeds]
    signs = [int(s) for s in signs]
    if len(seeds) == 0 or len(seeds) != len(signs) or len(seeds) != len(rewards):
        raise ValueError("seeds, signs and rewards must have the same nonzero length")
    if any(s not in (1, -1) for s in signs):
        raise ValueError("signs must be +1 or -1")
    theta_bits = np.asarray(theta_bits, dtype=np.uint16).ravel()
    if flags & ES_REWARDS_ARE_WEIGHTS:
        z = np.asarray(rewards, dtype=np.float32).astype(np.float64)
        status = 0 if np.all(np.isfinite(z)) else 1
    else:
        z, status = zscore(rewards, zscore_eps)
    if status:
        return theta_bits.copy(), status
    c = update_coefficient(alpha, sigma, len(seeds), flags)
    distinct, w = member_weights(seeds, signs, z, c)
    live = [(sd, wd) for sd, wd in zip(distinct, w) if wd != 0.0]
    if not live:
        return theta_bits.copy(), 0
    el = _elems(theta_bits, elems)
    delta = np.zeros(el.size, dtype=np.float64)
    for sd, wd in live:
        delta += wd * normals(sd, tensor_id, el)
    x = bf16_to_f64(theta_bits) + delta
    if flags & ES_UPDATE_STOCHASTIC_ROUND:
        return f64_to_bf16_sr(x, rounding_draws(round_seed, tensor_id, el)), 0
    return f64_to_bf16_rne(x), 0


def update_master(master, tensor_id, seeds, signs, rewards, alpha, sigma, flags=0,
                  zscore_eps=1e-8, elems=None):
    """The update into binary32 master copies (ES_UPDATE_MASTER, the
    library's update-numerics variant of Section 3's update):

        m' = binary32(m + sum_d w_d eps_d)     (the fp64 sum rounded once)
        working copy = RNE_bf16(m')

    with the z-score, coefficient and merged weights of update().  With
    nothing to add (no nonzero merged weight, or a non-finite reward: status
    1) m' = m, and the working copy is still RNE_bf16(m).
    Returns (m' as float32, working-copy bf16 bits, status).
    """
    seeds = [int(s) for s in seeds]
    signs = [int(s) for s in signs]
    if len(seeds) == 0 or len(seeds) != len(signs) or len(seeds) != len(rewards):
        raise ValueError("seeds, signs and rewards must have the same nonzero length")
    if any(s not in (1, -1) for s in signs):
        raise ValueError("signs must be +1 or -1")
    m = np.asarray(master, dtype=np.float32).ravel().astype(np.float64)
    if flags & ES_REWARDS_ARE_WEIGHTS:
        z = np.asarray(rewards, dtype=np.float32).astype(np.float64)
        status = 0 if np.all(np.isfinite(z)) else 1
    else:
        z, status = zscore(rewards, zscore_eps)
    live = []
    if not status:
        c = update_coefficient(alpha, sigma, len(seeds), flags)
        distinct, w = member_weights(seeds, signs, z, c)
        live = [(sd, wd) for sd, wd in zip(distinct, w) if wd != 0.0]
    out = m
    if live:
        el = np.arange(m.size, dtype=np.uint64) if elems is None else \
            np.asarray(elems, dtype=np.uint64).ravel()
        delta = np.zeros(el.size, dtype=np.float64)
        for sd, wd in live:
            delta += wd * normals(sd, tensor_id, el)
        with np.errstate(over="ignore", invalid="ignore"):
            out = m + delta
    with np.errstate(over="ignore"):
        m32 = out.astype(np.float32)
    return m32, f64_to_bf16_rne(m32.astype(np.float64)), status


def perturb_master(master, seed, tensor_id, sign, sigma, elems=None):
    """A member applied from binary32 masters (es_perturb_master): the bf16
    working copy RNE_bf16(m + sign sigma eps) of the masters m, rounded once
    from fp64 (Section 3's theta + sigma eps_i with theta the masters).
    sigma = 0 gives RNE_bf16(m)."""
    m = np.asarray(master, dtype=np.float32).ravel().astype(np.float64)
    el = np.arange(m.size, dtype=np.uint64) if elems is None else \
        np.asarray(elems, dtype=np.uint64).ravel()
    eps = normals(seed, tensor_id, el)
    return f64_to_bf16_rne(m + sign * _f32(sigma) * eps)


def sigma_cosine(sigma0, sigma_T, t, T):
    """sigma_t = sigma_T + (sigma_0 - sigma_T) (1 + cos(pi t / T)) / 2."""
    if T <= 0 or t < 0 or t > T:
        raise ValueError("need T >= 1 and 0 <= t <= T")
    return sigma_T + (sigma0 - sigma_T) * (1.0 + np.cos(np.pi * t / T)) / 2.0
