"""Helpers for GPU-vs-oracle parity checks (test infrastructure).

Error measure for bf16 results (the reading of the parity bar for floating
point): |got - expected| in units of the bf16 ulp at
max(|expected|, max(|theta|, |delta|) / 256), where delta is the oracle's
unrounded increment.  That is the ordinary ulp of the result, floored at the
operand scale minus 8 bits, so that results where theta and delta nearly
cancel (and any absolute error in eps is magnified into many result ulps)
are measured against the scale of the operands.  Plain result-ulp counts are
reported next to it.

Bar: at most 1 ulp on >= 99.99% of elements, never more than 2 ulp, and at
least 99.9% bit-exact (a bug detector: the GPU rounds binary32 to bf16 where
the oracle rounds fp64 once, so rare 1-ulp ties are expected).
"""
import numpy as np
import torch

import oracle


def to_device(bits, shape=None, device="cuda"):
    t = torch.from_numpy(np.ascontiguousarray(bits, dtype=np.uint16).view(np.int16))
    t = t.view(torch.bfloat16)
    if shape is not None:
        t = t.reshape(shape)
    return t.to(device)


def to_host(t):
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16).ravel().copy()


def ulp_errors(got, exp, theta, delta):
    """Floored ulp errors and plain result-ulp errors (fp64 arrays)."""
    g = oracle.bf16_to_f64(got)
    e = oracle.bf16_to_f64(exp)
    scale = np.maximum(np.abs(oracle.bf16_to_f64(theta)), np.abs(delta)) / 256.0
    floored = np.abs(g - e) / oracle.bf16_ulp(np.maximum(np.abs(e), scale))
    plain = np.abs(g - e) / oracle.bf16_ulp(e)
    return floored, plain


def report(got, exp, theta, delta):
    got = np.asarray(got, dtype=np.uint16).ravel()
    exp = np.asarray(exp, dtype=np.uint16).ravel()
    floored, plain = ulp_errors(got, exp, theta, delta)
    n = got.size
    return {
        "n": n,
        "exact": float(np.mean(got == exp)) if n else 1.0,
        "le1": float(np.mean(floored <= 1.0)) if n else 1.0,
        "max_ulp": float(floored.max()) if n else 0.0,
        "plain_max_ulp": float(plain.max()) if n else 0.0,
        "n_gt1": int(np.sum(floored > 1.0)),
        "n_cancel": int(np.sum(np.abs(oracle.bf16_to_f64(exp)) <
                               np.maximum(np.abs(oracle.bf16_to_f64(theta)), np.abs(delta)) / 256)),
    }


def assert_parity(rep, what=""):
    assert rep["max_ulp"] <= 2.0, (what, rep)
    assert rep["le1"] >= 0.9999, (what, rep)
    assert rep["exact"] >= 0.999, (what, rep)


def perturb_delta(seed, tensor_id, sign, sigma, elems):
    return sign * float(np.float32(sigma)) * oracle.normals(seed, tensor_id, elems)


def update_delta(tensor_id, seeds, signs, rewards, alpha, sigma, flags, elems, zscore_eps=1e-8):
    if flags & oracle.ES_REWARDS_ARE_WEIGHTS:
        z = np.asarray(rewards, np.float32).astype(np.float64)
    else:
        z, st = oracle.zscore(rewards, zscore_eps)
    c = oracle.update_coefficient(alpha, sigma, len(seeds), flags)
    distinct, w = oracle.member_weights(seeds, signs, z, c)
    d = np.zeros(np.asarray(elems).size)
    for s, wd in zip(distinct, w):
        if wd != 0.0:
            d += wd * oracle.normals(s, tensor_id, elems)
    return d


# ------------------------------------------------------------------ int8 path --
# The int8 passes turn a binary32 step d (in quanta) and a draw into the
# integer floor(v): v = d + (2 r + 1) 2^-10 for a perturbation (9-bit r),
# v = d + r 2^-16 for an update (16-bit r).  The GPU's d differs from the oracle's fp64
# d by the noise error (|d eps| <= 4e-6 + 2e-6 |eps| per unit weight) and a
# few binary32 roundings, so where v lies within that bound of an
# integer both floor values are correct; everywhere else the code is unique.

F32_EPS = 2.0 ** -23


def q_tolerance(abs_weight_sum, noise_abs_sum, d):
    """Bound on |d_gpu - d_oracle| in quanta: abs_weight_sum = sum_d |w_d| / s,
    noise_abs_sum = sum_d |w_d eps_d| / s (fp64 arrays)."""
    return (abs_weight_sum * 4e-6 + noise_abs_sum * (2e-6 + 8 * F32_EPS)
            + 4 * F32_EPS * (np.abs(d) + 2.0))


def qreport(got, q_in, v, tol, ok, negate=False):
    """Compare GPU codes with the oracle's rule code = clamp(q +- floor(v)),
    v the fp64 decision value (the step in quanta plus the draw's offset);
    near-integer cases (within tol) accept either floor."""
    got = np.asarray(got, dtype=np.int8).astype(np.int64)
    q = np.asarray(q_in, dtype=np.int8).astype(np.int64)
    k = np.floor(v).astype(np.int64)
    near = np.abs(v - np.round(v)) <= tol
    alt = np.where(v - np.round(v) < 0, k + 1, k - 1)     # the other side of the integer
    sgn = -1 if negate else 1

    def code(kk):
        return np.where(ok, np.clip(q + sgn * kk, -127, 127), q)
    exp, exp_alt = code(k), code(alt)
    good = (got == exp) | (near & (got == exp_alt))
    n = got.size
    return {"n": n, "exact": float(np.mean(got == exp)) if n else 1.0,
            "near": int(near.sum()), "bad": int((~good).sum()),
            "first_bad": np.flatnonzero(~good)[:5].tolist()}


def assert_qparity(rep, what=""):
    assert rep["bad"] == 0, (what, rep)
    assert rep["exact"] >= 0.9999, (what, rep)


# ------------------------------------------------------------------- fp8 path --
# An fp8 pass decides between the two grid neighbours lo and lo + h of
# x = v + step (binary32) by comparing f = (x - lo) / h with a threshold.
# The GPU's x differs from the oracle's by the noise error and binary32
# roundings, so where the oracle's f lies within that bound (over h) of the
# threshold both neighbours are correct; everywhere else the code is unique.
# (Where x is near a grid point instead, both sides reach that grid point.)


def f8_tolerance(abs_weight_sum, noise_abs_sum, x):
    """Bound on |x_gpu - x_oracle| in scale units: abs_weight_sum =
    sum_d |w_d| / s, noise_abs_sum = sum_d |w_d eps_d| / s (fp64 arrays)."""
    return (abs_weight_sum * 4e-6 + noise_abs_sum * (2e-6 + 8 * F32_EPS)
            + 4 * F32_EPS * (np.abs(x) + 2.0 ** -9))


def f8report(got, exp, x32, thr, tol, ok):
    """GPU codes against the oracle's codes `exp`: equal, or -- where the
    oracle's decision value is within tol of its threshold -- the other grid
    neighbour.  x32: the oracle's binary32 x (fp64 array), thr: the threshold
    of each element, ok: elements a pass may change."""
    from oracle import fp8 as of
    got = np.asarray(got, dtype=np.uint8).ravel()
    exp = np.asarray(exp, dtype=np.uint8).ravel()
    x32 = np.asarray(x32, dtype=np.float64)
    inside = ok & (np.abs(x32) < of.E4M3_MAX)
    xc = np.where(inside, x32, 0.0)
    lo, h = of.grid_floor(xc)
    f = (xc - lo) / h
    near = inside & (np.abs(f - thr) <= tol / h)
    v_exp = of.e4m3_decode(exp)
    alt_v = np.where(v_exp == lo, lo + h, lo)
    alt = of.e4m3_encode(np.where(near, alt_v, 0.0))
    good = (got == exp) | (near & (got == alt))
    n = got.size
    return {"n": n, "exact": float(np.mean(got == exp)) if n else 1.0,
            "near": int(near.sum()), "bad": int((~good).sum()),
            "first_bad": np.flatnonzero(~good)[:5].tolist()}


def assert_f8parity(rep, what=""):
    assert rep["bad"] == 0, (what, rep)
    assert rep["exact"] >= 0.9999, (what, rep)


# ----------------------------------------------------------- binary32 masters --
# An update into binary32 masters (ES_UPDATE_MASTER) rounds once to binary32
# on both sides, so its bar is the bound of their difference, derived from
# the kernel's arithmetic: the normals' error (the bar above: 4e-6 + 2e-6 |eps|
# per normal, times |w|), the binary32 products and accumulation over the
# live members (at most N + 3 roundings of a partial sum bounded by
# sum |w eps|), and the two final roundings (one ulp of the result).

def master_tolerance(m_exp, live, tensor_id, elems):
    """Per-element bound |got - exp| for an update into masters; live is the
    oracle's [(seed, weight)] of nonzero merged weights."""
    import oracle
    wsum = np.zeros(elems.size)
    weps = np.zeros(elems.size)
    for sd, w in live:
        e = np.abs(oracle.normals(sd, tensor_id, elems))
        wsum += abs(w) * (4e-6 + 2e-6 * e)
        weps += abs(w) * e
    ulp = np.spacing(np.abs(np.asarray(m_exp, np.float32))).astype(np.float64)
    return wsum + (len(live) + 3) * 2.0 ** -24 * weps + ulp


def master_report(got, exp, tol):
    got = np.asarray(got, np.float32).astype(np.float64)
    exp = np.asarray(exp, np.float32).astype(np.float64)
    err = np.abs(got - exp)
    bad = ~(err <= tol)
    return {"n": int(got.size), "exact": float(np.mean(got == exp)) if got.size else 1.0,
            "max_err_over_tol": float(np.max(err / tol)) if got.size else 0.0,
            "bad": int(bad.sum()), "first_bad": np.flatnonzero(bad)[:5].tolist()}


def assert_master_parity(rep, what=""):
    assert rep["bad"] == 0, (what, rep)
