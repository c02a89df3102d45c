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
