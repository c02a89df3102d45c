"""Degenerate parameter values through the passes: signed zeros, subnormals,
the smallest normal, values next to the largest finite bf16, infinities and
NaNs with payloads mixed into an ordinary tensor.  Finite values match the
oracle at the parity bar through perturb, swap, restore and both update
roundings; infinities keep their bits; NaNs stay NaN.  A radius small enough
that the results themselves are bf16 subnormals matches the oracle too (the
kernels keep binary32 subnormals; nothing is flushed to zero)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_17310_amd import esopt, workloads as wl
from parity import assert_parity, perturb_delta, report, to_device, to_host, update_delta

pytestmark = pytest.mark.gpu

SPECIAL = [0x0000, 0x8000, 0x0001, 0x8001, 0x007F, 0x807F, 0x0080, 0x8080, 0x7F7F, 0xFF7F,
           0x7F7E, 0xFF7E, 0x7F80, 0xFF80, 0x7FC0, 0xFFC0, 0x7F81, 0x7FC1, 0xFFFF]


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)


def _is_nan(b):
    return ((b & 0x7F80) == 0x7F80) & ((b & 0x007F) != 0)


def _is_inf(b):
    return (b & 0x7FFF) == 0x7F80


def _check(name, got, exp, base, delta):
    finite = ~_is_nan(base) & ~_is_inf(base)
    np.testing.assert_array_equal(got[_is_inf(base)], base[_is_inf(base)], err_msg=name)
    assert np.all(_is_nan(got[_is_nan(base)])), name
    rep = report(got[finite], exp[finite], base[finite], delta[finite])
    print(name, rep)
    assert_parity(rep, name)


def _passes(x, sigma, tid, r):
    """Every pass on the GPU, each compared with the oracle applied to the
    GPU's own state before it."""
    n = x.size
    el = np.arange(n, dtype=np.uint64)
    t = to_device(x)
    states = [x]
    with esopt.Plan([t], tensor_ids=[tid]) as p:
        for step in (lambda: p.perturb(5, 1, sigma),
                     lambda: p.swap(5, 1, 6, -1, sigma),
                     lambda: p.restore(6, -1, sigma),
                     lambda: p.update([7, 8, 9], [1, -1, 1], torch.from_numpy(r).cuda(), 5e-4,
                                      sigma=sigma),
                     lambda: p.update([7, 8, 9], [1, -1, 1], torch.from_numpy(r).cuda(), 5e-4,
                                      sigma=sigma, flags=esopt.ES_UPDATE_STOCHASTIC_ROUND,
                                      round_seed=11)):
            step()
            torch.cuda.synchronize()
            states.append(to_host(t))
    upd = update_delta(tid, [7, 8, 9], [1, -1, 1], r, 5e-4, sigma, 0, el)
    x0, x1, x2, x3, x4, x5 = states
    with np.errstate(invalid="ignore", over="ignore"):
        _check("perturb", x1, oracle.perturb(x0, 5, tid, 1, sigma), x0,
               perturb_delta(5, tid, 1, sigma, el))
        _check("swap", x2, oracle.swap(x1, tid, 5, 1, sigma, 6, -1, sigma), x1,
               perturb_delta(5, tid, -1, sigma, el) + perturb_delta(6, tid, -1, sigma, el))
        _check("restore", x3, oracle.restore(x2, 6, tid, -1, sigma), x2,
               perturb_delta(6, tid, 1, sigma, el))
        _check("update", x4, oracle.update(x3, tid, [7, 8, 9], [1, -1, 1], r, 5e-4, sigma)[0],
               x3, upd)
        _check("update_sr", x5, oracle.update(x4, tid, [7, 8, 9], [1, -1, 1], r, 5e-4, sigma,
                                              flags=esopt.ES_UPDATE_STOCHASTIC_ROUND,
                                              round_seed=11)[0], x4, upd)
    return states


def test_special_parameter_values_through_every_pass():
    x = wl.random_bf16_bits(70_001, 81)
    rng = np.random.default_rng(82)
    pos = rng.choice(x.size, size=4000, replace=False)
    x[pos] = np.array(SPECIAL, np.uint16)[np.arange(pos.size) % len(SPECIAL)]
    x[:len(SPECIAL)] = SPECIAL
    r = np.array([0.7, 0.1, 0.4], np.float32)
    _passes(x, 1e-3, 3, r)


def test_subnormal_results_are_not_flushed():
    """Parameters at 0 and at bf16 subnormals with a radius of 1e-39: every
    result is a subnormal (or zero) that the kernels must not flush."""
    rng = np.random.default_rng(83)
    x = np.zeros(20_000, np.uint16)
    x[1::2] = rng.integers(1, 0x80, 10_000).astype(np.uint16) | np.where(
        rng.random(10_000) < 0.5, 0x8000, 0).astype(np.uint16)
    r = np.array([0.2, 0.9, 0.5], np.float32)
    states = _passes(x, 1e-39, 4, r)
    assert np.count_nonzero(states[1] & 0x7FFF) > 10_000      # subnormal results exist
