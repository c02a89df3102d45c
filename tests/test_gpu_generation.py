"""es_swap against the oracle, and the generation driver / replay: a live run
over several generations is rebuilt bit for bit from its records."""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_17310_amd import esopt, workloads as wl
from paper_2608_17310_amd.generation import (run_generation, replay, sigma_schedule,
                                             antithetic_seeds)
from parity import to_device, to_host, report, assert_parity

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)


def _swap_delta(tid, a, sa, b, sb, sigma, el):
    s32 = float(np.float32(sigma))
    if a == b:
        return (sb - sa) * s32 * oracle.normals(a, tid, el)
    return -sa * s32 * oracle.normals(a, tid, el) + sb * s32 * oracle.normals(b, tid, el)


@pytest.mark.parametrize("sizes", [[1 << 20], [5, 4097, 65536 + 3, 200000]])
def test_swap_matches_oracle(sizes):
    bits = [wl.random_bf16_bits(n, 80 + i) for i, n in enumerate(sizes)]
    ts = [to_device(b) for b in bits]
    plan = esopt.Plan(ts)
    plan.swap(31, 1, 32, -1, 1e-3)
    torch.cuda.synchronize()
    for i, b in enumerate(bits):
        el = np.arange(b.size, dtype=np.uint64)
        exp = oracle.swap(b, i, 31, 1, 1e-3, 32, -1, 1e-3)
        rep = report(to_host(ts[i]), exp, b, _swap_delta(i, 31, 1, 32, -1, 1e-3, el))
        print("swap", sizes[i], rep)
        assert_parity(rep, f"swap tensor {i}")
    plan.close()


def test_swap_unaligned_and_identity():
    bits = wl.random_bf16_bits(30001, 90)
    buf = to_device(bits)
    view = buf[3:]
    plan = esopt.Plan([view])
    plan.swap(7, 1, 7, 1, 1e-3)                  # same member: nothing to do
    torch.cuda.synchronize()
    np.testing.assert_array_equal(to_host(buf), bits)
    plan.swap(7, 1, 7, -1, 2e-3)                 # antithetic partner: weight -2 sigma
    torch.cuda.synchronize()
    b = bits[3:]
    el = np.arange(b.size, dtype=np.uint64)
    exp = oracle.swap(b, 0, 7, 1, 2e-3, 7, -1, 2e-3)
    rep = report(to_host(view), exp, b, -2 * float(np.float32(2e-3)) * oracle.normals(7, 0, el))
    assert_parity(rep, "antithetic swap")
    assert to_host(buf[:3]).tolist() == bits[:3].tolist()
    plan.close()


def _fresh(W, stream_seed=0):
    host = wl.host_params(W, stream_seed)
    return host, [to_device(b, s) for b, s in zip(host, W.shapes)]


@pytest.mark.parametrize("fused,flags", [(True, 0), (False, 0),
                                         (True, esopt.ES_UPDATE_STOCHASTIC_ROUND)])
def test_generation_replay_is_bit_exact(fused, flags):
    W = wl.TINY
    host, live = _fresh(W)
    plan = esopt.Plan(live)
    rng = np.random.default_rng(3)
    sig = sigma_schedule(1e-3, 1e-4, 4)
    records = []
    for t in range(4):
        seeds, signs = antithetic_seeds(100 * t, 3)
        rec = run_generation(plan, seeds, signs, sig[t], 5e-4,
                             evaluate=lambda i: rng.random(), fused_swap=fused, flags=flags,
                             round_seed=1000 + t)
        records.append(rec)
    torch.cuda.synchronize()
    live_bits = [to_host(t) for t in live]
    plan.close()
    _, again = _fresh(W)
    plan2 = esopt.Plan(again)
    replay(plan2, records)
    torch.cuda.synchronize()
    for a, b in zip(live_bits, again):
        np.testing.assert_array_equal(a, to_host(b))
    plan2.close()
    # the updates alone: the oracle's chain of the same four updates
    _, upd_only = _fresh(W)
    plan3 = esopt.Plan(upd_only)
    replay(plan3, records, with_perturbations=False)
    torch.cuda.synchronize()
    for tid, (b0, dev) in enumerate(zip(host, upd_only)):
        x = b0
        for rec in records:
            x, st = oracle.update(x, tid, rec.seeds, rec.signs,
                                  np.array(rec.rewards, np.float32), rec.alpha, rec.sigma,
                                  flags=rec.flags, round_seed=rec.round_seed)
        got = to_host(dev)
        ex = oracle.bf16_to_f64(x)
        floor = np.abs(oracle.bf16_to_f64(b0)) / 256
        ulp = oracle.bf16_ulp(np.maximum(np.abs(ex), floor))
        assert np.mean(got == x) > 0.999
        assert np.all(np.abs(oracle.bf16_to_f64(got) - ex) <= 2 * ulp)
    plan3.close()


def test_generation_matches_oracle_sequence():
    """One generation (fused swaps) on the tiny set against the oracle's
    perturb -> swap ... -> restore -> update sequence applied to the same
    starting parameters."""
    W = wl.TINY
    host, ts = _fresh(W)
    plan = esopt.Plan(ts)
    seeds, signs, sigma, alpha = [5, 6, 7, 8], [1, 1, 1, 1], 1e-3, 5e-4
    rewards = np.array([0.1, 0.7, 0.3, 0.9], np.float32)
    rec = run_generation(plan, seeds, signs, sigma, alpha, evaluate=lambda i: rewards[i])
    torch.cuda.synchronize()
    for tid, b in enumerate(host):
        x = oracle.perturb(b, seeds[0], tid, signs[0], sigma)
        scale = np.maximum(np.abs(oracle.bf16_to_f64(b)), np.abs(oracle.bf16_to_f64(x)))
        for i in range(len(seeds) - 1):
            x = oracle.swap(x, tid, seeds[i], signs[i], sigma, seeds[i + 1], signs[i + 1], sigma)
            scale = np.maximum(scale, np.abs(oracle.bf16_to_f64(x)))
        x = oracle.restore(x, seeds[-1], tid, signs[-1], sigma)
        x, st = oracle.update(x, tid, seeds, signs, rewards, alpha, sigma)
        got = to_host(ts[tid])
        ex = oracle.bf16_to_f64(x)
        d = np.abs(oracle.bf16_to_f64(got) - ex)
        # a tie broken differently at one pass moves that pass's result by one
        # ulp of that intermediate, which later passes carry unchanged: the
        # tolerance is in ulps of the largest value along the chain
        ulp = oracle.bf16_ulp(np.maximum(np.abs(ex), scale))
        bad = np.flatnonzero(d > 2 * ulp)
        assert np.mean(got == x) > 0.999
        assert bad.size == 0, (tid, bad[:5], oracle.bf16_to_f64(b)[bad[:5]], ex[bad[:5]],
                               oracle.bf16_to_f64(got)[bad[:5]], scale[bad[:5]])
    assert rec.rewards == [float(r) for r in rewards]
    plan.close()
