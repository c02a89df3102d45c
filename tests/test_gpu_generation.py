"""es_swap against the oracle, and the generation driver / replay: a live run
over several generations is rebuilt bit for bit from its records."""
import json

import numpy as np
import pytest
import torch

import oracle
from paper_2608_17310_amd import esopt, workloads as wl
from paper_2608_17310_amd.generation import (run_generation, replay, sigma_schedule,
                                             antithetic_seeds, save_log, load_log)
from parity import to_device, to_host, report, assert_parity

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)


def _swap_delta(tid, a, sa, b, sb, sigma, el):
    s32 = float(np.float32(sigma))
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


@pytest.mark.parametrize("case", [
    (31, 1, 1e-3, 32, -1, 1e-3),        # two keys
    (7, 1, 1e-3, 7, -1, 1e-3),          # antithetic partner: one key, noise generated once
    (7, 1, 1e-3, 7, 1, 1e-3),           # the same member: restore then perturb again
    (9, -1, 2e-3, 10, 1, 5e-4),         # different sigmas
    (9, 1, 0.0, 10, 1, 1e-3),           # zero sigma halves
    (9, 1, 1e-3, 10, 1, 0.0),
])
def test_swap_is_restore_then_perturb_bit_for_bit(case):
    a, sa, siga, b, sb, sigb = case
    bits = [wl.random_bf16_bits(n, 85 + i) for i, n in enumerate([1 << 18, 4097, 30001])]
    one = [to_device(x) for x in bits]
    two = [to_device(x) for x in bits]
    views1 = [one[0], one[1], one[2][3:]]
    views2 = [two[0], two[1], two[2][3:]]
    p1, p2 = esopt.Plan(views1), esopt.Plan(views2)
    p1.swap(a, sa, b, sb, siga, sigma_to=sigb)
    p2.restore(a, sa, siga)
    p2.perturb(b, sb, sigb)
    torch.cuda.synchronize()
    for i, (x, y) in enumerate(zip(one, two)):
        np.testing.assert_array_equal(to_host(x), to_host(y))
        el = np.arange(bits[i].size - (3 if i == 2 else 0), dtype=np.uint64)
        src = bits[i][3:] if i == 2 else bits[i]
        got = to_host(x)[3:] if i == 2 else to_host(x)
        exp = oracle.swap(src, i, a, sa, siga, b, sb, sigb)
        rep = report(got, exp, src, _swap_delta(i, a, sa, b, sb, max(siga, sigb), el))
        assert_parity(rep, f"swap {case} tensor {i}")
    assert to_host(one[2][:3]).tolist() == bits[2][:3].tolist()
    p1.close()
    p2.close()


def _fresh(W, stream_seed=0):
    host = wl.host_params(W, stream_seed)
    return host, [to_device(b, s) for b, s in zip(host, W.shapes)]


@pytest.mark.parametrize("fused,flags", [(True, 0), (False, 0),
                                         (True, esopt.ES_UPDATE_STOCHASTIC_ROUND)])
def test_generation_replay_is_bit_exact(fused, flags, tmp_path):
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
    # through the seed log on disk, as a run is rebuilt from its base checkpoint
    save_log(tmp_path / "log.json", records, meta={"workload": W.name})
    records, meta = load_log(tmp_path / "log.json")
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


def test_drift_study_matches_oracle_walk(capsys):
    """The drift tool's first restore-walk checkpoint on the tiny set: its
    changed-element fraction agrees with the oracle's perturb/restore chain
    over the same members."""
    from paper_2608_17310_amd import drift
    assert drift.main(["--workload", "tiny-1m", "--generations", "2", "--members", "4"]) == 0
    rows = [json.loads(l) for l in capsys.readouterr().out.splitlines() if l.startswith("{")]
    first = [r for r in rows if r.get("walk") == "restore" and r["generation"] == 1][0]
    W = wl.TINY
    flat, views = wl.device_params(W)          # the tool's starting parameters
    start = [to_host(v) for v in views]
    del flat, views
    changed = 0
    for tid, b in enumerate(start):
        x = b
        for i in range(4):
            x = oracle.perturb(x, 1_000_003 + i, tid, 1, 1e-3)
            x = oracle.restore(x, 1_000_003 + i, tid, 1, 1e-3)
        changed += int(np.sum(x != b))
    frac = changed / W.n_params
    print("drift gen 1: gpu", first["changed"], "oracle", frac)
    assert abs(first["changed"] - frac) < 2e-4
    assert 0.0 < frac < 0.5
    swap = [r for r in rows if r.get("walk") == "swap" and r["generation"] == 2][0]
    rest = [r for r in rows if r.get("walk") == "restore" and r["generation"] == 2][0]
    assert swap["roundings"] == 10 and rest["roundings"] == 16


def test_generation_on_a_side_stream_matches_default_stream():
    """A generation issued on a stream of its own (torch Stream or raw
    handle) gives the bits of the same generation on the current stream; the
    update's rewards are staged on that stream."""
    W = wl.TINY
    _, ref = _fresh(W)
    seeds, signs = antithetic_seeds(40, 3)
    scores = [0.3, 0.8, 0.1, 0.6, 0.9, 0.2]
    with esopt.Plan(ref) as p:
        run_generation(p, seeds, signs, 1e-3, 5e-4, evaluate=lambda i: scores[i])
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    for handle in (side, side.cuda_stream):
        _, ts = _fresh(W)
        torch.cuda.synchronize()
        with esopt.Plan(ts) as p:
            run_generation(p, seeds, signs, 1e-3, 5e-4, evaluate=lambda i: scores[i],
                           stream=handle)
            side.synchronize()
        for a, b in zip(ref, ts):
            assert torch.equal(a.view(torch.int16), b.view(torch.int16))


def test_side_stream_evaluation_sees_each_member_applied():
    """The passes on a side stream, the evaluation reading the parameters on
    the current stream: each evaluation sees exactly its member applied, even
    when the side stream is held back by other work queued on it."""
    W = wl.TINY
    seeds, signs = antithetic_seeds(50, 3)
    busy = torch.empty(1 << 28, dtype=torch.uint8, device="cuda")

    def run(stream, hold):
        _, ts = _fresh(W)
        torch.cuda.synchronize()

        def evaluate(i):
            v = float(ts[0].float().sum() + ts[3].float().sum())
            if hold:                        # queue work ahead of the next pass
                with torch.cuda.stream(stream):
                    for _ in range(4):
                        busy.add_(1)
            return v
        with esopt.Plan(ts) as p:
            rec = run_generation(p, seeds, signs, 1e-3, 5e-4, evaluate=evaluate, stream=stream)
            torch.cuda.synchronize()
        return rec.rewards, [to_host(t) for t in ts]

    ref_r, ref_t = run(None, False)
    assert len(set(ref_r)) == len(ref_r)        # every member scored differently
    side = torch.cuda.Stream()
    got_r, got_t = run(side, True)
    assert got_r == ref_r
    for a, b in zip(ref_t, got_t):
        np.testing.assert_array_equal(a, b)
