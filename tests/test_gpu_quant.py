"""The int8 path on the GPU against the oracle: perturb, restore (exact
wherever nothing clamped), the stochastically rounded update in quanta, the
identities, launch-shape invariance, and the 27B-shaped int8 set on sampled
elements in the benchmark's launch configuration."""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_17310_amd import esopt, workloads as wl
from parity import q_tolerance, qreport, assert_qparity

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)


def _codes(n, seed):
    return np.random.default_rng(seed).integers(-127, 128, size=n).astype(np.int8)


def _scales(n_rows, seed, lo=2e-4, hi=1e-3):
    return np.random.default_rng(seed).uniform(lo, hi, max(n_rows, 1)).astype(np.float32)


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _host(t):
    return t.detach().cpu().numpy().copy()


def _perturb_expect(scales, row, seed, tid, sign, sigma, el):
    """(v, ok, tol): the oracle's decision value floor(v) = offset."""
    d, r, ok = oracle.offset_values(scales, row, seed, tid, sign, sigma, el)
    s = oracle.row_scales(scales, row, el)
    s = np.where(ok, s, 1.0)
    s32 = float(np.float32(sigma))
    eps = oracle.normals(seed, tid, el)
    tol = q_tolerance(s32 / s, np.abs(s32 * eps) / s, d)
    return d + (2 * r + 1) * 2.0 ** -10, ok, tol


def _update_expect(scales, row, tid, seeds, signs, rewards, alpha, sigma, flags, el, rs):
    """(v, ok, tol, live, status) of the update."""
    d, r, ok, live, st = oracle.update_values(scales, row, tid, seeds, signs, rewards, alpha,
                                              sigma, flags, elems=el, round_seed=rs)
    s = np.where(ok, oracle.row_scales(scales, row, el), 1.0)
    wsum = np.zeros(el.size)
    nsum = np.zeros(el.size)
    for sd, w in live:
        wsum += abs(w) / s
        nsum += np.abs(w * oracle.normals(sd, tid, el)) / s
    return d + r * 2.0 ** -16, ok, q_tolerance(wsum, nsum, d), live, st


def _tensor_set():
    """Codes, scales, rows, ids: row lengths 1024 / 8 / one scale / 5120, an
    unaligned view, rows with invalid scales, large tensor ids."""
    sizes = [1 << 18, 4096 * 5 + 24, 40, 300004]
    rows = [1024, 8, 0, 5120]
    ids = [0, 7, 1000, (1 << 32) - 1]
    codes = [_codes(n, 10 + i) for i, n in enumerate(sizes)]
    scales = []
    for i, (n, row) in enumerate(zip(sizes, rows)):
        sc = _scales(1 if row == 0 else -(-n // row), 20 + i)
        scales.append(sc)
    scales[1][[3, 50, 51]] = [0.0, np.inf, 1e-40]     # invalid: left unchanged
    scales[1][[7, 8]] = 2e-6                           # offsets large enough to clamp
    # -128 (outside the clamp range): kept in rows with an invalid scale,
    # clamped into [-127, 127] by a step in a valid row (row 10)
    codes[1][[3 * 8, 3 * 8 + 5, 50 * 8 + 1, 51 * 8 + 7, 10 * 8 + 2]] = -128
    return codes, scales, rows, ids


def _device_views(codes):
    """Device copies; the last tensor is a view at byte offset 3."""
    bufs = [_dev(c) for c in codes[:-1]]
    pad = np.concatenate([np.array([5, -5, 9], np.int8), codes[-1]])
    last = _dev(pad)
    return bufs + [last], bufs + [last[3:]]


def test_qperturb_and_restore_match_oracle():
    codes, scales, rows, ids = _tensor_set()
    bufs, views = _device_views(codes)
    sdev = [_dev(s) for s in scales]
    plan = esopt.QPlan(views, sdev, rows, tensor_ids=ids)
    assert plan.numel == sum(c.size for c in codes)
    seed, sign, sigma = (1 << 40) + 5, -1, 1e-3
    plan.perturb(seed, sign, sigma)
    torch.cuda.synchronize()
    pert = [_host(v) for v in views]
    plan.restore(seed, sign, sigma)
    torch.cuda.synchronize()
    back = [_host(v) for v in views]
    assert _host(bufs[-1][:3]).tolist() == [5, -5, 9]
    for i, (q, sc, row, tid) in enumerate(zip(codes, scales, rows, ids)):
        el = np.arange(q.size, dtype=np.uint64)
        v, ok, tol = _perturb_expect(sc, row, seed, tid, sign, sigma, el)
        rep = qreport(pert[i], q, v, tol, ok)
        print("qperturb", i, rep)
        assert_qparity(rep, f"qperturb tensor {i}")
        rep = qreport(back[i], pert[i], v, tol, ok, negate=True)
        print("qrestore", i, rep)
        assert_qparity(rep, f"qrestore tensor {i}")
        # exact revert wherever the perturbed code was not at a clamp bound
        # (and the code was inside the clamp range to begin with)
        free = (np.abs(pert[i].astype(np.int64)) < 127) & (q > -128)
        np.testing.assert_array_equal(back[i][free], q[free])
    assert np.mean(pert[0] != codes[0]) > 0.5
    plan.close()


@pytest.mark.parametrize("flags", [0, esopt.ES_UPDATE_DIV_SIGMA, esopt.ES_REWARDS_ARE_WEIGHTS])
def test_qupdate_matches_oracle(flags):
    codes, scales, rows, ids = _tensor_set()
    bufs, views = _device_views(codes)
    sdev = [_dev(s) for s in scales]
    plan = esopt.QPlan(views, sdev, rows, tensor_ids=ids)
    seeds = [21, 21, 22, 22, 23, 24, 25, 26]
    signs = [1, -1, 1, -1, 1, 1, 1, 1]
    r = np.random.default_rng(4).random(8).astype(np.float32)
    rs = 0xFEEDFACE01234567
    alpha = 5e-3 if flags != esopt.ES_REWARDS_ARE_WEIGHTS else 2e-3
    status = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    plan.update(seeds, signs, _dev(r), alpha, sigma=1e-3, flags=flags, round_seed=rs,
                status_out=status)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    for i, (q, sc, row, tid) in enumerate(zip(codes, scales, rows, ids)):
        el = np.arange(q.size, dtype=np.uint64)
        v, ok, tol, live, st = _update_expect(sc, row, tid, seeds, signs, r, alpha, 1e-3,
                                              flags, el, rs)
        got = _host(views[i])
        rep = qreport(got, q, v, tol, ok)
        print("qupdate", flags, i, rep)
        assert_qparity(rep, f"qupdate flags={flags} tensor {i}")
        assert np.mean(got != q) > 0.05 or q.size < 100
    plan.close()


def test_qupdate_large_population_and_oracle_function():
    q = _codes(1 << 16, 30)
    sc = _scales(64, 31)
    t = _dev(q)
    plan = esopt.QPlan([t], [_dev(sc)], [1024])
    seeds = list(range(500, 564))
    r = np.random.default_rng(6).standard_normal(64).astype(np.float32)
    plan.update(seeds, [1] * 64, _dev(r), 2e-2, round_seed=3)
    torch.cuda.synchronize()
    el = np.arange(q.size, dtype=np.uint64)
    v, ok, tol, live, st = _update_expect(sc, 1024, 0, seeds, [1] * 64, r, 2e-2, 0.0, 0, el, 3)
    rep = qreport(_host(t), q, v, tol, ok)
    print("qupdate N=64", rep)
    assert_qparity(rep, "qupdate N=64")
    exp, st = oracle.qupdate(q, sc, 1024, 0, seeds, [1] * 64, r, 2e-2, 0.0, round_seed=3)
    assert np.mean(_host(t) == exp) >= 0.9999
    plan.close()


def test_q_identities():
    q = _codes(50000, 40)
    sc = _scales(50000 // 8 + 1, 41)
    t = _dev(q)
    plan = esopt.QPlan([t], [_dev(sc)], [8])
    plan.perturb(3, 1, 0.0)
    plan.update([1, 2], [1, 1], _dev(np.array([0.5, 0.5], np.float32)), 5e-3)      # equal rewards
    plan.update([1, 2], [1, 1], _dev(np.array([0.1, 0.9], np.float32)), 0.0)       # alpha 0
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    plan.update([1, 2], [1, 1], _dev(np.array([0.1, np.nan], np.float32)), 5e-3, status_out=status)
    torch.cuda.synchronize()
    assert int(status.item()) == 1
    np.testing.assert_array_equal(_host(t), q)
    plan.close()


@pytest.mark.parametrize("shape", [(256, 2, 1), (512, 8, 3), (1024, 8, 8)])
def test_q_results_do_not_depend_on_launch_shape(shape, monkeypatch):
    codes, scales, rows, ids = _tensor_set()
    r = _dev(np.array([0.3, 0.9, 0.1, 0.5], np.float32))

    def run():
        bufs, views = _device_views(codes)
        plan = esopt.QPlan(views, [_dev(s) for s in scales], rows, tensor_ids=ids)
        plan.perturb(9, 1, 1e-3)
        plan.update([1, 2, 2, 5], [1, 1, -1, 1], r, 5e-3, round_seed=11)
        plan.restore(9, 1, 1e-3)
        torch.cuda.synchronize()
        out = [_host(v) for v in views]
        plan.close()
        return out

    ref = run()
    threads, groups, wg = shape
    monkeypatch.setenv("ESOPT_THREADS", str(threads))
    monkeypatch.setenv("ESOPT_QGROUPS", str(groups))
    monkeypatch.setenv("ESOPT_UPDATE_WG_PER_CU", str(wg))
    for a, b in zip(ref, run()):
        np.testing.assert_array_equal(a, b)


def _samples(numel, rng, k):
    fixed = [0, 1, 7, 8, 15, 16, 65535, 65536, numel // 2, numel - 17, numel - 1]
    idx = np.concatenate([np.array([i for i in fixed if 0 <= i < numel], dtype=np.int64),
                          rng.integers(0, numel, size=min(k, numel))])
    return np.unique(idx)


def test_int8_27b_set_sampled():
    """The 27B-shaped set as int8 codes with per-row scales, one plan, the
    benchmark's launch configuration: perturb, restore, N = 32 update, checked
    on sampled codes."""
    W = wl.DENSE_27B
    flat, views, scales, rows = wl.device_qparams(W)
    plan = esopt.QPlan(views, scales, rows)
    assert plan.numel == W.n_params
    rng = np.random.default_rng(3)
    idx = [_samples(v.numel(), rng, 64) for v in views]
    idx_dev = [torch.from_numpy(i).cuda() for i in idx]
    host_scales = [_host(s) for s in scales]

    def gather():
        return [_host(v.index_select(0, i)) for v, i in zip(views, idx_dev)]
    q0 = gather()
    seed, sigma = 31, W.sigma0
    plan.perturb(seed, 1, sigma)
    torch.cuda.synchronize()
    pert = gather()
    plan.restore(seed, 1, sigma)
    torch.cuda.synchronize()
    back = gather()
    seeds, signs = list(W.seeds), list(W.signs)
    r = wl.rewards(W)
    plan.update(seeds, signs, _dev(r), W.alpha, round_seed=77)
    torch.cuda.synchronize()
    upd = gather()
    plan.close()
    del flat, views
    torch.cuda.empty_cache()
    tot = {"perturb": [0, 0, 0], "restore": [0, 0, 0], "update": [0, 0, 0]}
    for t, el_i in enumerate(idx):
        el = el_i.astype(np.uint64)
        sc, row = host_scales[t], rows[t]
        v, ok, tol = _perturb_expect(sc, row, seed, t, 1, sigma, el)
        for name, got, base, neg in (("perturb", pert[t], q0[t], False),
                                     ("restore", back[t], pert[t], True)):
            rep = qreport(got, base, v, tol, ok, negate=neg)
            tot[name][0] += rep["n"]; tot[name][1] += rep["bad"]
            tot[name][2] += int(round(rep["exact"] * rep["n"]))
        free = np.abs(pert[t].astype(np.int64)) < 127
        np.testing.assert_array_equal(back[t][free], q0[t][free])
        v, ok, tol, live, st = _update_expect(sc, row, t, seeds, signs, r, W.alpha, sigma, 0,
                                              el, 77)
        rep = qreport(upd[t], back[t], v, tol, ok)
        tot["update"][0] += rep["n"]; tot["update"][1] += rep["bad"]
        tot["update"][2] += int(round(rep["exact"] * rep["n"]))
    for name, (n, bad, exact) in tot.items():
        print("int8 27b", name, {"n": n, "bad": bad, "exact": exact / n})
        assert bad == 0, name
        assert exact / n >= 0.9999, name


def test_int8_generation_replay_is_bit_exact():
    """Four generations of the driver on the tiny set as int8 codes (revert
    exact wherever nothing clamps, update rounded stochastically) are rebuilt
    bit for bit from their records; the update-only replay equals the
    oracle's chain of updates."""
    from paper_2608_17310_amd.generation import run_generation, replay, antithetic_seeds
    W = wl.TINY
    host = wl.host_qparams(W)

    def fresh():
        codes = [_dev(q) for q, _, _ in host]
        return codes, esopt.QPlan(codes, [_dev(s) for _, s, _ in host], [r for _, _, r in host])
    codes, plan = fresh()
    rng = np.random.default_rng(12)
    records = []
    for t in range(4):
        seeds, signs = antithetic_seeds(50 * t, 3)
        records.append(run_generation(plan, seeds, signs, 1e-3, 5e-3,
                                      evaluate=lambda i: rng.random(), round_seed=500 + t))
    torch.cuda.synchronize()
    live = [_host(c) for c in codes]
    plan.close()
    codes2, plan2 = fresh()
    replay(plan2, records)
    torch.cuda.synchronize()
    for a, b in zip(live, codes2):
        np.testing.assert_array_equal(a, _host(b))
    plan2.close()
    codes3, plan3 = fresh()
    replay(plan3, records, with_perturbations=False)
    torch.cuda.synchronize()
    for tid, ((q0, sc, row), dev) in enumerate(zip(host, codes3)):
        x = q0
        for rec in records:
            x, st = oracle.qupdate(x, sc, row, tid, rec.seeds, rec.signs,
                                   np.array(rec.rewards, np.float32), rec.alpha, rec.sigma,
                                   round_seed=rec.round_seed)
        assert np.mean(_host(dev) == x) >= 0.9999
        assert np.max(np.abs(_host(dev).astype(np.int64) - x)) <= 1
    plan3.close()
    # the live run against the oracle's whole chain (walks and updates)
    for tid, ((q0, sc, row), got) in enumerate(zip(host, live)):
        x = q0
        for rec in records:
            for sd, sg in zip(rec.seeds, rec.signs):
                x = oracle.qperturb(x, sc, row, sd, tid, sg, rec.sigma)
                x = oracle.qrestore(x, sc, row, sd, tid, sg, rec.sigma)
            x, st = oracle.qupdate(x, sc, row, tid, rec.seeds, rec.signs,
                                   np.array(rec.rewards, np.float32), rec.alpha, rec.sigma,
                                   round_seed=rec.round_seed)
        assert np.mean(got == x) >= 0.9999
        assert np.max(np.abs(got.astype(np.int64) - x)) <= 1


def test_int8_tensor_at_the_code_limit():
    """An int8 tensor of 2^31 - 9 codes (the largest accepted) with rows of 4096:
    codes near the end, across the last full tile and in the ragged tail are
    checked after perturb, restore and update."""
    n = (1 << 31) - 9
    row = 4096
    q = torch.randint(-100, 101, (n,), dtype=torch.int8, device="cuda")
    n_rows = -(-n // row)
    sc_host = _scales(n_rows, 50)
    sc = _dev(sc_host)
    plan = esopt.QPlan([q], [sc], [row], tensor_ids=[3])
    last_full = (n // 65536) * 65536
    idx = np.unique(np.concatenate([np.arange(0, 32), np.arange(last_full - 32, last_full + 32),
                                    np.arange(n - 40, n),
                                    np.random.default_rng(2).integers(0, n, 300)]).astype(np.int64))
    idx_dev = torch.from_numpy(idx).cuda()
    el = idx.astype(np.uint64)

    def gather():
        torch.cuda.synchronize()
        return _host(q.index_select(0, idx_dev))
    q0 = gather()
    plan.perturb(21, 1, 1e-3)
    q1 = gather()
    plan.restore(21, 1, 1e-3)
    q2 = gather()
    r = np.array([0.9, 0.1, 0.4, 0.6], np.float32)
    plan.update([7, 8, 9, 10], [1, 1, 1, 1], _dev(r), 2e-2, round_seed=5)
    q3 = gather()
    plan.close()
    del q
    torch.cuda.empty_cache()
    v, ok, tol = _perturb_expect(sc_host, row, 21, 3, 1, 1e-3, el)
    assert_qparity(qreport(q1, q0, v, tol, ok), "perturb at the limit")
    assert_qparity(qreport(q2, q1, v, tol, ok, negate=True), "restore at the limit")
    free = np.abs(q1.astype(np.int64)) < 127
    np.testing.assert_array_equal(q2[free], q0[free])
    v, ok, tol, live, st = _update_expect(sc_host, row, 3, [7, 8, 9, 10], [1] * 4, r, 2e-2, 0.0,
                                          0, el, 5)
    assert_qparity(qreport(q3, q2, v, tol, ok), "update at the limit")
