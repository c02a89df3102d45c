"""The fp8 (E4M3) path on the GPU against the oracle, through the C ABI:
perturb, restore (against the oracle's restore of the GPU's perturbed codes,
and exact wherever the revert stays inside a binade), the stochastically
rounded update in all three coefficient modes and at N = 64, the
identities, launch-shape invariance, the code checksum, random layouts, and
the 27B-shaped fp8 set on sampled elements in the benchmark's launch
configuration.  Codes include every byte value: not-a-number codes, -0, the
largest values +-448 and subnormals."""
import numpy as np
import pytest
import torch

import oracle
from oracle import fp8 as of
from paper_2608_17310_amd import esopt, workloads as wl
from parity import f8_tolerance, f8report, assert_f8parity

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)


def _f32(a):
    return np.asarray(a, dtype=np.float64).astype(np.float32).astype(np.float64)


def _codes(n, seed):
    """Quantized N(0, 1) values at scale 1/100 (most codes), with every byte
    value sprinkled in (not-a-number codes, -0, +-448, subnormals)."""
    rng = np.random.default_rng(seed)
    c = torch.from_numpy(np.clip(rng.normal(0, 100, n), -448, 448)).to(
        torch.float8_e4m3fn).view(torch.uint8).numpy().copy()
    k = max(1, n // 50)
    c[rng.integers(0, n, k)] = rng.integers(0, 256, k).astype(np.uint8)
    c[rng.integers(0, n, max(1, n // 500))] = rng.choice([0x7F, 0xFF, 0x80, 0x7E, 0xFE, 0x01, 0x81],
                                                          max(1, n // 500))
    return c


def _scales(n_rows, seed, lo=1.5e-4, hi=3e-4):
    return np.random.default_rng(seed).uniform(lo, hi, max(n_rows, 1)).astype(np.float32)


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _host(t):
    return t.detach().cpu().numpy().copy()


def _perturb_report(got, c_in, scales, row, seed, tid, sign, sigma, el, restore=False):
    v, d, u, ok = of.perturb_values(c_in, scales, row, seed, tid, sign, sigma, el)
    x = _f32(v - d if restore else v + d)
    thr = u if restore else 1.0 - u
    fn = of.f8restore if restore else of.f8perturb
    exp = fn(c_in, scales, row, seed, tid, sign, sigma, elems=el)
    s = np.where(ok, oracle.row_scales(scales, row, el), 1.0)
    s32 = float(np.float32(sigma))
    tol = f8_tolerance(s32 / s, np.abs(d), x)
    return f8report(got, exp, x, thr, tol, ok)


def _update_report(got, c_in, scales, row, tid, seeds, signs, rewards, alpha, sigma, flags, el,
                   rs):
    v, delta, u, ok, live, st = of.f8update_values(c_in, scales, row, tid, seeds, signs,
                                                   rewards, alpha, sigma, flags, elems=el,
                                                   round_seed=rs)
    assert st == 0
    exp, st = of.f8update(c_in, scales, row, tid, seeds, signs, rewards, alpha, sigma,
                          flags=flags, elems=el, round_seed=rs)
    if not live:
        return {"n": len(got), "exact": float(np.mean(got == exp)), "near": 0,
                "bad": int(np.sum(got != exp)), "first_bad": []}
    s = np.where(ok, oracle.row_scales(scales, row, el), 1.0)
    wsum = np.zeros(el.size)
    nsum = np.zeros(el.size)
    for sd, w in live:
        wsum += abs(w) / s
        nsum += np.abs(w * oracle.normals(sd, tid, el)) / s
    x = _f32(v + delta)
    return f8report(got, exp, x, 1.0 - u, f8_tolerance(wsum, nsum, x), ok)


def _tensor_set():
    """Codes, scales, rows, ids: row lengths 1024 / 8 / one scale / 5120, an
    unaligned view, rows with invalid scales, large tensor ids."""
    sizes = [1 << 18, 4096 * 5 + 24, 40, 300004]
    rows = [1024, 8, 0, 5120]
    ids = [0, 7, 1000, (1 << 32) - 1]
    codes = [_codes(n, 10 + i) for i, n in enumerate(sizes)]
    scales = [_scales(1 if row == 0 else -(-n // row), 20 + i)
              for i, (n, row) in enumerate(zip(sizes, rows))]
    scales[1][[3, 50, 51]] = [0.0, np.inf, 1e-40]      # invalid: left unchanged
    scales[1][[7, 8]] = 1e-7                            # steps large enough to clamp at 448
    return codes, scales, rows, ids


def _device_views(codes):
    """Device copies; the last tensor is a view at byte offset 3."""
    bufs = [_dev(c) for c in codes[:-1]]
    pad = np.concatenate([np.array([5, 0xFB, 9], np.uint8), codes[-1]])
    last = _dev(pad)
    return bufs + [last], bufs + [last[3:]]


def test_f8perturb_and_restore_match_oracle():
    codes, scales, rows, ids = _tensor_set()
    bufs, views = _device_views(codes)
    sdev = [_dev(s) for s in scales]
    plan = esopt.QPlan(views, sdev, rows, tensor_ids=ids, format="e4m3")
    assert plan.numel == sum(c.size for c in codes)
    seed, sign, sigma = (1 << 40) + 5, -1, 1e-3
    plan.perturb(seed, sign, sigma)
    torch.cuda.synchronize()
    pert = [_host(v) for v in views]
    plan.restore(seed, sign, sigma)
    torch.cuda.synchronize()
    back = [_host(v) for v in views]
    assert _host(bufs[-1][:3]).tolist() == [5, 0xFB, 9]
    n_exact = n_all = 0
    for i, (c, sc, row, tid) in enumerate(zip(codes, scales, rows, ids)):
        el = np.arange(c.size, dtype=np.uint64)
        rep = _perturb_report(pert[i], c, sc, row, seed, tid, sign, sigma, el)
        print("f8perturb", i, rep)
        assert_f8parity(rep, f"f8perturb tensor {i}")
        rep = _perturb_report(back[i], pert[i], sc, row, seed, tid, sign, sigma, el, restore=True)
        print("f8restore", i, rep)
        assert_f8parity(rep, f"f8restore tensor {i}")
        # not-a-number codes and invalid rows kept their bytes
        nan = (c & 0x7F) == 0x7F
        assert np.all(pert[i][nan] == c[nan]) and np.all(back[i][nan] == c[nan])
        v0, vb = of.e4m3_decode(c), of.e4m3_decode(back[i])
        fin = np.isfinite(v0)
        n_exact += int(np.sum(vb[fin] == v0[fin]))
        n_all += int(fin.sum())
    # the revert: exact for most codes (inside a binade always, as the oracle)
    print("exact reverts", n_exact / n_all)
    assert n_exact / n_all > 0.85
    assert np.mean(pert[0] != codes[0]) > 0.5
    invalid = np.repeat(np.isin(np.arange(scales[1].size), [3, 50, 51]), 8)[:codes[1].size]
    assert np.all(pert[1][invalid] == codes[1][invalid])
    plan.close()


@pytest.mark.parametrize("flags", [0, esopt.ES_UPDATE_DIV_SIGMA, esopt.ES_REWARDS_ARE_WEIGHTS])
def test_f8update_matches_oracle(flags):
    codes, scales, rows, ids = _tensor_set()
    bufs, views = _device_views(codes)
    sdev = [_dev(s) for s in scales]
    plan = esopt.QPlan(views, sdev, rows, tensor_ids=ids, format="e4m3")
    seeds = [21, 21, 22, 22, 23, 24, 25, 26]
    signs = [1, -1, 1, -1, 1, 1, 1, 1]
    r = np.random.default_rng(4).random(8).astype(np.float32)
    rs = 0xFEEDFACE01234567
    alpha = 5e-4 if flags != esopt.ES_REWARDS_ARE_WEIGHTS else 2e-4
    status = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    plan.update(seeds, signs, _dev(r), alpha, sigma=1e-3, flags=flags, round_seed=rs,
                status_out=status)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    for i, (c, sc, row, tid) in enumerate(zip(codes, scales, rows, ids)):
        el = np.arange(c.size, dtype=np.uint64)
        got = _host(views[i])
        rep = _update_report(got, c, sc, row, tid, seeds, signs, r, alpha, 1e-3, flags, el, rs)
        print("f8update", flags, i, rep)
        assert_f8parity(rep, f"f8update flags={flags} tensor {i}")
        assert np.mean(got != c) > 0.02 or c.size < 100
    plan.close()


def test_f8update_large_population():
    c = _codes(1 << 16, 30)
    sc = _scales(64, 31)
    t = _dev(c)
    plan = esopt.QPlan([t], [_dev(sc)], [1024], format="e4m3")
    seeds = list(range(500, 564))
    r = np.random.default_rng(6).standard_normal(64).astype(np.float32)
    plan.update(seeds, [1] * 64, _dev(r), 2e-3, round_seed=3)
    torch.cuda.synchronize()
    el = np.arange(c.size, dtype=np.uint64)
    rep = _update_report(_host(t), c, sc, 1024, 0, seeds, [1] * 64, r, 2e-3, 0.0, 0, el, 3)
    print("f8update N=64", rep)
    assert_f8parity(rep, "f8update N=64")
    plan.close()


def test_f8_identities():
    c = _codes(50000, 40)
    sc = _scales(50000 // 8 + 1, 41)
    t = _dev(c)
    plan = esopt.QPlan([t], [_dev(sc)], [8], format="e4m3")
    plan.perturb(3, 1, 0.0)
    plan.update([1, 2], [1, 1], _dev(np.array([0.5, 0.5], np.float32)), 5e-3)      # equal rewards
    plan.update([1, 2], [1, 1], _dev(np.array([0.1, 0.9], np.float32)), 0.0)       # alpha 0
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    plan.update([1, 2], [1, 1], _dev(np.array([0.1, np.nan], np.float32)), 5e-3, status_out=status)
    torch.cuda.synchronize()
    assert int(status.item()) == 1
    np.testing.assert_array_equal(_host(t), c)
    plan.close()
    with pytest.raises(ValueError):
        esopt.QPlan([t], [_dev(sc)], [8], format="e5m2")
    with pytest.raises(ValueError):
        esopt.QPlan([t.view(torch.int8)], [_dev(sc)], [8], format="e4m3")


@pytest.mark.parametrize("shape", [(256, 2, 1), (512, 8, 3), (1024, 8, 8)])
def test_f8_results_do_not_depend_on_launch_shape(shape, monkeypatch):
    codes, scales, rows, ids = _tensor_set()
    r = _dev(np.array([0.3, 0.9, 0.1, 0.5], np.float32))

    def run():
        bufs, views = _device_views(codes)
        plan = esopt.QPlan(views, [_dev(s) for s in scales], rows, tensor_ids=ids, format="e4m3")
        plan.perturb(9, 1, 1e-3)
        plan.update([1, 2, 2, 5], [1, 1, -1, 1], r, 5e-4, round_seed=11)
        plan.restore(9, 1, 1e-3)
        torch.cuda.synchronize()
        out = [_host(v) for v in views]
        plan.close()
        return out

    ref = run()
    monkeypatch.setenv("ESOPT_THREADS", str(shape[0]))
    monkeypatch.setenv("ESOPT_QGROUPS", str(shape[1]))
    monkeypatch.setenv("ESOPT_UPDATE_WG_PER_CU", str(shape[2]))
    got = run()
    for a, b in zip(ref, got):
        np.testing.assert_array_equal(a, b)


def test_f8_checksum_matches_oracle():
    codes, scales, rows, ids = _tensor_set()
    bufs, views = _device_views(codes)
    plan = esopt.QPlan(views, [_dev(s) for s in scales], rows, tensor_ids=ids, format="e4m3")
    plan.perturb(77, 1, 1e-3)
    torch.cuda.synchronize()
    exp = 0
    for v, tid in zip(views, ids):
        exp = (exp + oracle.qchecksum(_host(v).view(np.int8), tid)) & ((1 << 64) - 1)
    assert plan.checksum() == exp
    plan.close()


@pytest.mark.parametrize("case", range(3))
def test_random_f8_layout(case, monkeypatch):
    rng = np.random.default_rng(3000 + case)
    threads, groups = [(256, 4), (512, 8), (1024, 4)][case]
    monkeypatch.setenv("ESOPT_THREADS", str(threads))
    monkeypatch.setenv("ESOPT_QGROUPS", str(groups))
    n_t = int(rng.integers(1, 12))
    sizes = [int(x) for x in rng.integers(1, 300_000, n_t)]
    rows = [int(rng.choice([0, 8, 24, 64, 1024, 5120])) for _ in range(n_t)]
    offsets = [int(x) for x in rng.integers(0, 17, n_t)]
    ids = [int(x) for x in rng.choice(1 << 20, n_t, replace=False)]
    codes = [_codes(n, 3100 + 17 * case + i) for i, n in enumerate(sizes)]
    scales = [_scales(1 if r == 0 else -(-n // r), 3200 + i) for i, (n, r) in
              enumerate(zip(sizes, rows))]
    starts, cur = [], 0
    for n, off in zip(sizes, offsets):
        cur = (cur + 15) // 16 * 16 + off
        starts.append(cur)
        cur += n
    flat = np.zeros(cur + 16, np.uint8)
    for s0, c in zip(starts, codes):
        flat[s0:s0 + c.size] = c
    buf = _dev(flat)
    views = [buf[s0:s0 + n] for s0, n in zip(starts, sizes)]
    plan = esopt.QPlan(views, [_dev(s) for s in scales], rows, tensor_ids=ids, format="e4m3")
    seeds = [int(x) for x in rng.integers(0, 1 << 62, 3)]
    r = rng.random(3).astype(np.float32)
    plan.perturb(seeds[0], -1, 1e-3)
    torch.cuda.synchronize()
    c1 = [_host(v) for v in views]
    plan.update(seeds, [1, 1, 1], _dev(r), 5e-4, round_seed=case)
    torch.cuda.synchronize()
    c2 = [_host(v) for v in views]
    plan.close()
    full = _host(buf)
    mask = np.ones(full.size, bool)
    for s0, n in zip(starts, sizes):
        mask[s0:s0 + n] = False
    assert np.all(full[mask] == flat[mask])
    for i, (tid, row, sc) in enumerate(zip(ids, rows, scales)):
        el = np.arange(sizes[i], dtype=np.uint64)
        assert_f8parity(_perturb_report(c1[i], codes[i], sc, row, seeds[0], tid, -1, 1e-3, el),
                        f"case {case} tensor {i} perturb")
        assert_f8parity(_update_report(c2[i], c1[i], sc, row, tid, seeds, [1, 1, 1], r, 5e-4,
                                       0.0, 0, el, case), f"case {case} tensor {i} update")


def _samples(n, rng, k=256):
    fixed = [0, 1, 2, 15, 16, 17, n // 2, n - 17, n - 16, n - 2, n - 1]
    idx = np.concatenate([np.array([i for i in fixed if 0 <= i < n], dtype=np.int64),
                          rng.integers(0, n, size=min(k, n))])
    return np.unique(idx)


def test_f8_27b_set_sampled():
    """The 27B-shaped set as per-row E4M3 codes (22.7 G codes) in the
    benchmark's launch configuration: perturb, restore and the N = 32 update
    on sampled codes of every tensor against the oracle."""
    W = wl.WORKLOADS["dense-27b"]
    flat, views, scales, rows = wl.device_f8params(W)
    plan = esopt.QPlan(views, scales, rows, format="e4m3")
    assert plan.numel == W.n_params
    rng = np.random.default_rng(12)
    idx = [_samples(v.numel(), rng) for v in views]
    idx_dev = [torch.from_numpy(i).cuda() for i in idx]
    sc_host = [_host(s) for s in scales]

    def gather():
        torch.cuda.synchronize()
        return [_host(v.index_select(0, i)) for v, i in zip(views, idx_dev)]
    c0 = gather()
    seed, sigma = 4321, W.sigma0
    plan.perturb(seed, 1, sigma)
    c1 = gather()
    plan.restore(seed, 1, sigma)
    c2 = gather()
    seeds = list(W.seeds)
    r = wl.rewards(W, n=len(seeds))
    plan.update(seeds, list(W.signs), _dev(r), W.alpha, sigma=sigma, round_seed=7)
    c3 = gather()
    plan.close()
    del flat, views
    torch.cuda.empty_cache()
    bad = 0
    for t, el_i in enumerate(idx):
        el = el_i.astype(np.uint64)
        for rep in (_perturb_report(c1[t], c0[t], sc_host[t], rows[t], seed, t, 1, sigma, el),
                    _perturb_report(c2[t], c1[t], sc_host[t], rows[t], seed, t, 1, sigma, el,
                                    restore=True),
                    _update_report(c3[t], c2[t], sc_host[t], rows[t], t, seeds, list(W.signs), r,
                                   W.alpha, sigma, 0, el, 7)):
            bad += rep["bad"]
            assert rep["bad"] == 0, (t, rep)
    assert bad == 0


def test_f8_generation_replay_is_bit_exact():
    """Four generations of the driver on the tiny set as E4M3 codes are
    rebuilt bit for bit from their records (seeds, signs, rewards, sigma,
    alpha, rounding seed), and the update-only replay matches the oracle's
    chain of updates to the fp8 parity bar (each link checked against the
    oracle applied to the GPU's previous codes)."""
    from paper_2608_17310_amd.generation import run_generation, replay, antithetic_seeds
    W = wl.TINY
    host = wl.host_f8params(W)

    def fresh():
        codes = [_dev(c) for c, _, _ in host]
        return codes, esopt.QPlan(codes, [_dev(s) for _, s, _ in host],
                                  [r for _, _, r in host], format="e4m3")
    codes, plan = fresh()
    rng = np.random.default_rng(12)
    records = []
    for t in range(4):
        seeds, signs = antithetic_seeds(50 * t, 3)
        records.append(run_generation(plan, seeds, signs, 1e-3, 5e-4,
                                      evaluate=lambda i: rng.random(), round_seed=500 + t))
    torch.cuda.synchronize()
    live = [_host(c) for c in codes]
    assert any(np.mean(a != c) > 0.05 for a, (c, _, _) in zip(live, host))
    plan.close()
    codes2, plan2 = fresh()
    replay(plan2, records)
    torch.cuda.synchronize()
    for a, b in zip(live, codes2):
        np.testing.assert_array_equal(a, _host(b))
    plan2.close()
    # update-only replay, one update at a time against the oracle
    codes3, plan3 = fresh()
    prev = [c.copy() for c, _, _ in host]
    for rec in records:
        replay(plan3, [rec], with_perturbations=False)
        torch.cuda.synchronize()
        for tid, ((_, sc, row), dev) in enumerate(zip(host, codes3)):
            got = _host(dev)
            el = np.arange(got.size, dtype=np.uint64)
            rep = _update_report(got, prev[tid], sc, row, tid, rec.seeds, rec.signs,
                                 np.array(rec.rewards, np.float32), rec.alpha, rec.sigma, 0, el,
                                 rec.round_seed)
            assert_f8parity(rep, f"replayed update tensor {tid}")
            prev[tid] = got
    plan3.close()
