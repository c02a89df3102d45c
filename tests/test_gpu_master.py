"""Updates into binary32 master copies (es_plan_set_master, ES_UPDATE_MASTER):
the masters against the oracle's update_master within the bar derived from
the kernel's arithmetic (tests/parity.py), the bf16 values bit for bit the
nearest-even rounding of the GPU's masters (and never read: they start as
garbage), independence from the generation's perturbation walk, the cases
that add nothing, blocks and shards bit-identical to the whole tensors,
es_update_noalloc and HIP-graph replays equal to es_update, validation, and
the generation driver with replay from updates alone."""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_17310_amd import esopt, workloads as wl
from paper_2608_17310_amd.generation import replay, run_generation
from parity import assert_master_parity, master_report, master_tolerance, to_host

pytestmark = pytest.mark.gpu

M = esopt.ES_UPDATE_MASTER
SHAPES = [70_000, 4097, 77, 65536 * 3 + 11]
PADS = [0, 3, 8, 1]                          # bf16 views at assorted offsets


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)


def _masters(seed):
    rng = np.random.default_rng(seed)
    return [(rng.standard_normal(n) * 0.02).astype(np.float32) for n in SHAPES]


def _setup(seed, garbage=1):
    """bf16 views (garbage values: they are written, never read) and float32
    master tensors on the device, and a plan with the masters attached."""
    ms = _masters(seed)
    views = []
    for i, (n, pad) in enumerate(zip(SHAPES, PADS)):
        buf = torch.zeros(n + pad + 8, dtype=torch.bfloat16, device="cuda")
        v = buf[pad:pad + n]
        v.view(torch.int16).copy_(torch.from_numpy(
            wl.random_bf16_bits(n, 1000 * garbage + i).view(np.int16)).cuda())
        views.append(v)
    mdev = [torch.from_numpy(m).cuda() for m in ms]
    plan = esopt.Plan(views, tensor_ids=[3, 0, 9, 1 << 31])
    plan.set_master(mdev)
    return plan, views, mdev, ms


def _assert_same(ma, va, mb, vb):
    """Masters and bf16 values of two plans equal bit for bit."""
    for x, y in zip(ma, mb):
        np.testing.assert_array_equal(x.cpu().numpy().view(np.uint32),
                                      y.cpu().numpy().view(np.uint32))
    for x, y in zip(va, vb):
        np.testing.assert_array_equal(to_host(x), to_host(y))


def _rne(m):
    return oracle.f64_to_bf16_rne(np.asarray(m, np.float32).astype(np.float64))


@pytest.mark.parametrize("flags,sigma", [(0, 1e-3), (esopt.ES_UPDATE_DIV_SIGMA, 2e-3)],
                         ids=["alpha/G", "alpha/(G sigma)"])
def test_master_update_matches_oracle(flags, sigma):
    plan, views, mdev, ms = _setup(10)
    seeds, signs = [5, 5, 6, 7, 8, 8], [1, -1, 1, 1, 1, -1]
    r = np.array([0.7, 0.2, 0.9, 0.4, 0.1, 0.6], np.float32)
    plan.update(seeds, signs, torch.from_numpy(r).cuda(), 5e-4, sigma=sigma, flags=flags | M)
    torch.cuda.synchronize()
    z, _ = oracle.zscore(r)
    c = oracle.update_coefficient(5e-4, sigma, len(seeds), flags)
    d, w = oracle.member_weights(seeds, signs, z, c)
    live = [(sd, wd) for sd, wd in zip(d, w) if wd != 0.0]
    for i, (tid, m0) in enumerate(zip(plan.tensor_ids, ms)):
        exp, bits, st = oracle.update_master(m0, tid, seeds, signs, r, 5e-4, sigma, flags=flags)
        got = mdev[i].cpu().numpy()
        el = np.arange(m0.size, dtype=np.uint64)
        rep = master_report(got, exp, master_tolerance(exp, live, tid, el))
        print("master", i, rep)
        assert_master_parity(rep, f"master tensor {i}")
        np.testing.assert_array_equal(to_host(views[i]), _rne(got))
        assert np.mean(got != m0) > 0.99
    plan.close()


def test_the_walk_does_not_reach_the_masters():
    """A generation's perturbations, swaps and an unreverted last member
    leave the masters and the rewritten bf16 values exactly those of the
    update alone on other bf16 garbage."""
    pa, va, ma, _ = _setup(20, garbage=2)
    pb, vb, mb, _ = _setup(20, garbage=3)
    seeds, signs = [1, 2, 3, 4], [1, 1, -1, 1]
    r = torch.tensor([0.3, 0.9, 0.5, 0.1], device="cuda")
    pa.perturb(1, 1, 1e-3)
    for a, b, sa, sb in zip(seeds, seeds[1:], signs, signs[1:]):
        pa.swap(a, sa, b, sb, 1e-3)
    pa.update(seeds, signs, r, 5e-4, flags=M)
    pb.update(seeds, signs, r, 5e-4, flags=M)
    torch.cuda.synchronize()
    _assert_same(ma, va, mb, vb)
    pa.close()
    pb.close()


@pytest.mark.parametrize("rewards,status", [([0.5, 0.5], 0), ([0.5, float("nan")], 1)],
                         ids=["equal rewards", "non-finite reward"])
def test_nothing_to_add_still_rewrites_the_working_copy(rewards, status):
    plan, views, mdev, ms = _setup(30)
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    plan.perturb(7, 1, 1e-3)
    plan.update([7, 8], [1, 1], torch.tensor(rewards, device="cuda"), 5e-4, flags=M,
                status_out=st)
    torch.cuda.synchronize()
    assert int(st.item()) == status
    for v, m, m0 in zip(views, mdev, ms):
        np.testing.assert_array_equal(m.cpu().numpy(), m0)          # masters untouched
        np.testing.assert_array_equal(to_host(v), _rne(m0))         # bf16 rewritten
    plan.close()


def test_blocks_and_shards_equal_the_whole_tensor():
    rows, cols = 96, 1024
    rng = np.random.default_rng(40)
    m0 = (rng.standard_normal((rows, cols)) * 0.02).astype(np.float32)
    r = torch.tensor([0.2, 0.8, 0.5], device="cuda")
    seeds, signs = [3, 4, 5], [1, -1, 1]

    def run(plan, masters, views):
        plan.set_master(masters)
        plan.perturb(3, 1, 1e-3)
        plan.update(seeds, signs, r, 5e-4, flags=M)
        torch.cuda.synchronize()
        return [m.cpu().numpy() for m in masters], [to_host(v) for v in views]

    whole = torch.zeros(rows, cols, dtype=torch.bfloat16, device="cuda")
    wm = torch.from_numpy(m0.copy()).cuda()
    with esopt.Plan([whole.reshape(-1)], tensor_ids=[6]) as p:
        (gm,), (gb,) = run(p, [wm.reshape(-1)], [whole.reshape(-1)])
    gm, gb = gm.reshape(rows, cols), gb.reshape(rows, cols)
    # four column blocks (strided: the row-map launch)
    for k in range(4):
        c0 = 256 * k
        blk = torch.zeros(rows, 256, dtype=torch.bfloat16, device="cuda")
        bm = torch.from_numpy(np.ascontiguousarray(m0[:, c0:c0 + 256])).cuda()
        with esopt.Plan(blocks=[esopt.Block(blk, 6, cols, 0, c0)]) as p:
            (m,), (b,) = run(p, [bm], [blk])
        np.testing.assert_array_equal(m.reshape(rows, 256), gm[:, c0:c0 + 256])
        np.testing.assert_array_equal(b.reshape(rows, 256), gb[:, c0:c0 + 256])
    # a row shard (offset8), its bf16 view only 2-byte aligned
    buf = torch.zeros(40 * cols + 1, dtype=torch.bfloat16, device="cuda")
    sh = buf[1:]
    sm = torch.from_numpy(np.ascontiguousarray(m0[56:])).cuda().reshape(-1)
    with esopt.Plan([sh], tensor_ids=[6], offsets=[56 * cols]) as p:
        (m,), (b,) = run(p, [sm], [sh])
    np.testing.assert_array_equal(m, gm[56:].reshape(-1))
    np.testing.assert_array_equal(b, gb[56:].reshape(-1))


def test_noalloc_and_graph_replays_equal_the_update():
    pa, va, ma, _ = _setup(50)
    pb, vb, mb, _ = _setup(50)
    seeds, signs = [1, 2, 3], [1, -1, 1]
    r = torch.tensor([0.4, 0.1, 0.8], device="cuda")
    pa.update(seeds, signs, r, 5e-4, flags=M)
    pb.update_noalloc(seeds, signs, r, 5e-4, flags=M)
    torch.cuda.synchronize()
    _assert_same(ma, va, mb, vb)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        pa.update(seeds, signs, r, 5e-4, flags=M)
    torch.cuda.synchronize()
    for _ in range(3):
        g.replay()
        torch.cuda.synchronize()
        pb.update(seeds, signs, r, 5e-4, flags=M)
        torch.cuda.synchronize()
        _assert_same(ma, va, mb, vb)
    pa.close()
    pb.close()


def test_master_arguments_are_checked():
    plan, views, mdev, _ = _setup(60)
    r = torch.tensor([0.4, 0.1], device="cuda")
    bytes_with = plan.device_bytes
    with pytest.raises(ValueError):
        plan.set_master(mdev[:2])                                   # count (binding)
    lib = esopt.load()
    import ctypes
    arr = (ctypes.c_void_p * 4)(*[m.data_ptr() for m in mdev])
    assert lib.es_plan_set_master(plan.handle, arr, 3) == esopt.ES_ERR_INVALID_ARG
    big = torch.zeros(SHAPES[0] + 4, device="cuda")
    arr[0] = big.data_ptr() + 4                                      # 4-byte aligned only
    assert lib.es_plan_set_master(plan.handle, arr, 4) == esopt.ES_ERR_ALIGN
    arr[0] = views[0].data_ptr() - views[0].data_ptr() % 16 + 16    # inside a bf16 tensor
    assert lib.es_plan_set_master(plan.handle, arr, 4) != esopt.ES_OK
    arr[0] = 0
    assert lib.es_plan_set_master(plan.handle, arr, 4) == esopt.ES_ERR_INVALID_ARG
    with pytest.raises(esopt.EsError):                               # with stochastic rounding
        plan.update([1, 2], [1, 1], r, 5e-4, flags=M | esopt.ES_UPDATE_STOCHASTIC_ROUND)
    with pytest.raises(esopt.EsError):                               # a revert is pointless
        plan.restore_update(1, 1, 1e-3, [1, 2], [1, 1], r, 5e-4, flags=M)
    plan.set_master(None)                                            # detach
    assert plan.device_bytes == bytes_with - 8 * plan.tiles
    with pytest.raises(esopt.EsError):
        plan.update([1, 2], [1, 1], r, 5e-4, flags=M)
    plan.close()
    codes = torch.zeros(64, dtype=torch.int8, device="cuda")
    with esopt.QPlan([codes], [torch.ones(1, device="cuda")], [0]) as q:
        with pytest.raises(esopt.EsError):
            q.update([1, 2], [1, 1], r, 5e-4, flags=M)


def test_generation_driver_and_replay_from_updates():
    plan, views, mdev, ms = _setup(70)
    recs = []
    for g in range(3):
        seeds = [100 * g + i for i in range(4)]
        scores = [0.3, 0.9, 0.1, 0.5]
        recs.append(run_generation(plan, seeds, [1, 1, 1, 1], 1e-3, 5e-4,
                                   lambda i, s=scores: s[i], checksum=True))
        assert recs[-1].flags & M
    torch.cuda.synchronize()
    final_m = [m.cpu().numpy() for m in mdev]
    final_b = [to_host(v) for v in views]
    plan.close()
    pc, vc, mc, _ = _setup(70, garbage=5)                # other bf16 garbage, same masters
    replay(pc, recs)                                      # updates only; checksums verified
    torch.cuda.synchronize()
    for x, y in zip(mc, final_m):
        np.testing.assert_array_equal(x.cpu().numpy(), y)
    for x, y in zip(vc, final_b):
        np.testing.assert_array_equal(to_host(x), y)
    pc.close()


# ------------------------------------------------- members applied from masters --

def test_perturb_master_matches_oracle_and_leaves_the_masters():
    from parity import assert_parity, perturb_delta, report
    plan, views, mdev, ms = _setup(80)
    for seed, sign, sigma in [(11, 1, 1e-3), (12, -1, 1.5e-3), ((1 << 62) + 3, 1, 2e-3)]:
        plan.perturb_master(seed, sign, sigma)
        torch.cuda.synchronize()
        for i, (tid, m0) in enumerate(zip(plan.tensor_ids, ms)):
            el = np.arange(m0.size, dtype=np.uint64)
            exp = oracle.perturb_master(m0, seed, tid, sign, sigma)
            rep = report(to_host(views[i]), exp, _rne(m0), perturb_delta(seed, tid, sign, sigma, el))
            assert_parity(rep, f"perturb_master tensor {i}")
            np.testing.assert_array_equal(mdev[i].cpu().numpy(), m0)     # masters unchanged
    plan.perturb_master(1, 1, 0.0)                                         # refresh
    torch.cuda.synchronize()
    for v, m0 in zip(views, ms):
        np.testing.assert_array_equal(to_host(v), _rne(m0))
    with pytest.raises(esopt.EsError):
        plan.perturb_master(1, 0, 1e-3)
    plan.set_master(None)
    with pytest.raises(esopt.EsError):                                     # no masters
        plan.perturb_master(1, 1, 1e-3)
    plan.close()


def test_perturb_master_of_bf16_masters_is_es_perturb_bit_for_bit():
    """Masters equal to bf16 values: a member applied from them is es_perturb
    of those bf16 values, bit for bit (one FMA per element on the same
    binary32 value, then nearest-even) -- over full and tail tiles, views at
    odd offsets, a strided block and both signs; zeros of both signs,
    infinities, NaNs with payloads, subnormals and the largest finite values
    among them, in the head, a full tile and the tail."""
    plan, views, mdev, ms = _setup(85)
    bits = [_rne(m) for m in ms]
    special = [0x0000, 0x8000, 0x7F80, 0xFF80, 0x0001, 0x807F, 0x7FC1, 0xFF81, 0x7F81, 0x7F7F,
               0xFF7F, 0x0080]
    for at in (0, 100_000, bits[3].size - len(special)):
        bits[3][at:at + len(special)] = special
    for d, b in zip(mdev, bits):                     # masters := their bf16 values
        d.copy_(torch.from_numpy((b.astype(np.uint32) << 16).view(np.float32)).cuda())
    twins = [torch.from_numpy(b.view(np.int16)).cuda().view(torch.bfloat16) for b in bits]
    ref = esopt.Plan(twins, tensor_ids=plan.tensor_ids)
    for seed, sign, sigma in [(31, 1, 1e-3), (32, -1, 3e-2), ((1 << 63) + 5, 1, 7e-4)]:
        plan.perturb_master(seed, sign, sigma)
        ref.perturb(seed, sign, sigma)
        torch.cuda.synchronize()
        for v, t in zip(views, twins):
            np.testing.assert_array_equal(to_host(v), to_host(t))
        for t, b in zip(twins, bits):                # the twins back at the masters' values
            t.view(torch.int16).copy_(torch.from_numpy(b.view(np.int16)).cuda())
    ref.close()
    plan.close()
    rows, cols = 40, 1000
    b0 = _rne((np.random.default_rng(86).standard_normal((rows, 2 * cols)) * 0.02))
    blk = torch.zeros(rows, cols, dtype=torch.bfloat16, device="cuda")
    twin = torch.from_numpy(np.ascontiguousarray(b0[:, 600:600 + cols]).view(np.int16)).cuda()
    twin = twin.view(torch.bfloat16)
    m = (np.ascontiguousarray(b0[:, 600:600 + cols]).astype(np.uint32) << 16).view(np.float32)
    with esopt.Plan(blocks=[esopt.Block(blk, 4, 2 * cols, 0, 600)]) as p, \
            esopt.Plan(blocks=[esopt.Block(twin, 4, 2 * cols, 0, 600)]) as q:
        p.set_master([torch.from_numpy(m.reshape(-1).copy()).cuda()])
        p.perturb_master(77, -1, 2e-3)
        q.perturb(77, -1, 2e-3)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(to_host(blk), to_host(twin))


def _bf16_twins(x0, make_plan, shape):
    """A plan over bf16 values x0 with binary32 masters equal to them, and a
    plan over a copy of x0: es_perturb_master on the first and es_perturb on
    the second must agree bit for bit."""
    a = torch.from_numpy(x0.view(np.int16).reshape(shape)).cuda().view(torch.bfloat16)
    b = a.clone()
    m = torch.from_numpy((x0.astype(np.uint32) << 16).view(np.float32).copy()).cuda()
    pa, pb = make_plan(a), make_plan(b)
    pa.set_master([m])
    return pa, pb, a, b


@pytest.mark.parametrize("kind", ["shard", "block"])
def test_perturb_master_across_element_2_34_is_es_perturb_bit_for_bit(kind):
    """Whole-tensor indices from below to above 2^34, where the counter's high
    word changes (mid-tile for the block's rows): with bf16-representable
    masters every value is es_perturb's, full tiles, tails and row maps."""
    tid = 3
    if kind == "shard":
        a0, n = (1 << 34) - 200_000, 500_017
        x0 = wl.random_bf16_bits(n, 88)
        pa, pb, va, vb = _bf16_twins(
            x0, lambda t: esopt.Plan([t], tensor_ids=[tid], offsets=[a0]), (n,))
    else:
        row_len, rows, cols = (1 << 20) + 4096, 256, 1024     # 512 KB: full tiles too
        row0 = (1 << 34) // row_len - rows // 2
        col0 = (1 << 34) - ((1 << 34) // row_len) * row_len - 512
        x0 = wl.random_bf16_bits(rows * cols, 89)
        pa, pb, va, vb = _bf16_twins(
            x0, lambda t: esopt.Plan(blocks=[esopt.Block(t, tid, row_len, row0, col0)]),
            (rows, cols))
    pa.perturb_master(61, -1, 1.5e-3)
    pb.perturb(61, -1, 1.5e-3)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(to_host(va), to_host(vb))
    assert np.mean(to_host(va) != x0) > 0.9
    pa.close()
    pb.close()


def test_a_candidate_does_not_depend_on_the_ones_before_it():
    pa, va, _, _ = _setup(81, garbage=2)
    pb, vb, _, _ = _setup(81, garbage=3)
    for sd in (5, 6, 7):
        pa.perturb_master(sd, 1, 1e-3)
    pb.perturb_master(7, 1, 1e-3)
    torch.cuda.synchronize()
    for x, y in zip(va, vb):
        np.testing.assert_array_equal(to_host(x), to_host(y))
    pa.close()
    pb.close()


def test_perturb_master_replays_from_a_hip_graph():
    """With sigma > 0 a member applied from the masters uses no scratch, so a
    captured walk of members replays: each replay, after eager passes that
    leave other values behind, gives the eager result of its last member."""
    pa, va, _, _ = _setup(87, garbage=4)
    pb, vb, _, _ = _setup(87, garbage=5)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        pa.perturb_master(41, 1, 1e-3)
        pa.perturb_master(42, -1, 2e-3)
    torch.cuda.synchronize()
    pb.perturb_master(42, -1, 2e-3)
    for k in range(3):
        pa.perturb_master(100 + k, 1, 5e-3)          # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for x, y in zip(va, vb):
            np.testing.assert_array_equal(to_host(x), to_host(y))
    pa.close()
    pb.close()


def test_perturb_master_on_blocks_and_shards():
    rows, cols = 64, 1024
    m0 = (np.random.default_rng(82).standard_normal((rows, cols)) * 0.02).astype(np.float32)
    whole = torch.zeros(rows * cols, dtype=torch.bfloat16, device="cuda")
    with esopt.Plan([whole], tensor_ids=[2]) as p:
        p.set_master([torch.from_numpy(m0.reshape(-1).copy()).cuda()])
        p.perturb_master(9, -1, 1e-3)
        torch.cuda.synchronize()
        ref = to_host(whole).reshape(rows, cols)
    blk = torch.zeros(rows, 384, dtype=torch.bfloat16, device="cuda")
    with esopt.Plan(blocks=[esopt.Block(blk, 2, cols, 0, 512)]) as p:
        p.set_master([torch.from_numpy(np.ascontiguousarray(m0[:, 512:896])).cuda()])
        p.perturb_master(9, -1, 1e-3)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(to_host(blk).reshape(rows, 384), ref[:, 512:896])
    buf = torch.zeros(24 * cols + 3, dtype=torch.bfloat16, device="cuda")
    sh = buf[3:]
    with esopt.Plan([sh], tensor_ids=[2], offsets=[40 * cols]) as p:
        p.set_master([torch.from_numpy(m0[40:].reshape(-1).copy()).cuda()])
        p.perturb_master(9, -1, 1e-3)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(to_host(sh), ref[40:].reshape(-1))


def test_driver_evaluates_each_candidate_at_its_masters_perturbation():
    """run_generation over a plan with masters: while member i is visited the
    bf16 values are exactly the oracle's perturb_master of the masters (on
    sampled elements of every tensor), whatever came before it."""
    plan, views, mdev, ms = _setup(83)
    rng = np.random.default_rng(84)
    picks = [np.unique(rng.integers(0, n, 300)) for n in SHAPES]
    seeds, signs = [21, 21, 22, 23], [1, -1, 1, 1]
    seen = []

    from parity import assert_parity, perturb_delta, report
    parts = ([], [], [], [])

    def evaluate(i):
        torch.cuda.synchronize()
        for k, (tid, idx) in enumerate(zip(plan.tensor_ids, picks)):
            el = idx.astype(np.uint64)
            for lst, x in zip(parts, (to_host(views[k])[idx],
                                      oracle.perturb_master(ms[k][idx], seeds[i], tid, signs[i],
                                                            1e-3, elems=el),
                                      _rne(ms[k][idx]),
                                      perturb_delta(seeds[i], tid, signs[i], 1e-3, el))):
                lst.append(x)
        seen.append(i)
        return float(i)

    run_generation(plan, seeds, signs, 1e-3, 5e-4, evaluate)
    assert seen == [0, 1, 2, 3]
    rep = report(*[np.concatenate(x) for x in parts])
    print("candidates seen by the evaluation:", rep)
    assert_parity(rep, "candidates applied from the masters")
    plan.close()
