"""Quantized plans over shards (es_qplan_create_shards): every int8 and E4M3
pass over the k-th contiguous range of each tensor, as one GPU of a
tensor-parallel group holds it, leaves exactly the codes the same pass over
the whole tensors leaves there; the shards' checksums add up to the whole
plan's; and a shard's codes match the oracle at the whole-tensor indices
(Section 3: the noise is regenerated from the seed and the element's place
in its tensor)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_17310_amd import esopt
from parity import assert_f8parity, assert_qparity, qreport
from test_gpu_fp8 import _codes as _f8codes, _perturb_report as _f8perturb_report
from test_gpu_quant import _codes as _i8codes, _perturb_expect

pytestmark = pytest.mark.gpu

MASK = (1 << 64) - 1


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)


def _dev(a, pad=0):
    """A device copy of a, at byte offset pad of its allocation."""
    buf = torch.zeros(a.size + pad + 16, dtype=torch.uint8, device="cuda")
    v = buf[pad:pad + a.size]
    v.copy_(torch.from_numpy(np.ascontiguousarray(a).view(np.uint8)).cuda())
    return v


def _host(t):
    return t.cpu().numpy().copy()


# (numel, row, cut points): cuts are multiples of 16 and of the row length;
# shards span several 65 536-code tiles, end ragged, and one is empty
TENSORS = [
    (300_011, 1024, [0, 131_072, 132_096, 300_011]),
    (70_000, 0, [0, 16, 65_552, 70_000]),
    (196_640, 5120, [0, 102_400, 102_400, 196_640]),
    (4_100, 48, [0, 2_064, 2_112, 4_100]),
]
PADS = [0, 3, 16, 1]                 # byte offsets of the shards' copies


def _set(fmt, seed):
    codes, scales = [], []
    rng = np.random.default_rng(seed)
    for i, (n, row, _) in enumerate(TENSORS):
        c = (_i8codes(n, seed + i).view(np.uint8) if fmt == "int8" else _f8codes(n, seed + i))
        codes.append(c)
        lo, hi = (2e-4, 1e-3) if fmt == "int8" else (1.5e-4, 3e-4)
        scales.append(rng.uniform(lo, hi, 1 if row == 0 else -(-n // row)).astype(np.float32))
    return codes, scales


def _shard(codes, scales, k):
    """The k-th shard of every tensor: (codes, scales, offsets)."""
    cs, ss, offs = [], [], []
    for (n, row, cuts), c, s in zip(TENSORS, codes, scales):
        a, b = cuts[k], cuts[k + 1]
        cs.append(c[a:b])
        ss.append(s if row == 0 else s[a // row:-(-b // row)] if b > a else s[:1])
        offs.append(a)
    return cs, ss, offs


def _views(codes, pads, fmt):
    v = [_dev(c, p) for c, p in zip(codes, pads)]
    return v if fmt == "e4m3" else [t.view(torch.int8) for t in v]


def _passes(plan):
    r = torch.tensor([0.4, 0.9, 0.1, 0.6], device="cuda")
    plan.perturb(11, 1, 1e-3)
    plan.restore(11, 1, 1e-3)
    plan.perturb(12, -1, 1.5e-3)
    plan.update([12, 13, 13, 14], [-1, 1, -1, 1], r, 5e-4, sigma=1e-3, round_seed=7)
    plan.update([15, 16], [1, 1], r[:2], 2e-3, sigma=1e-3, round_seed=(1 << 40) + 3,
                flags=esopt.ES_UPDATE_DIV_SIGMA)


@pytest.mark.parametrize("fmt", ["int8", "e4m3"])
def test_shards_leave_the_whole_plans_codes(fmt):
    codes, scales = _set(fmt, 40)
    ids = [3, 0, 77, (1 << 32) - 1]
    rows = [t[1] for t in TENSORS]
    whole = _views(codes, [0] * len(codes), fmt)
    with esopt.QPlan(whole, [torch.from_numpy(s).cuda() for s in scales], rows,
                     tensor_ids=ids, format=fmt) as pw:
        _passes(pw)
        total = pw.checksum()
    torch.cuda.synchronize()
    expect = [_host(t).view(np.uint8) for t in whole]
    sums = 0
    for k in range(3):
        cs, ss, offs = _shard(codes, scales, k)
        views = _views(cs, PADS, fmt)
        with esopt.QPlan(views, [torch.from_numpy(s).cuda() for s in ss], rows, tensor_ids=ids,
                         format=fmt, offsets=offs) as ps:
            assert ps.numel == sum(c.size for c in cs)
            _passes(ps)
            got = ps.checksum()
            sums = (sums + got) & MASK
        torch.cuda.synchronize()
        for i, (v, (n, row, cuts)) in enumerate(zip(views, TENSORS)):
            np.testing.assert_array_equal(_host(v).view(np.uint8), expect[i][cuts[k]:cuts[k + 1]],
                                          err_msg=f"{fmt} shard {k} of tensor {i}")
        assert got == sum(oracle.qchecksum(_host(v), tid, o)
                          for v, tid, o in zip(views, ids, offs)) & MASK
    assert sums == total
    assert np.mean(expect[0] != codes[0]) > 0.3          # the passes moved codes


def test_int8_shard_matches_oracle_at_whole_tensor_indices():
    codes, scales = _set("int8", 50)
    k, i = 2, 0                                           # the last shard of tensor 0
    n, row, cuts = TENSORS[i]
    a, b = cuts[k], cuts[k + 1]
    q = codes[i].view(np.int8)
    v = _dev(q[a:b], 3).view(torch.int8)
    with esopt.QPlan([v], [torch.from_numpy(scales[i][a // row:]).cuda()], [row],
                     tensor_ids=[9], offsets=[a]) as p:
        p.perturb(21, 1, 1e-3)
    torch.cuda.synchronize()
    el = np.arange(a, b, dtype=np.uint64)
    d, ok, tol = _perturb_expect(scales[i], row, 21, 9, 1, 1e-3, el)
    rep = qreport(_host(v).view(np.int8), q[a:b], d, tol, ok)
    print("int8 shard vs oracle:", rep)
    assert_qparity(rep, "int8 shard")


def test_e4m3_shard_matches_oracle_at_whole_tensor_indices():
    codes, scales = _set("e4m3", 60)
    k, i = 1, 1                                           # a middle shard, one scale
    n, row, cuts = TENSORS[i]
    a, b = cuts[k], cuts[k + 1]
    v = _dev(codes[i][a:b], 16)
    with esopt.QPlan([v], [torch.from_numpy(scales[i]).cuda()], [row], tensor_ids=[4],
                     format="e4m3", offsets=[a]) as p:
        p.perturb(22, -1, 1e-3)
    torch.cuda.synchronize()
    el = np.arange(a, b, dtype=np.uint64)
    rep = _f8perturb_report(_host(v), codes[i][a:b], scales[i], row, 22, 4, -1, 1e-3, el)
    print("e4m3 shard vs oracle:", rep)
    assert_f8parity(rep, "e4m3 shard")


def test_shard_offsets_are_checked_by_the_binding_and_the_library():
    q = torch.zeros(64, dtype=torch.int8, device="cuda")
    s = torch.ones(2, device="cuda")
    with pytest.raises(ValueError):
        esopt.QPlan([q], [s], [0], offsets=[0, 16])
    with pytest.raises(ValueError):
        esopt.QPlan([q], [s], [0], offsets=[-16])
    with pytest.raises(esopt.EsError):
        esopt.QPlan([q], [s], [0], offsets=[8])
    with pytest.raises(esopt.EsError):
        esopt.QPlan([q], [s], [32], offsets=[16])
    with pytest.raises(esopt.EsError):
        esopt.QPlan([q], [s], [0], offsets=[(1 << 31) - 64])             # reaches 2^31
    with esopt.QPlan([q], [s], [0], offsets=[(1 << 31) - 80]) as p:       # the last range
        assert p.numel == 64
