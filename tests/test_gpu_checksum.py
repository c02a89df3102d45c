"""es_plan_checksum through the C ABI, bit for bit against the oracle: ragged
plans with tensors at every alignment and empty tensors, shards whose
checksums add up to the whole tensor's, independence from the launch shape,
the stream-ordered `out` form on a side stream, the 0.5B-shaped set in full,
and a generation log whose recorded checksums replay verifies."""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_17310_amd import esopt, workloads as wl
from paper_2608_17310_amd.generation import (run_generation, replay, antithetic_seeds,
                                             ReplayMismatch)
from parity import to_device, to_host

pytestmark = pytest.mark.gpu

M = (1 << 64) - 1


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)


def _ragged():
    """Tensors of ragged sizes placed at 2-byte, 16-byte and tile-crossing
    offsets of one buffer (the bytes between them never read)."""
    sizes = [0, 1, 7, 8, 4097, 65536 + 3, 300_001, 1 << 20, 2]
    pads = [0, 3, 1, 8, 5, 0, 64, 7, 1]
    total = sum(sizes) + sum(pads) + 8
    buf = torch.full((total,), 7.0, dtype=torch.bfloat16, device="cuda")
    views, bits, cur = [], [], 0
    for i, (n, pad) in enumerate(zip(sizes, pads)):
        cur += pad
        b = wl.random_bf16_bits(n, 70 + i)
        v = buf[cur:cur + n]
        if n:
            v.copy_(to_device(b))
        views.append(v)
        bits.append(b)
        cur += n
    ids = [11, 0, 5, (1 << 32) - 1, 3, 77, 2, 9, 1000]
    return buf, views, bits, ids


def test_ragged_plan_matches_oracle():
    buf, views, bits, ids = _ragged()
    with esopt.Plan(views, tensor_ids=ids) as p:
        got = p.checksum()
    assert got == oracle.plan_checksum(list(zip(bits, ids, [0] * len(ids))))
    # one element changed changes it; the bytes around the tensors do not count
    buf.fill_(3.0)
    for v, b in zip(views, bits):
        if b.size:
            v.copy_(to_device(b))
    with esopt.Plan(views, tensor_ids=ids) as p:
        assert p.checksum() == got
        views[6][123] = -views[6][123] if float(views[6][123]) != 0 else 1.0
        assert p.checksum() != got


def test_shard_checksums_add_up_to_the_whole_tensor():
    n = 3_000_017
    bits = wl.random_bf16_bits(n, 71)
    whole = to_device(bits)
    with esopt.Plan([whole], tensor_ids=[4]) as p:
        ref = p.checksum()
    assert ref == oracle.checksum(bits, 4)
    cuts = [0, 1_000_000, 2_000_008, 2_999_992, n]
    total = 0
    for (a, b), pad in zip(zip(cuts, cuts[1:]), [0, 3, 120, 1]):
        buf = torch.zeros(b - a + pad + 8, dtype=torch.bfloat16, device="cuda")
        shard = buf[pad:pad + b - a]
        shard.copy_(to_device(bits[a:b]))
        with esopt.Plan([shard], tensor_ids=[4], offsets=[a]) as p:
            c = p.checksum()
        assert c == oracle.checksum(bits[a:b], 4, a)
        total = (total + c) & M
    assert total == ref


@pytest.mark.parametrize("shape", [("256", "4", "1"), ("512", "8", "3"), ("1024", "4", "32")])
def test_launch_shape_does_not_change_it(shape, monkeypatch):
    _, views, bits, ids = _ragged()
    with esopt.Plan(views, tensor_ids=ids) as p:
        ref = p.checksum()
    t, u, wg = shape
    monkeypatch.setenv("ESOPT_THREADS", t)
    monkeypatch.setenv("ESOPT_GROUPS", u)
    monkeypatch.setenv("ESOPT_UPDATE_WG_PER_CU", wg)
    with esopt.Plan(views, tensor_ids=ids) as p:
        assert p.checksum() == ref


def test_out_tensor_on_a_side_stream():
    _, views, bits, ids = _ragged()
    side = torch.cuda.Stream()
    out = torch.zeros(1, dtype=torch.int64, device="cuda")
    with esopt.Plan(views, tensor_ids=ids) as p:
        ref = p.checksum()
        side.wait_stream(torch.cuda.current_stream())
        p.perturb(5, 1, 1e-3, stream=side)
        r = p.checksum(out=out, stream=side)
        p.restore(5, 1, 1e-3, stream=side)
        assert r is out
        side.synchronize()
        after = p.checksum()
    exp = oracle.plan_checksum([(to_host(v), i, 0) for v, i in zip(views, ids)])
    assert after == exp
    assert (after == ref) == all(np.array_equal(to_host(v), b) for v, b in zip(views, bits))
    assert (int(out.item()) & M) != ref


def test_full_0_5b_set_matches_oracle():
    W = wl.WORKLOADS["dense-0.5b"]
    flat, views = wl.device_params(W)
    with esopt.Plan(views) as p:
        got = p.checksum()
    torch.cuda.synchronize()
    exp = 0
    for i, v in enumerate(views):
        exp = (exp + oracle.checksum(to_host(v), i)) & M
    assert got == exp


def test_replay_verifies_recorded_checksums():
    W = wl.TINY
    host = wl.host_params(W)
    live = [to_device(b, s) for b, s in zip(host, W.shapes)]
    rng = np.random.default_rng(4)
    records = []
    with esopt.Plan(live) as p:
        for t in range(3):
            seeds, signs = antithetic_seeds(10 * t, 2)
            records.append(run_generation(p, seeds, signs, 1e-3, 5e-4,
                                          evaluate=lambda i: rng.random(), checksum=True))
        final = p.checksum()
    assert records[-1].checksum == final
    assert all(r.checksum is not None for r in records)
    again = [to_device(b, s) for b, s in zip(host, W.shapes)]
    with esopt.Plan(again) as p:
        replay(p, records)
        assert p.checksum() == final
    bad = [to_device(b, s) for b, s in zip(host, W.shapes)]
    records[1].rewards[0] += 0.25          # a wrong log entry
    with esopt.Plan(bad) as p, pytest.raises(ReplayMismatch, match="generation 1"):
        replay(p, records)


def _qset():
    """int8 codes of ragged sizes, one at byte offset 3 of its buffer, with
    per-row and per-tensor scales."""
    rng = np.random.default_rng(12)
    sizes, rows = [1, 15, 16 * 4096 + 5, 65536 * 2 + 7, 300_001], [0, 8, 16, 1024, 0]
    codes = [rng.integers(-128, 128, size=n).astype(np.int8) for n in sizes]
    bufs = [torch.from_numpy(np.concatenate([np.zeros(3, np.int8), c])).cuda() for c in codes]
    views = [b[3:] if i == 3 else b[3:].clone() for i, b in enumerate(bufs)]
    scales = [torch.full((1 if r == 0 else -(-n // r),), 2e-4, dtype=torch.float32, device="cuda")
              for n, r in zip(sizes, rows)]
    return codes, views, scales, rows, [4, 0, 9, 2, 77]


def test_int8_plan_checksum_matches_oracle():
    codes, views, scales, rows, ids = _qset()
    with esopt.QPlan(views, scales, rows, tensor_ids=ids) as p:
        got = p.checksum()
        p.perturb(3, 1, 1e-3)
        moved = p.checksum()
    torch.cuda.synchronize()
    exp = 0
    for c, i in zip(codes, ids):
        exp = (exp + oracle.qchecksum(c, i)) & M
    assert got == exp
    after = 0
    for v, i in zip(views, ids):
        after = (after + oracle.qchecksum(v.cpu().numpy(), i)) & M
    assert moved == after != got


def test_int8_replay_verifies_recorded_checksums():
    codes, views, scales, rows, ids = _qset()
    rng = np.random.default_rng(5)
    with esopt.QPlan(views, scales, rows, tensor_ids=ids) as p:
        records = [run_generation(p, *antithetic_seeds(20 * t, 2), 1e-3, 5e-4,
                                  evaluate=lambda i: rng.random(), checksum=True,
                                  round_seed=500 + t) for t in range(3)]
        final = p.checksum()
    assert records[-1].checksum == final
    _, again, scales2, _, _ = _qset()
    with esopt.QPlan(again, scales2, rows, tensor_ids=ids) as p:
        replay(p, records)
        assert p.checksum() == final
