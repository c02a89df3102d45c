"""Shards regenerate the whole tensor's noise (es_tensor_t.offset8): a plan
over one shard of a tensor -- a row-parallel slice of a matrix, or a piece of
a flat parameter vector -- gives, bit for bit, the corresponding slice of the
same pass over the whole tensor, for perturb, swap, restore and both update
roundings, whatever the shard's address alignment; and the oracle, asked for
the whole tensor's element numbers, agrees.  This is the part of a
tensor-parallel or sharded deployment one GPU can show: each GPU's plan over
its own shards, with no communication (the rewards aside)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_17310_amd import esopt, workloads as wl
from parity import to_device, to_host, report, assert_parity, perturb_delta, update_delta

pytestmark = pytest.mark.gpu

TID = 7


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)


def _passes(plan, r):
    plan.perturb(3, 1, 1e-3)
    plan.swap(3, 1, 4, -1, 1e-3)
    plan.restore(4, -1, 1e-3)
    plan.update([5, 5, 6, 7], [1, -1, 1, 1], r, 5e-4)
    plan.update([8, 9, 10], [1, 1, 1], r[:3], 5e-4, flags=esopt.ES_UPDATE_STOCHASTIC_ROUND,
                round_seed=99)


def _shards_match(bits, cuts, pad_elems):
    """The whole tensor through one plan; each shard, copied into a buffer at
    `pad_elems` elements past an aligned allocation, through a plan of its
    own with its offset."""
    r = torch.tensor([0.9, 0.1, 0.5, 0.3], device="cuda")
    whole = to_device(bits)
    with esopt.Plan([whole], tensor_ids=[TID]) as p:
        _passes(p, r)
    ref = to_host(whole)
    for (a, b), pad in zip(zip(cuts, cuts[1:]), pad_elems):
        buf = torch.zeros(b - a + pad + 8, dtype=torch.bfloat16, device="cuda")
        shard = buf[pad:pad + b - a]
        shard.copy_(to_device(bits[a:b]))
        with esopt.Plan([shard], tensor_ids=[TID], offsets=[a]) as p:
            _passes(p, r)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(to_host(shard), ref[a:b], err_msg=f"shard [{a}, {b})")
        assert torch.count_nonzero(buf[:pad].float()) == 0
        assert torch.count_nonzero(buf[pad + b - a:].float()) == 0
    return ref


def test_row_shards_of_a_matrix():
    rows, cols = 1024, 5120
    bits = wl.random_bf16_bits(rows * cols, 41)
    cuts = [i * (rows // 4) * cols for i in range(5)]       # 4-way row parallel
    _shards_match(bits, cuts, [0, 1024, 8, 65536 + 8])


def test_uneven_pieces_of_a_flat_vector():
    n = 3_000_017
    bits = wl.random_bf16_bits(n, 42)
    cuts = [0, 1_000_000, 2_000_008, 2_999_992, n]         # offsets multiples of 8
    _shards_match(bits, cuts, [0, 3, 120, 1])                # incl. 2-byte aligned shards


def test_shard_perturb_matches_oracle_at_whole_tensor_indices():
    n = 2_000_000
    bits = wl.random_bf16_bits(n, 43)
    a, b = 1_234_560, n
    shard = to_device(bits[a:b])
    with esopt.Plan([shard], tensor_ids=[TID], offsets=[a]) as p:
        p.perturb(11, -1, 2e-3)
    torch.cuda.synchronize()
    el = np.arange(a, b, dtype=np.uint64)
    exp = oracle.perturb(bits[a:b], 11, TID, -1, 2e-3, elems=el)
    rep = report(to_host(shard), exp, bits[a:b], perturb_delta(11, TID, -1, 2e-3, el))
    print(rep)
    assert_parity(rep, "shard perturb")
    # a shard planned at offset 0 is a different tensor's noise
    plain = to_device(bits[a:b])
    with esopt.Plan([plain], tensor_ids=[TID]) as p:
        p.perturb(11, -1, 2e-3)
    torch.cuda.synchronize()
    assert np.mean(to_host(plain) != to_host(shard)) > 0.5


def test_shard_across_element_2_34_matches_oracle_everywhere():
    """A shard of a 2^34+ element tensor that straddles element 2^34 (where
    the counter's high word changes and the tile split happens), checked
    element by element against the oracle after every pass, without the
    32 GiB tensor itself."""
    a = (1 << 34) - 200_000
    n = 500_017
    el = np.arange(a, a + n, dtype=np.uint64)
    x0 = wl.random_bf16_bits(n, 44)
    buf = torch.zeros(n + 16, dtype=torch.bfloat16, device="cuda")
    shard = buf[8:8 + n]
    shard.copy_(to_device(x0))
    r = np.array([0.2, 0.7, 0.4], np.float32)
    xs = [x0]
    with esopt.Plan([shard], tensor_ids=[TID], offsets=[a]) as p:
        for step in (lambda: p.perturb(11, -1, 1e-3),
                     lambda: p.swap(11, -1, 12, 1, 1e-3),
                     lambda: p.restore(12, 1, 1e-3),
                     lambda: p.update([3, 4, 5], [1, 1, 1], torch.from_numpy(r).cuda(), 5e-4),
                     lambda: p.update([3, 4, 5], [1, 1, 1], torch.from_numpy(r).cuda(), 5e-4,
                                      flags=esopt.ES_UPDATE_STOCHASTIC_ROUND,
                                      round_seed=(1 << 63) + 9)):
            step()
            torch.cuda.synchronize()
            xs.append(to_host(shard))
    assert torch.count_nonzero(buf[:8].float()) == 0
    assert torch.count_nonzero(buf[8 + n:].float()) == 0
    x0, x1, x2, x3, x4, x5 = xs
    upd = update_delta(TID, [3, 4, 5], [1, 1, 1], r, 5e-4, 1e-3, 0, el)
    checks = [
        ("perturb", x1, oracle.perturb(x0, 11, TID, -1, 1e-3, elems=el), x0,
         perturb_delta(11, TID, -1, 1e-3, el)),
        ("swap", x2, oracle.swap(x1, TID, 11, -1, 1e-3, 12, 1, 1e-3, elems=el), x1,
         perturb_delta(11, TID, 1, 1e-3, el) + perturb_delta(12, TID, 1, 1e-3, el)),
        ("restore", x3, oracle.restore(x2, 12, TID, 1, 1e-3, elems=el), x2,
         perturb_delta(12, TID, -1, 1e-3, el)),
        ("update", x4, oracle.update(x3, TID, [3, 4, 5], [1, 1, 1], r, 5e-4, 1e-3,
                                     elems=el)[0], x3, upd),
        ("update_sr", x5, oracle.update(x4, TID, [3, 4, 5], [1, 1, 1], r, 5e-4, 1e-3, elems=el,
                                        flags=esopt.ES_UPDATE_STOCHASTIC_ROUND,
                                        round_seed=(1 << 63) + 9)[0], x4, upd),
    ]
    for name, got, exp, base, delta in checks:
        rep = report(got, exp, base, delta)
        print("shard across 2^34:", name, rep)
        assert_parity(rep, name)


def test_offsets_are_validated():
    t = torch.zeros(64, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(ValueError):
        esopt.Plan([t], offsets=[4])
    with pytest.raises(ValueError):
        esopt.Plan([t], offsets=[8, 16])
