"""Rectangular blocks of row-major tensors (es_plan_create_blocks): a plan over
column shards or row-and-column shards of a matrix -- what a GPU holds of a
row-parallel layer under tensor parallelism -- gives, bit for bit, the
corresponding block of the same pass over the whole matrix, for perturb,
swap, restore and both update roundings, at aligned and 2-byte-aligned
addresses, in plans that mix blocks with whole tensors and contiguous shards;
block checksums add up to the whole matrix's; and the oracle, asked for the
whole-tensor indices of the block's elements, agrees element by element,
including a block that straddles element 2^34 and one of more than 2^31
elements (several row pieces)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_17310_amd import esopt, workloads as wl
from parity import to_device, to_host, report, assert_parity, perturb_delta, update_delta

pytestmark = pytest.mark.gpu

TID = 11
M64 = (1 << 64) - 1


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)


def _rewards():
    return torch.tensor([0.9, 0.1, 0.5, 0.3], device="cuda")


def _passes(plan, r):
    plan.perturb(3, 1, 1e-3)
    plan.swap(3, 1, 4, -1, 1e-3)
    plan.restore(4, -1, 1e-3)
    plan.update([5, 5, 6, 7], [1, -1, 1, 1], r, 5e-4)
    plan.update([8, 9, 10], [1, 1, 1], r[:3], 5e-4, flags=esopt.ES_UPDATE_STOCHASTIC_ROUND,
                round_seed=99)


def _whole(bits, rows, cols, tid=TID):
    """The whole matrix through a plan of its own, after every pass."""
    whole = to_device(bits, (rows, cols))
    with esopt.Plan([whole], tensor_ids=[tid]) as p:
        _passes(p, _rewards())
    torch.cuda.synchronize()
    return whole


def _block_buffer(src, pad):
    """A copy of `src` ([r, c] on the GPU) at `pad` elements past an aligned
    allocation, with the padding around it left zero."""
    r, c = src.shape
    buf = torch.zeros(r * c + pad + 8, dtype=torch.bfloat16, device="cuda")
    blk = buf[pad:pad + r * c].view(r, c)
    blk.copy_(src)
    return buf, blk


def _grid_blocks(bits, rows, cols, row_cuts, col_cuts, pads):
    whole = _whole(bits, rows, cols)
    src = to_device(bits, (rows, cols))
    k = 0
    for r0, r1 in zip(row_cuts, row_cuts[1:]):
        for c0, c1 in zip(col_cuts, col_cuts[1:]):
            pad = pads[k % len(pads)]
            k += 1
            buf, blk = _block_buffer(src[r0:r1, c0:c1].contiguous(), pad)
            with esopt.Plan(blocks=[esopt.Block(blk, TID, cols, r0, c0)]) as p:
                _passes(p, _rewards())
            torch.cuda.synchronize()
            assert torch.equal(blk.view(torch.int16), whole[r0:r1, c0:c1].view(torch.int16)), \
                f"block rows [{r0}, {r1}) cols [{c0}, {c1}) pad {pad}"
            n = (r1 - r0) * (c1 - c0)
            assert torch.count_nonzero(buf[:pad].float()) == 0
            assert torch.count_nonzero(buf[pad + n:].float()) == 0


def test_column_shards_of_a_matrix():
    rows, cols = 300, 5120
    bits = wl.random_bf16_bits(rows * cols, 61)
    _grid_blocks(bits, rows, cols, [0, rows], [0, 1280, 2560, 3840, 5120], [0, 1024, 8, 65536 + 8])


def test_row_and_column_blocks_with_ragged_edges():
    """A 3 x 4 grid of blocks of uneven sizes, the narrowest 8 columns wide,
    including 2-byte-aligned copies (element-wise path)."""
    rows, cols = 531, 2200
    bits = wl.random_bf16_bits(rows * cols, 62)
    _grid_blocks(bits, rows, cols, [0, 1, 260, rows], [0, 8, 1000, 2192, cols], [0, 3, 120, 1])


def test_real_shape_column_shard_spans_many_tiles():
    """One of eight column shards of a 5120 x 17408 down-projection ([5120,
    2176], 11 M elements, ~170 full tiles in the strided launch)."""
    rows, cols, k = 5120, 17408, 8
    w = cols // k
    bits = wl.random_bf16_bits(rows * cols, 63)
    whole = _whole(bits, rows, cols)
    src = to_device(bits, (rows, cols))
    for s in (0, 5):
        blk = src[:, s * w:(s + 1) * w].contiguous()
        with esopt.Plan(blocks=[esopt.Block(blk, TID, cols, 0, s * w)]) as p:
            assert p.tiles >= blk.numel() // 65536
            _passes(p, _rewards())
        torch.cuda.synchronize()
        assert torch.equal(blk.view(torch.int16), whole[:, s * w:(s + 1) * w].view(torch.int16))


def test_blocks_mixed_with_tensors_and_shards_in_one_plan():
    """One plan holding a strided block, a whole vector and a contiguous
    shard of a third tensor: each matches its own whole-tensor pass."""
    ra, ca = 96, 1024                               # tensor 1: column block [96, 256] at col 512
    a_bits = wl.random_bf16_bits(ra * ca, 64)
    b_bits = wl.random_bf16_bits(4097, 65)          # tensor 2: whole
    c_bits = wl.random_bf16_bits(70_000, 66)        # tensor 3: elements [8000, 70000)
    wa = _whole(a_bits, ra, ca, tid=1)
    wb = _whole(b_bits, 1, 4097, tid=2)
    wc = _whole(c_bits, 1, 70_000, tid=3)
    a = to_device(a_bits, (ra, ca))[:, 512:768].contiguous()
    b = to_device(b_bits)
    c = to_device(c_bits)[8000:].contiguous()
    blocks = [esopt.Block(a, 1, ca, 0, 512), esopt.Block(b, 2, 4097),
              esopt.Block(c, 3, 70_000, 0, 8000)]
    with esopt.Plan(blocks=blocks) as p:
        _passes(p, _rewards())
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int16), wa[:, 512:768].view(torch.int16))
    assert torch.equal(b.view(torch.int16), wb.view(-1).view(torch.int16))
    assert torch.equal(c.view(torch.int16), wc.view(-1)[8000:].view(torch.int16))


def test_block_checksums_add_up_to_the_whole_matrix():
    rows, cols = 777, 1536
    bits = wl.random_bf16_bits(rows * cols, 67)
    src = to_device(bits, (rows, cols))
    with esopt.Plan([src], tensor_ids=[TID]) as p:
        whole = p.checksum()
    assert whole == oracle.checksum(bits, TID)
    total = 0
    for r0, r1 in ((0, 400), (400, rows)):
        for c0, c1 in ((0, 512), (512, 1024), (1024, cols)):
            blk = src[r0:r1, c0:c1].contiguous()
            with esopt.Plan(blocks=[esopt.Block(blk, TID, cols, r0, c0)]) as p:
                c = p.checksum()
            host = to_host(blk).reshape(r1 - r0, c1 - c0)
            exp = 0
            for i in range(r1 - r0):
                exp = (exp + oracle.checksum(host[i], TID, (r0 + i) * cols + c0)) & M64
            assert c == exp, (r0, c0)
            total = (total + c) & M64
    assert total == whole


def _oracle_steps(xs, el, r):
    """Each pass below checked on its own: the oracle applied to the GPU's
    state before the pass (xs[k - 1]) at whole-tensor indices el, so that a
    legitimate 1-ulp tie of one pass is not carried into the next one's
    expected values."""
    upd = update_delta(TID, [3, 4, 5], [1, 1, 1], r, 5e-4, 1e-3, 0, el)
    return [
        ("perturb", oracle.perturb(xs[0], 11, TID, -1, 1e-3, elems=el), xs[0],
         perturb_delta(11, TID, -1, 1e-3, el)),
        ("swap", oracle.swap(xs[1], TID, 11, -1, 1e-3, 12, 1, 1e-3, elems=el), xs[1],
         perturb_delta(11, TID, 1, 1e-3, el) + perturb_delta(12, TID, 1, 1e-3, el)),
        ("restore", oracle.restore(xs[2], 12, TID, 1, 1e-3, elems=el), xs[2],
         perturb_delta(12, TID, -1, 1e-3, el)),
        ("update", oracle.update(xs[3], TID, [3, 4, 5], [1, 1, 1], r, 5e-4, 1e-3, elems=el)[0],
         xs[3], upd),
        ("update_sr", oracle.update(xs[4], TID, [3, 4, 5], [1, 1, 1], r, 5e-4, 1e-3, elems=el,
                                    flags=esopt.ES_UPDATE_STOCHASTIC_ROUND,
                                    round_seed=(1 << 63) + 9)[0], xs[4], upd),
    ]


def _run_chain(plan, views, r):
    xs = [[to_host(v)] for v in views]
    for step in (lambda: plan.perturb(11, -1, 1e-3),
                 lambda: plan.swap(11, -1, 12, 1, 1e-3),
                 lambda: plan.restore(12, 1, 1e-3),
                 lambda: plan.update([3, 4, 5], [1, 1, 1], torch.from_numpy(r).cuda(), 5e-4),
                 lambda: plan.update([3, 4, 5], [1, 1, 1], torch.from_numpy(r).cuda(), 5e-4,
                                     flags=esopt.ES_UPDATE_STOCHASTIC_ROUND,
                                     round_seed=(1 << 63) + 9)):
        step()
        torch.cuda.synchronize()
        for x, v in zip(xs, views):
            x.append(to_host(v))
    return xs


def _block_indices(rows, cols, row_len, row0, col0):
    i = np.arange(rows, dtype=np.uint64)[:, None]
    j = np.arange(cols, dtype=np.uint64)[None, :]
    return ((np.uint64(row0) + i) * np.uint64(row_len) + np.uint64(col0) + j).ravel()


@pytest.mark.parametrize("pad", [8, 1])
def test_block_matches_oracle_at_whole_tensor_indices_across_2_34(pad):
    """A [64, 1024] block of a tensor with 2^20 + 4096 columns whose rows run
    from below to above whole-tensor element 2^34, which falls inside one of
    the block's rows (the counter's high word changes mid-row and mid-tile),
    checked element by element against the oracle after every pass; pad 1
    puts it at a 2-byte-aligned address (element-wise accesses)."""
    row_len = (1 << 20) + 4096
    rows, cols = 64, 1024
    row0 = (1 << 34) // row_len - rows // 2
    col0 = (1 << 34) - ((1 << 34) // row_len) * row_len - 512   # 2^34 at column 512 of a row
    el = _block_indices(rows, cols, row_len, row0, col0)
    k = int(np.searchsorted(el, 1 << 34))
    assert 0 < k < el.size and el[k] == (1 << 34) and k % cols == 512
    x0 = wl.random_bf16_bits(rows * cols, 68)
    r = np.array([0.2, 0.7, 0.4], np.float32)
    buf, blk = _block_buffer(to_device(x0, (rows, cols)), pad)
    with esopt.Plan(blocks=[esopt.Block(blk, TID, row_len, row0, col0)]) as p:
        (xs,) = _run_chain(p, [blk], r)
    assert torch.count_nonzero(buf[:pad].float()) == 0
    for (name, exp, base, delta), got in zip(_oracle_steps(xs, el, r), xs[1:]):
        rep = report(got, exp, base, delta)
        print(f"block across 2^34 (pad {pad}):", name, rep)
        assert_parity(rep, name)


def test_block_whose_rows_pass_many_multiples_of_2_34():
    """Rows just under 2^32 elements apart: the whole-tensor index passes a
    multiple of 2^34 every four rows, so the block's tiles are cut there (the
    counter's high word is per tile); every pass and the checksum match the
    oracle element by element."""
    row_len = (1 << 32) - 64
    rows, cols, row0, col0 = 96, 64, 5, 128
    el = _block_indices(rows, cols, row_len, row0, col0)
    assert len(np.unique(el >> np.uint64(34))) > 20
    x0 = wl.random_bf16_bits(rows * cols, 70)
    r = np.array([0.6, 0.1, 0.9], np.float32)
    blk = to_device(x0, (rows, cols))
    with esopt.Plan(blocks=[esopt.Block(blk, TID, row_len, row0, col0)]) as p:
        assert p.tiles > 20
        (xs,) = _run_chain(p, [blk], r)
        got_sum = p.checksum()
    for (name, exp, base, delta), got in zip(_oracle_steps(xs, el, r), xs[1:]):
        rep = report(got, exp, base, delta)
        print("rows 2^32 apart:", name, rep)
        assert_parity(rep, name)
    host = xs[-1].reshape(rows, cols)
    exp_sum = 0
    for i in range(rows):
        exp_sum = (exp_sum + oracle.checksum(host[i], TID, (row0 + i) * row_len + col0)) & M64
    assert got_sum == exp_sum


def test_large_block_in_two_row_pieces():
    """A column block of more than 2^31 elements ([2100, 2^20] of a tensor
    with 2^20 + 5120 columns, 4.4 GB) is cut into pieces of 2048 and 52 rows:
    the whole tensor's perturb and update leave the same bits there, and the
    oracle agrees on the first and last 4096 columns of the two rows on
    either side of the cut."""
    rows, cols, row_len, col0 = 2100, 1 << 20, (1 << 20) + 5120, 2560
    n = rows * cols
    assert n > (1 << 31)
    g = torch.Generator(device="cuda").manual_seed(69)
    whole = (torch.randn(rows, row_len, device="cuda", generator=g) * 0.02).to(torch.bfloat16)
    blk = whole[:, col0:col0 + cols].contiguous()
    cols_s = np.r_[0:4096, cols - 4096:cols]

    def sample(t):
        return to_host(t[2047:2049][:, torch.from_numpy(cols_s).cuda()])

    x0 = sample(blk)
    r = torch.tensor([0.3, 0.8, 0.1, 0.6], device="cuda")
    with esopt.Plan(blocks=[esopt.Block(blk, TID, row_len, 0, col0)]) as p:
        assert p.tiles >= n // 65536
        p.perturb(21, 1, 1e-3)
        p.update([1, 2, 3, 4], [1, -1, 1, -1], r, 5e-4)
    with esopt.Plan([whole], tensor_ids=[TID]) as p:
        p.perturb(21, 1, 1e-3)
        p.update([1, 2, 3, 4], [1, -1, 1, -1], r, 5e-4)
    torch.cuda.synchronize()
    assert torch.equal(blk.view(torch.int16), whole[:, col0:col0 + cols].view(torch.int16))
    got = sample(blk)
    del whole, blk
    torch.cuda.empty_cache()
    el = (np.uint64(row_len) * np.arange(2047, 2049, dtype=np.uint64)[:, None]
          + np.uint64(col0) + cols_s.astype(np.uint64)[None, :]).ravel()
    x1 = oracle.perturb(x0, 21, TID, 1, 1e-3, elems=el)
    exp = oracle.update(x1, TID, [1, 2, 3, 4], [1, -1, 1, -1], r.cpu().numpy(), 5e-4, 1e-3,
                        elems=el)[0]
    delta = perturb_delta(21, TID, 1, 1e-3, el) + update_delta(
        TID, [1, 2, 3, 4], [1, -1, 1, -1], r.cpu().numpy(), 5e-4, 1e-3, 0, el)
    rep = report(got, exp, x0, delta)
    print("large block, rows 2047..2048:", rep)
    assert_parity(rep, "large block")


def test_block_geometry_is_validated():
    t = torch.zeros(4, 60, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(esopt.EsError):                      # cols not a multiple of 8
        esopt.Plan(blocks=[esopt.Block(t, 0, 256)])
    t = torch.zeros(4, 64, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(esopt.EsError):                      # first index 4
        esopt.Plan(blocks=[esopt.Block(t, 0, 256, 0, 4)])
    with pytest.raises(esopt.EsError):                      # past the row end
        esopt.Plan(blocks=[esopt.Block(t, 0, 256, 0, 200)])
    with pytest.raises(ValueError):
        esopt.Plan(blocks=[esopt.Block(t, 0, 256)], tensor_ids=[0])
    with pytest.raises(ValueError):
        esopt.Plan(blocks=[esopt.Block(t.t(), 0, 256)])     # not contiguous


def test_random_block_grids_match_the_whole_matrix():
    """Random matrices cut into random grids of blocks (row cuts anywhere,
    column cuts at multiples of 8, blocks copied to random sub-16-byte and
    larger offsets), each block through a plan of its own: every block
    bit-identical to the same block of the whole-matrix pass."""
    rng = np.random.default_rng(2026)
    for case in range(12):
        rows = int(rng.integers(1, 700))
        cols = 8 * int(rng.integers(1, 900))
        bits = wl.random_bf16_bits(rows * cols, 500 + case)
        whole = _whole(bits, rows, cols)
        src = to_device(bits, (rows, cols))
        rc = sorted(set([0, rows] + [int(x) for x in rng.integers(0, rows, int(rng.integers(0, 4)))]))
        cc = sorted(set([0, cols] + [8 * int(x) for x in rng.integers(0, cols // 8,
                                                                      int(rng.integers(0, 5)))]))
        for r0, r1 in zip(rc, rc[1:]):
            for c0, c1 in zip(cc, cc[1:]):
                pad = int(rng.choice([0, 1, 3, 8, 13, 64, 4096 + 5]))
                buf, blk = _block_buffer(src[r0:r1, c0:c1].contiguous(), pad)
                with esopt.Plan(blocks=[esopt.Block(blk, TID, cols, r0, c0)]) as p:
                    _passes(p, _rewards())
                torch.cuda.synchronize()
                assert torch.equal(blk.view(torch.int16),
                                   whole[r0:r1, c0:c1].view(torch.int16)), \
                    f"case {case}: [{rows}, {cols}] block rows [{r0}, {r1}) cols [{c0}, {c1}) pad {pad}"
                n = (r1 - r0) * (c1 - c0)
                assert torch.count_nonzero(buf[:pad].float()) == 0
                assert torch.count_nonzero(buf[pad + n:].float()) == 0


def test_allocation_free_update_on_a_block_plan():
    """es_update_noalloc on a plan with a strided block and a whole vector
    (two launches, the static scratch) leaves the bits es_update leaves."""
    rows, cols = 200, 1024
    bits = wl.random_bf16_bits(rows * cols, 71)
    v_bits = wl.random_bf16_bits(3000, 72)
    r = torch.tensor([0.4, 0.9, 0.2], device="cuda")
    out = []
    for noalloc in (False, True):
        a = to_device(bits, (rows, cols))[:, 256:768].contiguous()
        v = to_device(v_bits)
        with esopt.Plan(blocks=[esopt.Block(a, 1, cols, 0, 256), esopt.Block(v, 2, 3000)]) as p:
            fn = p.update_noalloc if noalloc else p.update
            fn([4, 5, 6], [1, -1, 1], r, 5e-4)
            fn([7, 8, 9], [1, 1, 1], r, 5e-4, flags=esopt.ES_UPDATE_STOCHASTIC_ROUND,
               round_seed=3)
        torch.cuda.synchronize()
        out.append((to_host(a), to_host(v)))
    for x, y in zip(*out):
        np.testing.assert_array_equal(x, y)
