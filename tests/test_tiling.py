"""The host-side tiling of a bf16 plan (es_tile_layout exposes it; no device
access): every element of a tensor lies in exactly one tile, full tiles are
tile-sized and start on a tile-sized boundary of the address space, every tile
starts on an 8-element group and keeps its Philox counter's high word (element
index >> 34) constant, and a tensor whose base is not 16-byte aligned has only
tail tiles; a shard's tiles carry the whole tensor's element numbers.  These
are the invariants the kernels rely on for bit-identical noise whatever the
layout."""
import numpy as np
import pytest

from paper_2608_17310_amd import esopt

TILE = 1024 * 8 * 8            # default launch shape: 1024 lanes x 8 groups x 8 elements
HI = 1 << 34


def _check(addr, numel, offset=0):
    """Invariants of one tensor's tiles; elements are numbered in the whole
    tensor, the shard starting `offset` elements into it."""
    tiles = esopt.tile_layout(addr, numel, offset)
    if numel == 0:
        assert tiles == []
        return tiles
    full = [t for t in tiles if t[2]]
    tail = [t for t in tiles if not t[2]]
    assert tiles == full + tail                        # full tiles first
    spans = sorted((t[0], t[1]) for t in tiles)
    assert spans[0][0] == offset and spans[-1][1] == offset + numel
    for (a0, a1), (b0, b1) in zip(spans, spans[1:]):
        assert a1 == b0                                # disjoint, no gap
    for e0, e1, is_full, aligned in tiles:
        assert 0 < e1 - e0 <= TILE
        assert e0 % 8 == 0
        assert e0 // HI == (e1 - 1) // HI              # counter high word constant
        assert aligned == (1 if addr % 16 == 0 else 0)
        if is_full:
            assert e1 - e0 == TILE
            # on a tile-sized boundary of the address space (the shard's own addresses)
            assert (addr + 2 * (e0 - offset)) % (2 * TILE) == 0
    if addr % 16:
        assert not full
    return tiles


@pytest.mark.parametrize("addr", [0x10000000, 0x10000000 + 256, 0x10000000 + 2048,
                                  0x10000000 + 131072 - 16, 0x10000000 + 2, 0x10000000 + 8])
@pytest.mark.parametrize("numel", [0, 1, 7, 8, 9, 65535, 65536, 65537, 131072 + 5120,
                                   26214400, 5120])
def test_tiles_cover_each_element_once(addr, numel):
    _check(addr, numel)


def test_random_layouts():
    rng = np.random.default_rng(5)
    for _ in range(200):
        addr = int(rng.integers(1, 1 << 30)) * 2
        numel = int(rng.integers(0, 1 << 22))
        _check(addr, numel)


def test_aligned_tensor_has_at_most_two_tail_pieces():
    # a head before the first boundary and a remainder after the last full tile
    for addr in (0x20000000, 0x20000000 + 4096, 0x20000000 + 65536):
        tiles = _check(addr, 89128960)                  # a 17408 x 5120 matrix
        assert sum(1 for t in tiles if not t[2]) <= 2
        assert sum(t[1] - t[0] for t in tiles if t[2]) >= 89128960 - 2 * TILE


def test_tiles_split_at_the_counter_high_word():
    # a tensor longer than 2^34 elements (32 GB): no tile straddles element 2^34
    addr = 0x40000000 + 1024                            # head of 65024 elements
    tiles = _check(addr, HI + 3 * TILE + 17)
    assert any(t[0] == HI for t in tiles)
    assert any(t[1] == HI for t in tiles)


@pytest.mark.parametrize("offset", [8, 5120 * 640, 65536 * 3 + 8, (1 << 34) - 65536 * 2 + 40])
@pytest.mark.parametrize("addr", [0x10000000, 0x10000000 + 2048, 0x10000000 + 2])
def test_shard_tiles_use_the_whole_tensors_element_numbers(addr, offset):
    # a row shard of a [5120, 5120] matrix, and shards near 2^34 elements of
    # their whole tensor: tiles are placed by the shard's own addresses, and
    # still never straddle a multiple of 2^34 elements of the whole tensor
    tiles = _check(addr, 5120 * 640 + 24, offset)
    whole = offset + 5120 * 640 + 24
    if offset < (1 << 34) < whole:
        assert any(t[0] == 1 << 34 for t in tiles)


def test_validation():
    lib = esopt.load()
    n = esopt._u64(0)
    br = esopt.ctypes.byref
    assert lib.es_tile_layout(3, 10, 0, None, 0, br(n)) == esopt.ES_ERR_ALIGN
    assert lib.es_tile_layout(2, 10, 0, None, 0, None) == esopt.ES_ERR_INVALID_ARG
    assert lib.es_tile_layout(2, (1 << 60) + 1, 0, None, 0, br(n)) == esopt.ES_ERR_INVALID_ARG
    assert lib.es_tile_layout(2, (1 << 60) - 7, 1, None, 0, br(n)) == esopt.ES_ERR_INVALID_ARG
    assert lib.es_tile_layout(2, 10, 0, None, 5, br(n)) == esopt.ES_ERR_INVALID_ARG
    # the host-side list is bounded: 2^40 elements would be 2^24 tiles
    assert lib.es_tile_layout(2, 1 << 40, 0, None, 0, br(n)) == esopt.ES_ERR_INVALID_ARG
    assert "2^22" in esopt.last_error()
    with pytest.raises(ValueError):
        esopt.tile_layout(2, 10, offset=4)              # not a multiple of 8
