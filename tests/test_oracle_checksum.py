"""Pins of the checksum oracle (oracle/checksum.py): SplitMix64's published
outputs through its mix64, mix64 undone by a separately written inverse, a
pure-Python big-integer sum on small tensors, additivity over split ranges
(so shard checksums add up to the whole tensor's), and sensitivity to every
element's bits, its position and the tensor id."""
import os

import numpy as np

import oracle
from paper_2608_17310_amd import workloads as wl

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "splitmix64.txt")
M = (1 << 64) - 1


def _golden():
    gamma, outs = None, []
    with open(GOLDEN) as fh:
        for line in fh:
            line = line.split("#")[0].strip()
            if not line:
                continue
            if line.startswith("gamma"):
                gamma = int(line.split()[1], 16)
            else:
                outs.append(int(line, 16))
    return gamma, outs


def test_mix64_gives_the_splitmix64_outputs():
    gamma, outs = _golden()
    states = np.array([(gamma * (i + 1)) & M for i in range(len(outs))], dtype=np.uint64)
    assert [int(v) for v in oracle.mix64(states)] == outs


def _undo_xorshift(y, s):
    """x with x ^ (x >> s) == y: each pass fixes s more high bits."""
    x = y
    for _ in range(64 // s + 1):
        x = y ^ (x >> s)
    return x & M


def test_mix64_is_undone_by_its_inverse():
    inv1 = pow(0xBF58476D1CE4E5B9, -1, 1 << 64)
    inv2 = pow(0x94D049BB133111EB, -1, 1 << 64)
    rng = np.random.default_rng(5)
    xs = rng.integers(0, np.iinfo(np.uint64).max, size=3000, dtype=np.uint64, endpoint=True)
    ys = oracle.mix64(xs)
    for x, y in zip(xs.tolist(), ys.tolist()):
        z = _undo_xorshift(y, 31)
        z = (z * inv2) & M
        z = _undo_xorshift(z, 27)
        z = (z * inv1) & M
        z = _undo_xorshift(z, 30)
        assert z == x


def _bigint_checksum(bits, tid, elem0):
    tot = 0
    for i, b in enumerate(bits.tolist()):
        x = ((elem0 + i) * 0x9E3779B97F4A7C15 + tid * 0xC2B2AE3D27D4EB4F
             + b * 0x165667B19E3779F9) & M
        x ^= x >> 30
        x = (x * 0xBF58476D1CE4E5B9) & M
        x ^= x >> 27
        x = (x * 0x94D049BB133111EB) & M
        x ^= x >> 31
        tot = (tot + x) & M
    return tot


def test_small_tensors_match_a_big_integer_sum():
    for n, tid, e0 in [(1, 0, 0), (37, 5, 8), (500, (1 << 32) - 1, (1 << 60) - 500),
                       (257, 3, 1 << 34)]:
        bits = wl.random_bf16_bits(n, 60 + n)
        assert oracle.checksum(bits, tid, e0) == _bigint_checksum(bits, tid, e0)
    assert oracle.checksum(np.zeros(0, np.uint16), 1) == 0


def test_split_ranges_add_up():
    bits = wl.random_bf16_bits(100_003, 61)
    whole = oracle.checksum(bits, 9, 1 << 20)
    rng = np.random.default_rng(6)
    for _ in range(20):
        cuts = np.sort(rng.integers(0, bits.size, size=3))
        edges = [0, *cuts.tolist(), bits.size]
        parts = [(bits[a:b], 9, (1 << 20) + a) for a, b in zip(edges, edges[1:])]
        assert oracle.plan_checksum(parts) == whole
    assert oracle.checksum(bits, 9, 1 << 20, chunk=997) == whole


def test_every_element_position_and_id_count():
    bits = wl.random_bf16_bits(5000, 62)
    base = oracle.checksum(bits, 4)
    rng = np.random.default_rng(7)
    for p in rng.integers(0, bits.size, size=300):
        x = bits.copy()
        x[p] ^= np.uint16(1 << int(rng.integers(0, 16)))       # one bit of one element
        assert oracle.checksum(x, 4) != base
    i, j = 10, 4000
    assert bits[i] != bits[j]
    x = bits.copy()
    x[[i, j]] = x[[j, i]]                                        # same values, swapped
    assert oracle.checksum(x, 4) != base
    assert oracle.checksum(bits, 5) != base
    assert oracle.checksum(bits, 4, elem0=8) != base


def test_int8_codes_are_summed_as_unsigned_bytes():
    codes = np.random.default_rng(8).integers(-128, 128, size=999).astype(np.int8)
    assert oracle.qchecksum(codes, 6) == _bigint_checksum(codes.view(np.uint8), 6, 0)
    assert oracle.qchecksum(codes, 6, chunk=100) == oracle.qchecksum(codes, 6)
    assert oracle.qchecksum(codes, 6, 1 << 30) == _bigint_checksum(codes.view(np.uint8), 6,
                                                                    1 << 30)
    cut = 512                                   # a shard at a whole-tensor offset
    assert (oracle.qchecksum(codes[:cut], 6) + oracle.qchecksum(codes[cut:], 6, cut)) & M == \
        oracle.qchecksum(codes, 6)
    x = codes.copy()
    x[17] = -x[17] if x[17] not in (0, -128) else 5
    assert oracle.qchecksum(x, 6) != oracle.qchecksum(codes, 6)
