"""Pins of the oracle's noise definition: the word-to-element assignment (via
the counter/offset APIs of PyTorch's and rocRAND's Philox engines), the
uniform map's closed-form values, hand-worked Box-Muller values, and the
distribution of the generated normals (moments, KS distance, bound,
independence)."""
import math

import numpy as np
import pytest
from scipy import stats

from oracle import uniform_from_word, angle_from_word, box_muller, normals, noise_words

BM_BOUND = math.sqrt(48.0 * math.log(2.0))     # sqrt(-2 ln 2^-24)


@pytest.mark.parametrize("engine", ["torch", "rocrand"])
def test_assignment_matches_engine_counter_api(kat_harness, engine):
    if engine not in kat_harness:
        pytest.skip("engine harness not available")
    rng = np.random.default_rng(5)
    seeds = [int(x) for x in rng.integers(0, 1 << 63, size=40)] + [0, 1, (1 << 64) - 1]
    cases = []
    for s in seeds:
        tid = int(rng.integers(0, 700))
        elems = rng.integers(0, 1 << 34, size=8).astype(np.uint64)
        elems[:4] = np.arange(4, dtype=np.uint64) + np.uint64(4 * int(rng.integers(0, 1 << 20)))
        cases.append((s, tid, elems))
    for s, tid, elems in cases:
        # the engine keys on the raw 64-bit seed; tensor_id (domain 0) is the
        # subsequence and the quad index j >> 2 the offset
        words = kat_harness[engine]([(s, tid, int(j) >> 2) for j in elems])
        expect = []
        for j, w in zip(elems, words):
            lane = int(j) & 3
            pair = (w[0], w[1]) if lane < 2 else (w[2], w[3])
            c, sn = box_muller(np.uint64(pair[0]), np.uint64(pair[1]))
            expect.append(float(c if lane % 2 == 0 else sn))
        got = normals(s, tid, elems)
        np.testing.assert_array_equal(got, np.array(expect))
        nw = noise_words(s, tid, elems >> np.uint64(2))
        assert [tuple(int(x) for x in nw[:, i]) for i in range(len(elems))] == words


def test_uniform_map_closed_forms():
    assert uniform_from_word(0) == 2.0 ** -24
    assert uniform_from_word(0x7FFFFF) == 1.0 - 2.0 ** -24
    assert uniform_from_word(0xFFFFFFFF) == 1.0 - 2.0 ** -24
    assert uniform_from_word(1 << 22) == 0.5 + 2.0 ** -24
    assert uniform_from_word(0xFF800000) == 2.0 ** -24     # high 9 bits are dropped
    assert angle_from_word(0) == 0.0
    assert angle_from_word(1 << 22) == 0.5
    assert angle_from_word(1 << 21) == 0.25
    assert angle_from_word(0x7FFFFF) == 1.0 - 2.0 ** -23
    assert angle_from_word(0xFF800000 | 5) == 5 * 2.0 ** -23
    w = np.random.default_rng(0).integers(0, 1 << 32, size=100000, dtype=np.uint64)
    for f in (uniform_from_word, angle_from_word):
        u = f(w)
        assert np.all(u.astype(np.float32).astype(np.float64) == u)   # exact in binary32
        assert np.all((u >= 0) & (u < 1))
        grid = f(np.arange(0, 1 << 14, dtype=np.uint64))
        assert np.all(np.diff(grid) == 2.0 ** -23)
    assert np.all(uniform_from_word(w) > 0)


def test_box_muller_hand_values():
    half = np.uint64(1 << 22)            # u = 1/2 + 2^-24, or half a turn
    zero = np.uint64(0)                  # u = 2^-24, or angle 0
    quarter = np.uint64(1 << 21)         # a quarter turn
    r_half = math.sqrt(2.0 * math.log(2.0))          # Rayleigh median, 1.17741...
    c, s = box_muller(half, zero)        # phi = 0: (r, 0) exactly
    assert abs(float(c) - r_half) < 1e-6
    assert float(s) == 0.0
    c, s = box_muller(half, quarter)     # phi = pi/2
    assert abs(float(s) - r_half) < 1e-6
    assert abs(float(c)) < 1e-15
    c, s = box_muller(zero, half)        # largest radius, phi = pi
    assert abs(float(c) + BM_BOUND) < 1e-12
    assert abs(float(s)) < 1e-14
    c, s = box_muller(np.uint64(0x7FFFFF), half)   # smallest radius
    assert abs(abs(float(c)) - math.sqrt(2.0 ** -23)) < 1e-9
    # the high bits of the words play no part
    c2, s2 = box_muller(np.uint64(0xABC00000 | (1 << 22)), np.uint64(0x12800000 | (1 << 21)))
    assert (float(c2), float(s2)) == tuple(float(x) for x in box_muller(half, quarter))


def test_normal_moments_and_ks():
    n = 1 << 21
    e = normals(42, 3, np.arange(n, dtype=np.uint64))
    se = 1.0 / math.sqrt(n)
    assert abs(e.mean()) < 5 * se
    assert abs(e.var() - 1.0) < 5 * math.sqrt(2.0) * se
    assert abs(stats.skew(e)) < 5 * math.sqrt(6.0) * se
    assert abs(stats.kurtosis(e)) < 5 * math.sqrt(24.0) * se
    d, p = stats.kstest(e, "norm")
    assert p > 1e-4, (d, p)
    assert np.abs(e).max() <= BM_BOUND
    # each of the four lanes of a call is itself N(0,1)
    for lane in range(4):
        x = e[lane::4]
        assert abs(x.var() - 1.0) < 5 * math.sqrt(2.0 * 4) * se


def test_normal_independence():
    n = 1 << 20
    idx = np.arange(n, dtype=np.uint64)
    e = normals(7, 0, idx)
    lim = 5.0 / math.sqrt(n / 4)
    for a, b in [(0, 1), (2, 3), (0, 2), (1, 3)]:
        assert abs(np.corrcoef(e[a::4], e[b::4])[0, 1]) < lim
    other_seed = normals(8, 0, idx)
    other_tensor = normals(7, 1, idx)
    lim = 5.0 / math.sqrt(n)
    assert abs(np.corrcoef(e, other_seed)[0, 1]) < lim
    assert abs(np.corrcoef(e, other_tensor)[0, 1]) < lim
    # the pair (cos, sin) shares its radius: squared values are correlated
    # only through r, and r^2/2 ~ Exp(1) for the pair
    r2 = e[0::4] ** 2 + e[1::4] ** 2
    assert abs(r2.mean() / 2 - 1.0) < 5 / math.sqrt(n / 4)


def test_sampled_elements_match_dense():
    dense = normals(3, 9, np.arange(4096, dtype=np.uint64))
    pick = np.array([4095, 0, 17, 1024, 3, 2], dtype=np.uint64)
    np.testing.assert_array_equal(normals(3, 9, pick), dense[pick.astype(np.int64)])
