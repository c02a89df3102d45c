"""Pins of the oracle's int8 path: the stochastic offset rounding enumerated
over all draws, exact revert wherever nothing clamps, the offsets'
distribution against its closed form, an element-by-element pure-Python
rendering (big-integer Philox, math library Box-Muller, explicit row lookup),
the update's unbiasedness and multi-step slope, and the identities."""
import math

import numpy as np
import pytest

import oracle
from oracle import (round_offset, round_offset9, qperturb, qrestore, qupdate,
                    philox4x32_10_bigint, spare_draws, noise_words,
                    ES_REWARDS_ARE_WEIGHTS, ES_UPDATE_DIV_SIGMA)

ALL_DRAWS = np.arange(65536, dtype=np.int64)


@pytest.mark.parametrize("d", [0.0, 2 ** -16, 0.5, -0.5, 1 - 2 ** -16, 3.25, -7.0001220703125,
                               -2 ** -16, 126.99998474121094, 13 * 2 ** -16 - 4])
def test_round_offset_enumerated_draws(d):
    k = round_offset(np.full(65536, d), ALL_DRAWS)
    lo = math.floor(d)
    assert set(np.unique(k)) <= {lo, lo + 1}
    frac = d - lo
    assert np.sum(k == lo + 1) == round(frac * 65536)      # d is on the 2^-16 grid
    assert np.sum(k) / 65536.0 == d                          # exact mean
    # the step is taken by the top draws
    if frac:
        assert np.all(k[ALL_DRAWS >= 65536 - round(frac * 65536)] == lo + 1)


def test_round_offset_rejects_bad_draws():
    with pytest.raises(ValueError):
        round_offset(0.5, 65536)
    with pytest.raises(ValueError):
        round_offset9(0.5, 512)


@pytest.mark.parametrize("d", [0.0, 0.5, -0.5, 2 ** -11, 1 - 2 ** -11, 3.3, -7.77, 126.999,
                               -0.000244140625, 0.123456789])
def test_round_offset9_enumerated_draws(d):
    """Over all 512 draws: results floor(d) or floor(d) + 1, the step taken by
    the top draws, exactly round(frac(d) * 512) of them when frac(d) * 512 is
    not a half-integer, and the mean within 2^-10 of d."""
    r = np.arange(512)
    k = round_offset9(np.full(512, d), r)
    lo = math.floor(d)
    assert set(np.unique(k)) <= {lo, lo + 1}
    ups = int(np.sum(k == lo + 1))
    assert np.all(k[r >= 512 - ups] == lo + 1) and np.all(k[r < 512 - ups] == lo)
    assert abs(np.sum(k) / 512.0 - d) <= 2.0 ** -10
    frac = d - lo
    if abs(frac * 512 - round(frac * 512) - 0.5) > 1e-9 and abs(frac * 512 % 1 - 0.5) > 1e-9:
        assert ups == round(frac * 512)


def test_spare_draws_are_the_top_bits_of_each_elements_own_word():
    rng = np.random.default_rng(13)
    for seed in (0, (1 << 64) - 1, 123456789):
        el = np.concatenate([np.arange(12), rng.integers(0, 1 << 36, 30)]).astype(np.uint64)
        w = noise_words(seed, 5, el >> np.uint64(2))
        got = spare_draws(seed, 5, el)
        for i, j in enumerate(el.tolist()):
            assert got[i] == int(w[j & 3, i]) >> 23
    d = spare_draws(77, 1, np.arange(1 << 18, dtype=np.uint64))
    assert d.min() == 0 and d.max() == 511
    assert abs(d.mean() - 255.5) < 5 * math.sqrt((512 ** 2 - 1) / 12 / d.size)


def _codes(n, seed):
    return np.random.default_rng(seed).integers(-127, 128, size=n).astype(np.int8)


def test_revert_is_exact_wherever_nothing_clamps():
    n, row = 1 << 16, 64
    q = _codes(n, 1)
    rng = np.random.default_rng(2)
    scales = rng.uniform(3e-4, 1.2e-3, n // row).astype(np.float32)
    scales[::7] = 5e-5                                   # rows where offsets are large
    p = qperturb(q, scales, row, 9, 3, 1, 1e-3)
    back = qrestore(p, scales, row, 9, 3, 1, 1e-3)
    d, r, ok = oracle.offset_values(scales, row, 9, 3, 1, 1e-3, np.arange(n, dtype=np.uint64))
    k = round_offset9(d, r)
    unclamped = np.abs(q.astype(np.int64) + k) <= 127
    assert unclamped.mean() > 0.8 and (~unclamped).sum() > 100
    np.testing.assert_array_equal(back[unclamped], q[unclamped])
    assert np.mean(back[~unclamped] != q[~unclamped]) > 0.9
    assert p.min() >= -127 and back.min() >= -127


def test_offsets_match_their_closed_form_distribution():
    """With one scale, k = floor(d + (2 r + 1) 2^-10), d = (sigma / s) eps:
    mean 0 and variance (sigma / s)^2 + 1/6 (the stochastic rounding adds
    f(1 - f) with the fractional part f uniform; the 9-bit grid changes that
    by under 1e-6)."""
    n = 1 << 20
    s = np.float32(7e-4)
    ratio = float(np.float32(1e-3)) / float(s)
    k = qperturb(np.zeros(n, np.int8), [s], 0, 1234, 0, 1, 1e-3).astype(np.float64)
    var = ratio ** 2 + 1.0 / 6.0
    assert abs(k.mean()) < 5 * math.sqrt(var / n)
    # the variance of a sample variance of a near-normal variable is ~2 var^2 / n
    assert abs(k.var() - var) < 5 * var * math.sqrt(2.0 / n) + 0.002, (k.var(), var)
    # most offsets are nonzero at this sigma / s, and symmetric
    assert np.mean(k == 0) < 0.3
    assert abs(np.mean(k > 0) - np.mean(k < 0)) < 0.01


def _word_normal(w_a, w_b, first):
    m_a, m_b = w_a & 0x7FFFFF, w_b & 0x7FFFFF
    u = (m_a + 0.5) * 2.0 ** -23
    phi = 2.0 * math.pi * m_b * 2.0 ** -23
    rad = math.sqrt(-2.0 * math.log(u))
    return rad * math.cos(phi) if first else rad * math.sin(phi)


def _eps(seed, tid, j):
    q = j >> 2
    w = philox4x32_10_bigint((q & 0xFFFFFFFF, q >> 32, tid, 0), (seed & 0xFFFFFFFF, seed >> 32))
    lane = j & 3
    pair = (w[0], w[1]) if lane < 2 else (w[2], w[3])
    return _word_normal(pair[0], pair[1], lane % 2 == 0)


def _draw(seed, tid, j, domain):
    g = j >> 3
    w = philox4x32_10_bigint((g & 0xFFFFFFFF, g >> 32, tid, domain), (seed & 0xFFFFFFFF, seed >> 32))
    return (w[(j & 7) >> 1] >> (16 * (j & 1))) & 0xFFFF


def test_pure_python_rendering_matches_perturb_and_update():
    rng = np.random.default_rng(5)
    n, row, tid, seed = 5000, 24, 11, (1 << 40) + 17
    q = _codes(n, 6)
    scales = rng.uniform(2e-4, 1e-3, n // row + 1).astype(np.float32)
    scales[3] = 0.0                                      # an invalid row: left unchanged
    elems = np.concatenate([np.arange(80), rng.integers(0, n, 60)]).astype(np.uint64)
    got = qperturb(q[elems.astype(np.int64)], scales, row, seed, tid, -1, 1e-3, elems=elems)
    sig = float(np.float32(1e-3))
    for j, g in zip(elems.tolist(), got.tolist()):
        s = float(scales[j // row])
        if not s >= 2.0 ** -126:
            assert g == q[j]
            continue
        d = -sig * _eps(seed, tid, j) / s
        qd = j >> 2
        word = philox4x32_10_bigint((qd & 0xFFFFFFFF, qd >> 32, tid, 0),
                                    (seed & 0xFFFFFFFF, seed >> 32))[j & 3]
        k = math.floor(d + (2 * (word >> 23) + 1) * 2.0 ** -10)
        assert g == max(-127, min(127, int(q[j]) + k)), j
    # the update: two members, weights as given, domain-1 draws under round_seed
    seeds, signs, w = [3, 8], [1, -1], np.array([0.7, -0.2], np.float32)
    alpha, rs = 2e-3, 99
    got, st = qupdate(q[elems.astype(np.int64)], scales, row, tid, seeds, signs, w, alpha, 0.0,
                      flags=ES_REWARDS_ARE_WEIGHTS, elems=elems, round_seed=rs)
    assert st == 0
    c = float(np.float32(alpha)) / 2
    for j, g in zip(elems.tolist(), got.tolist()):
        s = float(scales[j // row])
        if not s >= 2.0 ** -126:
            assert g == q[j]
            continue
        delta = sum(c * sg * float(wi) * _eps(sd, tid, j) for sd, sg, wi in zip(seeds, signs, w))
        k = math.floor(delta / s + _draw(rs, tid, j, 1) * 2.0 ** -16)
        assert g == max(-127, min(127, int(q[j]) + k)), j


def test_update_is_unbiased_in_quantum_units():
    n = 1 << 18
    s = np.float32(7e-4)
    q = np.zeros(n, np.int8)
    r = np.random.default_rng(8).random(8).astype(np.float32)
    seeds = list(range(100, 108))
    got, st = qupdate(q, [s], 0, 0, seeds, [1] * 8, r, 5e-4, 0.0, round_seed=4)
    assert st == 0
    z, _ = oracle.zscore(r)
    c = oracle.update_coefficient(5e-4, 0.0, 8, 0)
    el = np.arange(n, dtype=np.uint64)
    delta = sum(c * zi * oracle.normals(sd, 0, el) for sd, zi in zip(seeds, z)) / float(s)
    f = delta - np.floor(delta)
    err = got.astype(np.float64).sum() - delta.sum()
    assert abs(err) < 5 * math.sqrt(np.sum(f * (1 - f)))
    # the steps are a fraction of a quantum: nearest rounding would drop most
    assert np.mean(np.abs(delta) < 0.5) > 0.9
    assert np.mean(got != 0) > 0.1


def test_multistep_update_tracks_unrounded_sum():
    """70 updates (G = 8, alpha = 2.5e-4, as in the paper's update-magnitude
    table, Appendix A.1) on codes of N(0, 0.02) weights quantized per row:
    the dequantized total step regresses on the unrounded sum with slope 1."""
    n, row, T, G, alpha = 1 << 14, 256, 70, 8, 2.5e-4
    w = np.random.default_rng(9).normal(0, 0.02, n)
    scales = (np.abs(w).reshape(-1, row).max(axis=1) / 127).astype(np.float32)
    s = np.repeat(scales.astype(np.float64), row)
    q0 = np.clip(np.round(w / s), -127, 127).astype(np.int8)
    q = q0.copy()
    exact = np.zeros(n)
    rng = np.random.default_rng(10)
    el = np.arange(n, dtype=np.uint64)
    for t in range(T):
        seeds = [700 * t + i for i in range(G)]
        r = rng.random(G).astype(np.float32)
        z, _ = oracle.zscore(r)
        c = oracle.update_coefficient(alpha, 0.0, G, 0)
        for sd, zi in zip(seeds, z):
            exact += c * zi * oracle.normals(sd, 0, el)
        q, st = qupdate(q, scales, row, 0, seeds, [1] * G, r, alpha, 0.0, round_seed=t)
    moved = (q.astype(np.float64) - q0) * s
    b = moved @ exact / (exact @ exact)
    se = math.sqrt(np.sum((moved - b * exact) ** 2 * exact ** 2)) / (exact @ exact)
    assert abs(b - 1.0) < 5 * se + 1e-3, (b, se)


def test_identities_and_validation():
    q = _codes(4096, 12)
    sc = np.full(64, 7e-4, np.float32)
    np.testing.assert_array_equal(qperturb(q, sc, 64, 1, 0, 1, 0.0), q)
    bad = sc.copy()
    bad[[0, 1, 2, 3]] = [0.0, -1.0, np.inf, 1e-40]          # 1e-40: subnormal
    p = qperturb(q, bad, 64, 1, 0, 1, 1e-3)
    np.testing.assert_array_equal(p[:256], q[:256])
    assert np.mean(p[256:] != q[256:]) > 0.5
    # equal rewards, alpha = 0, non-finite reward: unchanged
    for rew, alpha, want in [([0.5, 0.5], 5e-4, 0), ([0.1, 0.9], 0.0, 0), ([0.1, np.inf], 5e-4, 1)]:
        out, st = qupdate(q, sc, 64, 0, [1, 2], [1, 1], rew, alpha, 0.0)
        assert st == want
        np.testing.assert_array_equal(out, q)
    # the 1/(G sigma) mode scales the step
    a, _ = qupdate(np.zeros(4096, np.int8), [7e-4], 0, 0, [1, 2], [1, 1], [0.1, 0.9], 5e-4, 0.5,
                   flags=ES_UPDATE_DIV_SIGMA, round_seed=1)
    b, _ = qupdate(np.zeros(4096, np.int8), [7e-4], 0, 0, [1, 2], [1, 1], [0.1, 0.9], 1e-3, 0.5,
                   round_seed=1)
    np.testing.assert_array_equal(a, b)
    with pytest.raises(ValueError):
        qperturb(q, sc, 64, 1, 0, 2, 1e-3)


def test_out_of_range_code_is_kept_under_an_invalid_scale_and_clamped_otherwise():
    # -128 lies outside the clamp range [-127, 127]: a step under a valid
    # scale clamps it into the range (even a zero offset), and a row whose
    # scale is not a normal positive finite value is left exactly as it is
    q = np.full(16, -128, dtype=np.int8)
    scales = np.array([7e-4, 0.0], dtype=np.float32)       # row 0 valid, row 1 invalid
    out = qperturb(q, scales, 8, 5, 0, 1, 1e-3)
    assert np.all(out[:8] >= -127)
    assert np.all(out[8:] == -128)
    back = qrestore(out, scales, 8, 5, 0, 1, 1e-3)
    assert np.all(back[8:] == -128)
