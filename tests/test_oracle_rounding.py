"""Pins of the oracle's stochastic rounding of the update: the rounding of one
binary32 value against bit-level truncation of its pattern, enumerated over
all 65536 draws (the mean is the value itself, exactly); the special values;
the draws (Philox domain 1) against the engines' counter API and the
big-integer Philox, and their uniformity; and, statistically, that the
stochastically rounded update is unbiased where round-to-nearest drops small
steps."""
import math

import numpy as np
import pytest
from scipy import stats

import oracle
from oracle import (f64_to_bf16_sr, f64_to_bf16_rne, bf16_to_f64, bf16_ulp, rounding_draws,
                    noise_words, philox4x32_10_bigint, ES_UPDATE_STOCHASTIC_ROUND,
                    ES_REWARDS_ARE_WEIGHTS)
from paper_2608_17310_amd.workloads import random_bf16_bits

ALL_DRAWS = np.arange(65536, dtype=np.int64)


def _f32_patterns():
    rng = np.random.default_rng(11)
    pats = rng.integers(0, 1 << 32, size=48, dtype=np.uint64).astype(np.uint32)
    finite = (pats & np.uint32(0x7F800000)) != np.uint32(0x7F800000)
    fixed = np.array([0x3F800000, 0x3F800001, 0x3F80FFFF, 0x3F808000, 0xBF808000,
                      0x00000001, 0x0000FFFF, 0x00010000, 0x807F0001, 0x007FFFFF,
                      0x00800000, 0x3C23D70A, 0xBCA3D70A, 0x7F7F0000, 0x7F7EFFFF,
                      0x00000000, 0x80000000], dtype=np.uint32)
    return np.concatenate([pats[finite], fixed])


@pytest.mark.parametrize("bits", list(_f32_patterns()))
def test_sr_enumerated_draws(bits):
    """Over all 65536 draws: results are the truncation of the binary32
    pattern toward zero or the next bf16 away from zero; the step is taken
    for exactly (low 16 bits) draws, the top ones; the mean is x32."""
    x32 = np.array([bits], dtype=np.uint32).view(np.float32).astype(np.float64)[0]
    res = f64_to_bf16_sr(np.full(65536, x32), ALL_DRAWS).astype(np.int64)
    trunc = int(bits) >> 16
    low = int(bits) & 0xFFFF
    expect = np.where(ALL_DRAWS >= 65536 - low, trunc + 1, trunc) if low else np.full(65536, trunc)
    np.testing.assert_array_equal(res, expect)
    vals = bf16_to_f64(res.astype(np.uint16))
    # sum of 65536 bf16 values of two adjacent magnitudes: exact in fp64
    assert vals.sum() / 65536.0 == x32


def test_sr_special_values():
    r = np.array([0, 1, 32768, 65535])
    for x, want in [(np.inf, 0x7F80), (-np.inf, 0xFF80), (np.nan, 0x7FC0), (0.0, 0x0000),
                    (-0.0, 0x8000), (3.5e38, 0x7F80), (-3.5e38, 0xFF80)]:
        np.testing.assert_array_equal(f64_to_bf16_sr(np.full(4, x), r), want)
    # the largest finite binary32: the step away from zero reaches infinity
    fmax = float(np.finfo(np.float32).max)
    np.testing.assert_array_equal(f64_to_bf16_sr(np.full(4, fmax), r),
                                  [0x7F7F, 0x7F80, 0x7F80, 0x7F80])
    # a value above FLT_MAX that binary32 rounds down to FLT_MAX
    assert f64_to_bf16_sr(fmax * (1 + 2.0 ** -26), 0)[0] == 0x7F7F
    with pytest.raises(ValueError):
        f64_to_bf16_sr(1.0, 65536)
    with pytest.raises(ValueError):
        f64_to_bf16_sr(1.0, -1)


def test_sr_takes_the_binary32_value():
    """The decision is taken on the binary32 rounding of the fp64 sum: a sum a
    hair below a bf16 value that binary32 rounds onto it is that value for
    every draw (directly from fp64 it would truncate for small draws)."""
    x = 1.0 + 2.0 ** -7 - 2.0 ** -40
    assert np.all(f64_to_bf16_sr(np.full(65536, x), ALL_DRAWS) == 0x3F81)
    # 1 + 2^-16 is 1/512 of a bf16 step (2^-7) above 1: 128 of 65536 draws step
    res = f64_to_bf16_sr(np.full(65536, 1.0 + 2.0 ** -16), ALL_DRAWS)
    assert np.sum(res == 0x3F81) == 128
    assert np.sum(res == 0x3F80) == 65536 - 128


def test_sr_within_one_step_of_rne():
    rng = np.random.default_rng(3)
    x = rng.normal(0, 0.02, 200000) * np.exp(rng.uniform(-20, 20, 200000))
    r = rng.integers(0, 65536, x.size)
    sr = f64_to_bf16_sr(x, r)
    rne = f64_to_bf16_rne(x)
    x32 = x.astype(np.float32).astype(np.float64)
    d = np.abs(bf16_to_f64(sr) - x32)
    assert np.all(d < bf16_ulp(x32))
    assert np.all(np.abs(bf16_to_f64(sr) - bf16_to_f64(rne)) <= bf16_ulp(x32))
    assert np.all(np.sign(bf16_to_f64(sr)) * np.sign(x32) >= 0)


# ------------------------------------------------------------------- draws --

def test_rounding_draws_against_bigint_philox():
    rng = np.random.default_rng(8)
    for seed in [0, 1, (1 << 64) - 1] + [int(s) for s in rng.integers(0, 1 << 63, size=5)]:
        tid = int(rng.integers(0, 1000))
        elems = np.concatenate([np.arange(16), rng.integers(0, 1 << 40, size=24),
                                [(1 << 35) * 8 + 5, (1 << 35) * 8 - 1]]).astype(np.uint64)
        got = rounding_draws(seed, tid, elems)
        for j, v in zip(elems, got):
            j = int(j)
            g = j >> 3
            w = philox4x32_10_bigint((g & 0xFFFFFFFF, g >> 32, tid, 1),
                                     (seed & 0xFFFFFFFF, seed >> 32))
            word = w[(j & 7) >> 1]
            assert int(v) == ((word >> (16 * (j & 1))) & 0xFFFF), (seed, tid, j)


def test_rounding_draws_match_engine_counter_api(kat_harness):
    """Domain 1 is the high word of the engines' 64-bit subsequence."""
    rng = np.random.default_rng(9)
    for engine, run in kat_harness.items():
        for _ in range(4):
            seed = int(rng.integers(0, 1 << 63))
            tid = int(rng.integers(0, 700))
            groups = [int(g) for g in rng.integers(0, 1 << 33, size=6)]
            words = run([(seed, tid | (1 << 32), g) for g in groups])
            for g, w in zip(groups, words):
                el = np.arange(8 * g, 8 * g + 8, dtype=np.uint64)
                want = [(w[k // 2] >> (16 * (k & 1))) & 0xFFFF for k in range(8)]
                assert rounding_draws(seed, tid, el).tolist() == want, engine


def test_rounding_draws_uniform_and_separate_from_noise():
    el = np.arange(1 << 20, dtype=np.uint64)
    d = rounding_draws(12345, 3, el)
    assert d.min() >= 0 and d.max() <= 0xFFFF
    for part in (d >> 8, d & 0xFF):
        counts = np.bincount(part, minlength=256)
        assert stats.chisquare(counts).pvalue > 1e-4
    se = math.sqrt((65536 ** 2 - 1) / 12 / d.size)
    assert abs(d.mean() - 32767.5) < 5 * se
    assert abs(np.corrcoef(d[0::2], d[1::2])[0, 1]) < 5 / math.sqrt(d.size / 2)
    # the same counter in the noise domain gives other words
    nw = noise_words(12345, 3, np.arange(1 << 17, dtype=np.uint64))
    same = np.mean((nw[0] & np.uint64(0xFFFF)).astype(np.int64) == d[0::8])
    assert same < 1e-3


# ------------------------------------------------------------------ update --

def test_sr_update_is_unbiased_for_sub_half_ulp_steps():
    """A single-member update too small for round-to-nearest to move most
    elements: RNE leaves them, stochastic rounding moves them so that the
    sum over elements of (theta' - x32) is zero within its standard error."""
    n = 1 << 18
    theta = random_bf16_bits(n, 21)
    el = np.arange(n, dtype=np.uint64)
    alpha = 2e-5
    rne, _ = oracle.update(theta, 0, [77], [1], np.array([1.0], np.float32), alpha, 0.0,
                           flags=ES_REWARDS_ARE_WEIGHTS)
    sr, _ = oracle.update(theta, 0, [77], [1], np.array([1.0], np.float32), alpha, 0.0,
                          flags=ES_REWARDS_ARE_WEIGHTS | ES_UPDATE_STOCHASTIC_ROUND,
                          round_seed=99)
    assert np.mean(rne == theta) > 0.7
    assert np.mean(sr == theta) < np.mean(rne == theta) - 0.05
    t = bf16_to_f64(theta)
    delta = float(np.float32(alpha)) * oracle.normals(77, 0, el)
    x32 = (t + delta).astype(np.float32).astype(np.float64)
    lo = np.floor(np.abs(x32) / bf16_ulp(x32)) * bf16_ulp(x32)
    f = (np.abs(x32) - lo) / bf16_ulp(x32)
    var = (bf16_ulp(x32) ** 2) * f * (1 - f)
    err = (bf16_to_f64(sr) - x32).sum()
    assert abs(err) < 5 * math.sqrt(var.sum()), (err, math.sqrt(var.sum()))
    # round-to-nearest is biased toward theta: its steps fall short of delta
    moved_rne = (bf16_to_f64(rne) - t) @ delta / (delta @ delta)
    moved_sr = (bf16_to_f64(sr) - t) @ delta / (delta @ delta)
    assert moved_rne < 0.6
    assert abs(moved_sr - 1.0) < 0.05


def test_sr_multistep_tracks_unrounded_accumulation():
    """70 updates of G = 8 (alpha = 2.5e-4, the setting of the paper's
    update-magnitude table, Appendix A.1) from N(0, 0.02) weights: with
    stochastic rounding the bf16 trajectory's total step regresses on the
    unrounded sum of the steps with slope 1; with round-to-nearest it falls
    short."""
    n, T, G, alpha = 1 << 15, 70, 8, 2.5e-4
    theta0 = random_bf16_bits(n, 5)
    el = np.arange(n, dtype=np.uint64)
    rng = np.random.default_rng(2025)
    rne, sr = theta0.copy(), theta0.copy()
    exact = np.zeros(n)
    for t in range(T):
        seeds = [500 * t + i for i in range(G)]
        r = rng.random(G).astype(np.float32)
        z, _ = oracle.zscore(r)
        c = oracle.update_coefficient(alpha, 0.0, G, 0)
        for s, zi in zip(seeds, z):
            exact += c * zi * oracle.normals(s, 0, el)
        rne, _ = oracle.update(rne, 0, seeds, [1] * G, r, alpha, 0.0)
        sr, _ = oracle.update(sr, 0, seeds, [1] * G, r, alpha, 0.0,
                              flags=ES_UPDATE_STOCHASTIC_ROUND, round_seed=1000 + t)
    t0 = bf16_to_f64(theta0)
    # where |theta| >= 0.04 a typical step is below half a bf16 spacing
    for sel in (np.abs(t0) >= 0.0, np.abs(t0) >= 0.04):
        e = exact[sel]
        fit = {}
        for name, run in (("sr", sr), ("rne", rne)):
            y = (bf16_to_f64(run) - t0)[sel]
            b = y @ e / (e @ e)
            se = math.sqrt(np.sum((y - b * e) ** 2 * e ** 2)) / (e @ e)
            fit[name] = (b, se)
        print("elements", sel.sum(), fit)
        assert abs(fit["sr"][0] - 1.0) < 5 * fit["sr"][1] + 1e-3
        assert fit["rne"][0] < 1.0 - 5 * fit["rne"][1]
