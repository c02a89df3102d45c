"""Pins of the oracle's fp8 (E4M3) path: the decoder against an exact
enumeration of the format written here and against PyTorch's float8_e4m3fn,
the grid floor against a brute-force scan, the rounding rules enumerated over
all their draws, exact revert inside a binade for every code, an
element-by-element pure-Python rendering (big-integer Philox, math-library
Box-Muller, explicit grid search), unbiasedness, the multi-step update and
the identities."""
import math
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle
from oracle import fp8, philox4x32_10_bigint, ES_REWARDS_ARE_WEIGHTS, ES_UPDATE_DIV_SIGMA


def _exact_value(code):
    """The value of one E4M3 code as an exact fraction (None: not a number),
    from the format: significand (8 [e > 0] + m) / 8 times 2^(max(e, 1) - 7)."""
    sign = -1 if code & 0x80 else 1
    e, m = (code >> 3) & 0xF, code & 7
    if e == 15 and m == 7:
        return None
    sig = (8 if e else 0) + m
    return sign * Fraction(sig, 8) * Fraction(2) ** (max(e, 1) - 7)


EXACT = {c: _exact_value(c) for c in range(256)}
FINITE = sorted({v for v in EXACT.values() if v is not None})


def test_decoder_matches_the_exact_enumeration():
    got = fp8.e4m3_decode(np.arange(256))
    for c in range(256):
        if EXACT[c] is None:
            assert math.isnan(got[c]), c
        else:
            assert Fraction(got[c]) == EXACT[c], c
    assert len(FINITE) == 253 and FINITE[-1] == 448 and FINITE[0] == -448
    assert np.array_equal(fp8.GRID, np.array([float(v) for v in FINITE]))
    # smallest subnormal, smallest normal, one below and one at a binade edge
    assert got[0x01] == 2.0 ** -9 and got[0x08] == 2.0 ** -6 and got[0x37] == 0.9375 and got[0x3F] == 1.875
    assert got[0x38] == 1.0 and got[0x80] == 0.0 and math.copysign(1, got[0x80]) < 0


def test_decoder_matches_torch_float8_e4m3fn():
    codes = torch.arange(256, dtype=torch.uint8)
    ref = codes.view(torch.float8_e4m3fn).to(torch.float64).numpy()
    got = fp8.e4m3_decode(np.arange(256))
    assert np.array_equal(np.isnan(ref), np.isnan(got))
    ok = ~np.isnan(ref)
    assert np.array_equal(ref[ok], got[ok])


def test_encode_inverts_decode_and_matches_torch_on_the_grid():
    finite = [c for c in range(256) if EXACT[c] is not None and c != 0x80]
    vals = fp8.e4m3_decode(np.array(finite))
    assert np.array_equal(fp8.e4m3_encode(vals), np.array(finite, dtype=np.uint8))
    assert fp8.e4m3_encode(np.array([-0.0]))[0] == 0
    ref = torch.from_numpy(fp8.GRID).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    enc = fp8.e4m3_encode(fp8.GRID)
    assert np.array_equal(ref[fp8.GRID != 0], enc[fp8.GRID != 0])
    with pytest.raises(ValueError):
        fp8.e4m3_encode(np.array([0.3]))


def test_grid_floor_against_a_brute_force_scan():
    rng = np.random.default_rng(1)
    grid = [float(v) for v in FINITE]
    xs = np.concatenate([
        fp8.GRID[:-1], (fp8.GRID[:-1] + fp8.GRID[1:]) / 2,
        np.nextafter(fp8.GRID[1:], -np.inf), rng.uniform(-448, 448, 3000),
        rng.normal(0, 0.02, 1000), rng.normal(0, 3, 1000)])
    xs = xs[(xs >= -448) & (xs < 448)]
    lo, h = fp8.grid_floor(xs)
    for x, l, hh in zip(xs.tolist(), lo.tolist(), h.tolist()):
        below = [g for g in grid if g <= x]
        assert l == below[-1]
        assert l + hh == grid[grid.index(l) + 1]
    with pytest.raises(ValueError):
        fp8.grid_floor(np.array([448.0]))


def _f32(x):
    return float(np.float32(x))


@pytest.mark.parametrize("x", [0.0, 1.0, 1.06, -1.06, 100.3, -100.3, 2.0 ** -12, -3e-3,
                               0.01, 447.0, -447.9, 15.99, 16.01, -0.9999])
def test_perturbation_rounding_enumerated_over_all_512_draws(x):
    x = _f32(x)
    r = np.arange(512)
    u = (2 * r + 1) * 2.0 ** -10
    res = fp8.round_onto_grid(np.full(512, x), "perturb", u)
    lo, h = fp8.grid_floor(np.array([x]))
    lo, h = float(lo[0]), float(h[0])
    assert set(np.unique(res)) <= {lo, lo + h}
    f = (x - lo) / h
    assert np.sum(res == lo + h) == np.sum(u >= 1 - f)
    assert abs(res.mean() - x) <= 2.0 ** -10 * h


@pytest.mark.parametrize("k1024,g", [(1, 120), (511, 100), (512, 30), (513, -30), (1023, 60),
                                     (77, 0), (601, -100), (3, -126)])
def test_restore_rounding_enumerated_over_all_512_draws(k1024, g):
    """y at a fraction k / 1024 of its grid interval (on the draws' own
    2^-10 grid, so f equals some u exactly): restore steps for exactly the
    draws with u < f, strictly."""
    lo = fp8.GRID[fp8.GRID.size // 2 + g]
    h = fp8.GRID[fp8.GRID.size // 2 + g + 1] - lo
    y = lo + k1024 * 2.0 ** -10 * h
    assert _f32(y) == y
    u = (2 * np.arange(512) + 1) * 2.0 ** -10
    res = fp8.round_onto_grid(np.full(512, y), "restore", u)
    assert set(np.unique(res)) <= {lo, lo + h}
    f = k1024 / 1024.0
    assert np.sum(res == lo + h) == np.sum(u < f)
    if k1024 % 2:                               # f equals one of the u: that draw does not step
        assert res[(k1024 - 1) // 2] == lo


def test_decisions_are_taken_on_the_binary32_value():
    """The rounding decides on x rounded to binary32 (the kernels' precision):
    elements whose fp64 x lies just below a perturbation threshold and whose
    binary32 x reaches it step, checked against a grid scan on the binary32
    value and shown to differ from deciding on the fp64 value."""
    n, sig, seed, tid = 1 << 21, 1e-3, 4242, 3          # this seed has two such elements
    el = np.arange(n, dtype=np.uint64)
    eps = oracle.normals(seed, tid, el)
    scale = np.float32(1e-4)
    v = 96.0                                    # code 0x6C: grid spacing 8 around it
    d = _f32(sig) * eps / float(scale)
    u = (2 * oracle.spare_draws(seed, tid, el).astype(np.float64) + 1) * 2.0 ** -10
    x64 = v + d
    x32 = np.vectorize(_f32)(x64)
    # elements whose result depends on the precision of the decision
    flips = np.flatnonzero((fp8.round_onto_grid(x64, "perturb", u)
                            != fp8.round_onto_grid(x32, "perturb", u)) & (np.abs(x64) < 440))
    assert flips.size >= 2
    codes = np.full(flips.size, 0x6C, np.uint8)
    assert fp8.e4m3_decode(codes)[0] == v
    got = fp8.f8perturb(codes, np.array([scale]), 0, seed, tid, 1, sig, elems=el[flips])
    for j, g in zip(flips.tolist(), got.tolist()):
        expect = _py_round(x32[j], lambda f, uu=u[j]: f >= 1 - uu)
        assert float(EXACT[g]) == expect
        assert expect != _py_round(float(x64[j]), lambda f, uu=u[j]: f >= 1 - uu)


@pytest.mark.parametrize("n16,k", [(0, 5), (1, 5), (32768, 40), (65535, 77), (12345, -40),
                                   (7, -120), (40000, 3), (99, -7)])
def test_update_rounding_enumerated_over_all_65536_draws(n16, k):
    # x on the 2^-16 h sub-grid of the interval above grid point k
    lo = fp8.GRID[fp8.GRID.size // 2 + k]
    h = fp8.GRID[fp8.GRID.size // 2 + k + 1] - lo
    x = lo + n16 * 2.0 ** -16 * h
    assert _f32(x) == x
    u = np.arange(65536) * 2.0 ** -16
    res = fp8.round_onto_grid(np.full(65536, x), "update", u)
    assert set(np.unique(res)) <= {lo, lo + h}
    assert np.sum(res == lo + h) == n16
    assert res.sum() / 65536.0 == x                       # exact mean
    # the step is taken by the top draws
    assert np.all(res[65536 - n16:] == lo + h)


def test_clamping_at_the_largest_value():
    u = np.array([0.001, 0.5, 0.999])
    for rule in ("perturb", "restore", "update"):
        assert np.all(fp8.round_onto_grid(np.full(3, 460.0), rule, u) == 448)
        assert np.all(fp8.round_onto_grid(np.full(3, 448.0), rule, u) == 448)
        assert np.all(fp8.round_onto_grid(np.full(3, -1e6), rule, u) == -448)
        assert np.all(fp8.round_onto_grid(np.full(3, -448.0), rule, u) == -448)


def test_restore_is_exact_inside_a_binade_for_every_code():
    """For every finite code, steps d of many sizes and every 16th 9-bit
    draw: wherever x = c + d, the perturbed value and y = p - d keep the
    code's sign and binary32 exponent (one binade of the grid, outside the
    subnormal band) and x does not clamp at 448, restore returns the code
    exactly."""
    rng = np.random.default_rng(2)
    codes = np.array([c for c in range(256) if EXACT[c] is not None and EXACT[c] != 0])
    v = fp8.e4m3_decode(codes)
    n_exact = n_in = 0
    for r9 in range(0, 512, 16):
        u = (2 * r9 + 1) * 2.0 ** -10
        d = rng.normal(0, 1, (codes.size, 60)) * np.abs(v)[:, None] * rng.choice(
            [0.01, 0.05, 0.2], (codes.size, 60))
        x = np.vectorize(_f32)(v[:, None] + d)
        p = fp8.round_onto_grid(x, "perturb", np.full(x.shape, u))
        y = np.vectorize(_f32)(p - d)
        back = fp8.round_onto_grid(y, "restore", np.full(x.shape, u))
        e = lambda a: np.frexp(np.abs(a))[1]
        same = ((np.sign(x) == np.sign(v[:, None])) & (np.sign(y) == np.sign(v[:, None]))
                & (np.sign(p) == np.sign(v[:, None]))
                & (e(x) == e(v)[:, None]) & (e(p) == e(v)[:, None]) & (e(y) == e(v)[:, None])
                & (np.abs(v)[:, None] >= 2.0 ** -6) & (np.abs(x) < 448))
        exact = back == v[:, None]
        assert np.all(exact[same]), np.argwhere(same & ~exact)[:5]
        n_in += int(same.sum())
        n_exact += int(exact.sum())
    assert n_in > 100000


def test_perturb_then_restore_on_quantized_weights():
    """Seed replay on per-row E4M3 codes of N(0, 0.02) weights at sigma = 1e-3:
    the perturbation moves most codes, most reverts are exact, and a revert
    that is not exact (a perturbation that crossed into a coarser binade, or
    clamped) is off by at most one step of the coarser grid it touched."""
    n, row = 1 << 16, 1024
    w = np.random.default_rng(3).normal(0, 0.02, n)
    scales = (np.abs(w).reshape(-1, row).max(axis=1) / 448).astype(np.float32)
    s = np.repeat(scales.astype(np.float64), row)
    c0 = torch.from_numpy(w / s).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    p = fp8.f8perturb(c0, scales, row, 77, 5, 1, 1e-3)
    back = fp8.f8restore(p, scales, row, 77, 5, 1, 1e-3)
    v0, vp, vb = fp8.e4m3_decode(c0), fp8.e4m3_decode(p), fp8.e4m3_decode(back)
    exact = vb == v0
    assert np.mean(vp != v0) > 0.5
    assert np.mean(exact) > 0.9, np.mean(exact)
    coarse = np.minimum(np.maximum(np.abs(v0), np.abs(vp)), 447.99)
    _, h = fp8.grid_floor(coarse)
    assert np.all(np.abs(vb - v0) <= h), np.max(np.abs(vb - v0) / h)


def _word_normal(w_a, w_b, first):
    m_a, m_b = w_a & 0x7FFFFF, w_b & 0x7FFFFF
    u = (m_a + 0.5) * 2.0 ** -23
    phi = 2.0 * math.pi * m_b * 2.0 ** -23
    rad = math.sqrt(-2.0 * math.log(u))
    return rad * math.cos(phi) if first else rad * math.sin(phi)


def _words(seed, tid, j):
    q = j >> 2
    return philox4x32_10_bigint((q & 0xFFFFFFFF, q >> 32, tid, 0), (seed & 0xFFFFFFFF, seed >> 32))


def _eps(seed, tid, j):
    w = _words(seed, tid, j)
    lane = j & 3
    pair = (w[0], w[1]) if lane < 2 else (w[2], w[3])
    return _word_normal(pair[0], pair[1], lane % 2 == 0)


def _draw16(seed, tid, j):
    g = j >> 3
    w = philox4x32_10_bigint((g & 0xFFFFFFFF, g >> 32, tid, 1), (seed & 0xFFFFFFFF, seed >> 32))
    return (w[(j & 7) >> 1] >> (16 * (j & 1))) & 0xFFFF


def _py_round(x, step_if):
    """Round a float onto the grid of exact values by a linear scan."""
    if x >= 448:
        return 448.0
    if x <= -448:
        return -448.0
    grid = [float(g) for g in FINITE]
    i = max(k for k, g in enumerate(grid) if g <= x)
    lo, hi = grid[i], grid[i + 1]
    return (hi if step_if((x - lo) / (hi - lo)) else lo) + 0.0


def test_pure_python_rendering_matches_perturb_restore_and_update():
    rng = np.random.default_rng(5)
    n, row, tid, seed = 3000, 24, 11, (1 << 40) + 17
    c = rng.integers(0, 256, n).astype(np.uint8)
    scales = rng.uniform(2e-4, 1e-3, n // row + 1).astype(np.float32)
    scales[3] = 0.0                                       # an invalid row: left unchanged
    elems = np.concatenate([np.arange(80), rng.integers(0, n, 60)]).astype(np.uint64)
    cs = c[elems.astype(np.int64)]
    sig = _f32(1e-3)
    for name, fn, sgn in (("perturb", fp8.f8perturb, 1), ("restore", fp8.f8restore, -1)):
        got = fn(cs, scales, row, seed, tid, -1, 1e-3, elems=elems)
        for j, code, g in zip(elems.tolist(), cs.tolist(), got.tolist()):
            s = float(scales[j // row])
            val = EXACT[code]
            if not s >= 2.0 ** -126 or val is None:
                assert g == code
                continue
            d = -sig * _eps(seed, tid, j) / s
            u = (2 * (_words(seed, tid, j)[j & 3] >> 23) + 1) * 2.0 ** -10
            x = _f32(float(val) + sgn * d)
            rule = (lambda f, u=u: f >= 1 - u) if name == "perturb" else (lambda f, u=u: f > u)
            assert float(EXACT[g]) == _py_round(x, rule), (name, j)
    seeds, signs, w = [3, 8], [1, -1], np.array([0.7, -0.2], np.float32)
    alpha, rs = 2e-3, 99
    got, st = fp8.f8update(cs, scales, row, tid, seeds, signs, w, alpha, 0.0,
                           flags=ES_REWARDS_ARE_WEIGHTS, elems=elems, round_seed=rs)
    assert st == 0
    coef = _f32(alpha) / 2
    for j, code, g in zip(elems.tolist(), cs.tolist(), got.tolist()):
        s = float(scales[j // row])
        val = EXACT[code]
        if not s >= 2.0 ** -126 or val is None:
            assert g == code
            continue
        delta = sum(coef * sg * float(wi) * _eps(sd, tid, j) for sd, sg, wi in zip(seeds, signs, w))
        x = _f32(float(val) + delta / s)
        r = _draw16(rs, tid, j)
        assert float(EXACT[g]) == _py_round(x, lambda f: f >= 1 - r * 2.0 ** -16), j


def test_perturbation_and_update_are_unbiased():
    n, row = 1 << 17, 0
    scales = np.array([2.2e-4], np.float32)
    rng = np.random.default_rng(6)
    c = torch.from_numpy(rng.normal(0, 90, n)).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    v = fp8.e4m3_decode(c)
    el = np.arange(n, dtype=np.uint64)
    p = fp8.f8perturb(c, scales, row, 41, 2, 1, 1e-3)
    d = _f32(1e-3) * oracle.normals(41, 2, el) / float(scales[0])
    x = np.vectorize(_f32)(v + d)
    lo, h = fp8.grid_floor(np.clip(x, -448, 447.99))
    f = (x - lo) / h
    err = np.sum(fp8.e4m3_decode(p) - x)
    assert abs(err) < 5 * math.sqrt(np.sum(h * h * f * (1 - f))) + n * 2.0 ** -10 * h.mean()
    r = rng.random(8).astype(np.float32)
    got, st = fp8.f8update(c, scales, row, 2, list(range(50, 58)), [1] * 8, r, 5e-4, 0.0,
                           round_seed=4)
    z, _ = oracle.zscore(r)
    coef = oracle.update_coefficient(5e-4, 0.0, 8, 0)
    delta = sum(coef * zi * oracle.normals(sd, 2, el) for sd, zi in zip(range(50, 58), z))
    x = np.vectorize(_f32)(v + delta / float(scales[0]))
    lo, h = fp8.grid_floor(np.clip(x, -448, 447.99))
    f = (x - lo) / h
    err = np.sum(fp8.e4m3_decode(got) - x)
    assert abs(err) < 5 * math.sqrt(np.sum(h * h * f * (1 - f)))
    # the steps are a fraction of a grid step: rounding to nearest would drop most
    assert np.mean(np.abs(delta / float(scales[0])) < h / 2) > 0.8
    assert np.mean(got != c) > 0.02


def test_multistep_update_tracks_unrounded_sum():
    """70 updates (G = 8, alpha = 2.5e-4, as in the paper's update-magnitude
    table, Appendix A.1) on per-row E4M3 codes of N(0, 0.02) weights: the
    dequantized total step regresses on the unrounded sum with slope 1."""
    n, row, T, G, alpha = 1 << 14, 256, 70, 8, 2.5e-4
    w = np.random.default_rng(9).normal(0, 0.02, n)
    scales = (np.abs(w).reshape(-1, row).max(axis=1) / 448).astype(np.float32)
    s = np.repeat(scales.astype(np.float64), row)
    c0 = torch.from_numpy(w / s).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    c = c0.copy()
    exact = np.zeros(n)
    rng = np.random.default_rng(10)
    el = np.arange(n, dtype=np.uint64)
    for t in range(T):
        seeds = [700 * t + i for i in range(G)]
        r = rng.random(G).astype(np.float32)
        z, _ = oracle.zscore(r)
        coef = oracle.update_coefficient(alpha, 0.0, G, 0)
        for sd, zi in zip(seeds, z):
            exact += coef * zi * oracle.normals(sd, 0, el)
        c, st = fp8.f8update(c, scales, row, 0, seeds, [1] * G, r, alpha, 0.0, round_seed=t)
        assert st == 0
    moved = (fp8.e4m3_decode(c) - fp8.e4m3_decode(c0)) * s
    b = moved @ exact / (exact @ exact)
    se = math.sqrt(np.sum((moved - b * exact) ** 2 * exact ** 2)) / (exact @ exact)
    assert abs(b - 1.0) < 5 * se + 1e-3, (b, se)


def test_identities():
    rng = np.random.default_rng(11)
    c = rng.integers(0, 256, 4000).astype(np.uint8)
    c[:4] = [0x7F, 0xFF, 0x80, 0x7E]
    scales = rng.uniform(2e-4, 1e-3, 4000 // 8).astype(np.float32)
    scales[5] = np.nan                                    # rows 40..47 left unchanged
    scales[6] = 1e-40                                     # subnormal scale: unchanged
    for fn in (fp8.f8perturb, fp8.f8restore):
        assert np.array_equal(fn(c, scales, 8, 1, 0, 1, 0.0), c)         # sigma = 0
        out = fn(c, scales, 8, 1, 0, 1, 5e-3)
        assert out[0] == 0x7F and out[1] == 0xFF                           # not a number
        assert np.array_equal(out[40:56], c[40:56])                        # invalid scales
        assert np.all(fp8.e4m3_decode(out)[np.isfinite(fp8.e4m3_decode(c))] <= 448)
    r = np.array([0.3, 0.3, 0.3], np.float32)
    out, st = fp8.f8update(c, scales, 8, 0, [1, 2, 3], [1, 1, 1], r, 1e-3, 0.0)
    assert st == 0 and np.array_equal(out, c)                             # equal rewards
    out, st = fp8.f8update(c, scales, 8, 0, [1, 2, 3], [1, 1, 1], np.array([0.1, 0.5, 0.9],
                           np.float32), 0.0, 0.0)
    assert st == 0 and np.array_equal(out, c)                             # alpha = 0
    out, st = fp8.f8update(c, scales, 8, 0, [1, 2], [1, 1], np.array([0.1, np.inf], np.float32),
                           1e-3, 0.0)
    assert st == 1 and np.array_equal(out, c)                             # non-finite reward
    # an antithetic pair with equal rewards cancels
    out, st = fp8.f8update(c, scales, 8, 0, [4, 4, 5], [1, -1, 1],
                           np.array([0.7, 0.7, 0.7], np.float32), 1e-3, 0.0,
                           flags=ES_REWARDS_ARE_WEIGHTS)
    assert st == 0
    # 1/(G sigma) scales the step: a large enough step moves -0 to a nonzero code
    big, _ = fp8.f8update(np.array([0x80] * 64, np.uint8), np.array([1e-3], np.float32), 0, 0,
                          [9], [1], np.array([1.0], np.float32), 1.0, 1e-3,
                          flags=ES_REWARDS_ARE_WEIGHTS | ES_UPDATE_DIV_SIGMA)
    assert np.all(big != 0x80)
    # the largest codes saturate instead of overflowing into not-a-number
    top = np.full(256, 0x7E, np.uint8)
    up, _ = fp8.f8update(top, np.array([1.0], np.float32), 0, 0, [9], [1],
                         np.array([1.0], np.float32), 100.0, 0.0, flags=ES_REWARDS_ARE_WEIGHTS)
    eps = oracle.normals(9, 0, np.arange(256, dtype=np.uint64))
    assert np.all(np.isfinite(fp8.e4m3_decode(up)))
    assert np.all(up[eps > 0] == 0x7E) and np.all(fp8.e4m3_decode(up[eps < -0.5]) < 448)


def test_parity_report_accepts_only_near_threshold_neighbours():
    """The fp8 parity check (tests/parity.py): a result equal to the oracle's
    passes; the other grid neighbour passes only where the oracle's decision
    lies within the tolerance of its threshold; any other code fails."""
    from parity import f8report
    x = np.array([1.0 + 0.5 * 0.125, 1.0 + 0.3 * 0.125, 100.0 + 0.9 * 8, -3.0 - 0.2 * 0.25])
    thr = np.array([0.5 + 1e-9, 0.6, 0.1, 0.7])            # element 0 sits on its threshold
    ok = np.ones(4, bool)
    exp = fp8.e4m3_encode(fp8.round_onto_grid(x, "update", 1.0 - thr))
    tol = np.full(4, 1e-6)
    assert f8report(exp, exp, x, thr, tol, ok)["bad"] == 0
    lo, h = fp8.grid_floor(x)
    v = fp8.e4m3_decode(exp)
    other = fp8.e4m3_encode(np.where(v == lo, lo + h, lo))
    got = exp.copy()
    got[0] = other[0]                                        # near its threshold: accepted
    rep = f8report(got, exp, x, thr, tol, ok)
    assert rep["bad"] == 0 and rep["near"] == 1
    got[1] = other[1]                                        # far from it: rejected
    assert f8report(got, exp, x, thr, tol, ok)["bad"] == 1
    got = exp.copy()
    got[2] = fp8.e4m3_encode(np.array([lo[2] - 8.0]))[0]     # two steps away: rejected
    assert f8report(got, exp, x, thr, tol, ok)["bad"] == 1
