"""es_update_noalloc (the update for callers that cannot allocate) against
es_update through the C ABI: two calls in a row on fresh copies of the same
parameters, the second with a smaller plan and fewer members, give the same
bits, z-scores and status as es_update, and both meet the parity bar against
the oracle; populations above the static array's capacity are refused with
nothing launched; and the calls take no device memory."""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_17310_amd import esopt, workloads as wl
from parity import to_host, report, assert_parity, update_delta

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)


def _copies(sizes, seed):
    bits = [wl.random_bf16_bits(n, seed + i) for i, n in enumerate(sizes)]
    a = [torch.from_numpy(b.view(np.int16)).view(torch.bfloat16).cuda() for b in bits]
    return bits, a, [t.clone() for t in a]


def _update(plan, noalloc, seeds, signs, r, alpha, **kw):
    z = torch.full((len(seeds),), float("nan"), device="cuda")
    st = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    (plan.update_noalloc if noalloc else plan.update)(seeds, signs, r, alpha, z_out=z,
                                                      status_out=st, **kw)
    return z, st


# first call: five tensors (one with three full tiles and ragged ends), 64
# members in antithetic pairs, stochastic rounding; second call: a smaller
# plan, three distinct members, the 1/(G sigma) coefficient
CASES = [
    ([3 * 65536 + 1001, 4097, 1, 70000, 12345], 64,
     dict(flags=esopt.ES_UPDATE_STOCHASTIC_ROUND, round_seed=77)),
    ([20000, 333], 3, dict(flags=esopt.ES_UPDATE_DIV_SIGMA, sigma=1e-3)),
]


def test_two_calls_in_a_row_match_es_update():
    for k, (sizes, n, kw) in enumerate(CASES):
        bits, a, b = _copies(sizes, 500 + 10 * k)
        pa, pb = esopt.Plan(a), esopt.Plan(b)
        rng = np.random.default_rng(k)
        if n % 2 == 0:
            base = [int(x) for x in rng.integers(0, 1 << 63, n // 2)]
            seeds = [s for s in base for _ in (0, 1)]
            signs = [1, -1] * (n // 2)
        else:
            seeds = [int(x) for x in rng.integers(0, 1 << 63, n)]
            signs = [1] * n
        r = torch.from_numpy(rng.random(n).astype(np.float32)).cuda()
        alpha = 5e-4
        za, sa = _update(pa, False, seeds, signs, r, alpha, **kw)
        zb, sb = _update(pb, True, seeds, signs, r, alpha, **kw)
        torch.cuda.synchronize()
        assert int(sa.item()) == 0 and int(sb.item()) == 0
        assert torch.equal(za.view(torch.int32), zb.view(torch.int32)), f"call {k}: z differs"
        pooled = ([], [], [], [])
        for i, (ta, tb) in enumerate(zip(a, b)):
            ga, gb = to_host(ta), to_host(tb)
            assert np.array_equal(ga, gb), f"call {k} tensor {i}: bits differ from es_update"
            el = np.arange(ga.size, dtype=np.uint64)
            exp, st = oracle.update(bits[i], i, seeds, signs, r.cpu().numpy(), alpha,
                                    kw.get("sigma", 0.0), flags=kw.get("flags", 0),
                                    round_seed=kw.get("round_seed", 0))
            assert st == 0
            for acc, part in zip(pooled, (gb, exp, bits[i],
                                          update_delta(i, seeds, signs, r.cpu().numpy(), alpha,
                                                       kw.get("sigma", 0.0), kw.get("flags", 0),
                                                       el))):
                acc.append(part)
        rep = report(*(np.concatenate(x) for x in pooled))
        print("es_update_noalloc call", k, rep)
        assert_parity(rep, f"es_update_noalloc call {k}")
        assert np.mean(np.concatenate(pooled[0]) != np.concatenate(pooled[2])) > 0.3
        pa.close()
        pb.close()


def test_non_finite_reward_and_oversized_population():
    bits, a, b = _copies([5000], 900)
    p = esopt.Plan(b)
    r = torch.tensor([0.1, float("inf"), 0.3], device="cuda")
    z, st = _update(p, True, [1, 2, 3], [1, 1, 1], r, 5e-4)
    torch.cuda.synchronize()
    assert int(st.item()) == 1 and torch.all(z == 0)
    assert np.array_equal(to_host(b[0]), bits[0])
    # more members than the static array holds: refused before any launch
    n = esopt.ES_MAX_MEMBERS + 1
    r = torch.rand(n, device="cuda")
    with pytest.raises(esopt.EsError, match="n_members out of range"):
        p.update_noalloc(list(range(n)), [1] * n, r, 5e-4)
    torch.cuda.synchronize()
    assert np.array_equal(to_host(b[0]), bits[0])
    p.close()


def test_calls_take_no_device_memory():
    bits, a, b = _copies([1 << 20, 4099], 950)
    p = esopt.Plan(b)
    r = torch.rand(32, device="cuda")
    # first calls on this device (the array's address is looked up once; the
    # runtime loads both kernels)
    p.update_noalloc(list(range(32)), [1] * 32, r, 5e-4)
    p.update_noalloc(list(range(32)), [1] * 32, r, 5e-4, flags=esopt.ES_UPDATE_STOCHASTIC_ROUND)
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    free0 = torch.cuda.mem_get_info()[0]
    for rep in range(3):
        p.update_noalloc(list(range(32)), [1] * 32, r, 5e-4,
                         flags=esopt.ES_UPDATE_STOCHASTIC_ROUND, round_seed=rep)
        torch.cuda.synchronize()
        assert torch.cuda.mem_get_info()[0] == free0
    p.close()
