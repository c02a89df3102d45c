"""es_perturb / es_restore on the GPU against the oracle, element by element,
on the 1M-parameter tiny set (4 tensors, several hundred tiles) and on edge
cases: ragged tails, unaligned bases, empty and one-element tensors, zero
sigma, determinism, tensor-id independence."""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_17310_amd import esopt, workloads as wl
from parity import to_device, to_host, report, assert_parity, perturb_delta

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)


def _check_perturb(theta_bits, got_bits, seed, tid, sign, sigma, what):
    el = np.arange(theta_bits.size, dtype=np.uint64)
    exp = oracle.perturb(theta_bits, seed, tid, sign, sigma)
    rep = report(got_bits, exp, theta_bits, perturb_delta(seed, tid, sign, sigma, el))
    print(what, rep)
    assert_parity(rep, what)
    return exp


def test_tiny_config_perturb_restore():
    W = wl.TINY
    host = wl.host_params(W)
    ts = [to_device(b, s) for b, s in zip(host, W.shapes)]
    plan = esopt.Plan(ts)
    assert plan.numel == W.n_params
    for m, (seed, sign) in enumerate(zip(W.seeds, W.signs)):
        before = [to_host(t) for t in ts]
        plan.perturb(seed, sign, W.sigma0)
        torch.cuda.synchronize()
        pert = [to_host(t) for t in ts]
        for i in range(len(ts)):
            _check_perturb(before[i], pert[i], seed, i, sign, W.sigma0, f"perturb m{m} t{i}")
        plan.restore(seed, sign, W.sigma0)
        torch.cuda.synchronize()
        for i in range(len(ts)):
            got = to_host(ts[i])
            # isolated: oracle restore applied to the GPU's perturbed values
            _check_perturb(pert[i], got, seed, i, -sign, W.sigma0, f"restore m{m} t{i}")
            # chained: oracle restore of the oracle perturb
            chained = oracle.restore(oracle.perturb(before[i], seed, i, sign, W.sigma0),
                                     seed, i, sign, W.sigma0)
            el = np.arange(got.size, dtype=np.uint64)
            rep = report(got, chained, before[i], perturb_delta(seed, i, sign, W.sigma0, el))
            # two roundings compound here (a perturb-stage 1-ulp tie carries
            # into the restore), so the share allowed above 1 ulp is the
            # bar's 1e-4 per pass, twice; the isolated check above holds the
            # restore alone to the bar itself
            assert rep["max_ulp"] <= 2.0 and rep["le1"] >= 0.9998, rep
            drift = np.mean(got != before[i])
            assert drift < 0.1, drift
    plan.close()


@pytest.mark.parametrize("sizes", [
    [1, 7, 8, 9, 4095, 4096, 4097, 8191 + 4096],
    [0, 3, 0, 12289],                      # empty tensors in the list
])
def test_ragged_and_empty_tensors(sizes):
    bits = [wl.random_bf16_bits(n, 10 + i) for i, n in enumerate(sizes)]
    ts = [to_device(b) for b in bits]
    plan = esopt.Plan(ts, tensor_ids=[100 + i for i in range(len(ts))])
    plan.perturb(99, -1, 2e-3)
    torch.cuda.synchronize()
    for i, b in enumerate(bits):
        if b.size:
            _check_perturb(b, to_host(ts[i]), 99, 100 + i, -1, 2e-3, f"ragged {sizes[i]}")
    plan.close()


def test_unaligned_tensor_base_uses_checked_path():
    n = 3 * 4096 + 5
    bits = wl.random_bf16_bits(n + 3, 21)
    buf = to_device(bits)
    views = [buf[1:1 + 4100], buf[4101:n + 3]]          # 2-byte, not 16-byte aligned
    plan = esopt.Plan(views)
    before = [to_host(v) for v in views]
    plan.perturb(5, 1, 1e-3)
    torch.cuda.synchronize()
    for i, v in enumerate(views):
        _check_perturb(before[i], to_host(v), 5, i, 1, 1e-3, f"unaligned {i}")
    assert to_host(buf[:1])[0] == bits[0]                 # outside the views untouched
    assert np.array_equal(to_host(buf[n + 3 - 0:]), bits[n + 3:])
    plan.close()


def test_neighbours_untouched_and_zero_sigma_identity():
    n = 10000
    bits = wl.random_bf16_bits(n + 64, 22)
    bits[40:48] = [0x8000, 0, 0x8000, 0, 1, 0x8001, 0x7F7F, 0xFF7F]
    buf = to_device(bits)
    view = buf[32:32 + n]
    plan = esopt.Plan([view])
    plan.perturb(1, 1, 0.0)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(to_host(buf), bits)
    plan.perturb(1, 1, 1e-3)
    torch.cuda.synchronize()
    out = to_host(buf)
    np.testing.assert_array_equal(out[:32], bits[:32])
    np.testing.assert_array_equal(out[32 + n:], bits[32 + n:])
    plan.close()


def test_deterministic_and_restore_equals_negated_perturb():
    bits = wl.random_bf16_bits(1 << 18, 23)
    a, b = to_device(bits), to_device(bits)
    pa, pb = esopt.Plan([a]), esopt.Plan([b])
    pa.perturb(8, 1, 1e-3)
    pb.perturb(8, 1, 1e-3)
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    pa.restore(9, 1, 1e-3)
    pb.perturb(9, -1, 1e-3)
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    pa.close(); pb.close()


def test_tensor_id_and_seed_select_the_noise():
    bits = np.zeros(1 << 14, dtype=np.uint16)
    a, b, c = to_device(bits), to_device(bits), to_device(bits)
    plan = esopt.Plan([a, b, c], tensor_ids=[3, 4, 3 + (1 << 20)])
    plan.perturb(1, 1, 1.0)
    torch.cuda.synchronize()
    ha, hb, hc = to_host(a), to_host(b), to_host(c)
    assert np.mean(ha == hb) < 0.01 and np.mean(ha == hc) < 0.01
    _check_perturb(bits, ha, 1, 3, 1, 1.0, "tid 3")
    _check_perturb(bits, hc, 1, 3 + (1 << 20), 1, 1.0, "tid 2^20+3")
    plan.close()


def test_invalid_arguments_raise():
    t = to_device(wl.random_bf16_bits(64, 1))
    with pytest.raises(ValueError):
        esopt.Plan([t.float()])
    with pytest.raises(esopt.EsError):
        esopt.Plan([t, t])                               # overlapping / duplicate storage
    plan = esopt.Plan([t])
    with pytest.raises(esopt.EsError):
        plan.perturb(1, 0, 1e-3)
    with pytest.raises(esopt.EsError):
        plan.perturb(1, 1, float("nan"))
    plan.close()


@pytest.mark.parametrize("shape", [(256, 4, 1, 1), (512, 8, 2, 3), (1024, 4, 1, 8), (256, 8, 4, 2)])
def test_results_do_not_depend_on_launch_shape(shape, monkeypatch):
    """Noise is a function of (seed, tensor, element) only, so the tile shape
    and grid (environment overrides read at plan creation) change no bit of
    perturb, swap, restore, update (both roundings, and into masters) or a
    member applied from the masters."""
    threads, groups, wg_p, wg_u = shape
    sizes = [300001, 1 << 16, 4097, 9]
    bits = [wl.random_bf16_bits(n, 90 + i) for i, n in enumerate(sizes)]
    r = torch.tensor([0.3, 0.9, 0.1, 0.5], dtype=torch.float32, device="cuda")

    def run():
        ts = [to_device(b) for b in bits]
        views = [ts[0][1:], ts[1], ts[2], ts[3]]
        plan = esopt.Plan(views)
        out = []
        plan.perturb(3, 1, 1e-3)
        plan.swap(3, 1, 4, -1, 1e-3)
        plan.restore(4, -1, 1e-3)
        out.append([to_host(t) for t in ts])
        plan.update([1, 2, 2, 5], [1, 1, -1, 1], r, 5e-4)
        plan.update([1, 2, 2, 5], [1, 1, -1, 1], r, 5e-4, flags=esopt.ES_UPDATE_STOCHASTIC_ROUND,
                    round_seed=77)
        torch.cuda.synchronize()
        out.append([to_host(t) for t in ts])
        masters = [v.float() for v in views]             # binary32 masters of the result
        plan.set_master(masters)
        plan.update([6, 7], [1, -1], r[:2], 5e-4, flags=esopt.ES_UPDATE_MASTER)
        torch.cuda.synchronize()
        out.append([to_host(t) for t in ts] + [m.cpu().numpy() for m in masters])
        plan.perturb_master(8, -1, 2e-3)                 # a member applied from them
        torch.cuda.synchronize()
        out.append([to_host(t) for t in ts])
        plan.close()
        return out

    ref = run()
    for k, v in (("ESOPT_THREADS", threads), ("ESOPT_GROUPS", groups),
                 ("ESOPT_PERTURB_WG_PER_CU", wg_p), ("ESOPT_UPDATE_WG_PER_CU", wg_u)):
        monkeypatch.setenv(k, str(v))
    got = run()
    for a, b in zip(ref, got):
        for x, y in zip(a, b):
            np.testing.assert_array_equal(x, y)


def test_stream_pass_rewrites_values_unchanged():
    bits = [wl.random_bf16_bits(n, 95 + i) for i, n in enumerate([300001, 1 << 16, 9])]
    # zeros, infinities, subnormals and NaNs with payloads: written back bit for bit
    bits[0][:9] = [0x0000, 0x8000, 0x7F80, 0xFF80, 0x0001, 0x807F, 0x7FC1, 0xFF81, 0x7F81]
    ts = [to_device(b) for b in bits]
    plan = esopt.Plan([ts[0][1:], ts[1], ts[2]])
    plan.stream_pass()
    plan.stream_pass()
    torch.cuda.synchronize()
    for b, t in zip(bits, ts):
        np.testing.assert_array_equal(to_host(t), b)
    plan.close()
