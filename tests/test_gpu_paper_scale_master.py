"""The paper-length run of tests/test_gpu_paper_scale.py (27B-shaped set, G = 8
one-sided members, 70 updates, sigma 1.5e-3, alpha 2.5e-4: Appendix D.4) with
binary32 masters of all 22.7 G parameters (91 GB beside the 45 GB bf16 copy):
after every update the sampled masters match the oracle's update_master of
the GPU's masters before it, within the bar derived from the kernel's
arithmetic, and the sampled bf16 values are their nearest-even rounding bit
for bit; the run is then rebuilt from its JSON seed log by its updates alone
(no perturbation is replayed) on regenerated starting masters and other
bf16 values, every recorded checksum verified."""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_17310_amd import esopt, workloads as wl
from paper_2608_17310_amd.generation import load_log, replay, run_generation, save_log
from parity import assert_master_parity, master_report, master_tolerance, to_host

pytestmark = pytest.mark.gpu

G, T, SIGMA, ALPHA = 8, 70, 1.5e-3, 2.5e-4


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)


def _plan(W, seed):
    """bf16 parameters from `seed` and binary32 masters of the set's
    parameters drawn with seed 1958 (the same masters for any `seed`)."""
    flat, views = wl.device_params(W, seed=1958)
    mflat = flat.float()
    base = flat.data_ptr()
    masters = [mflat[(v.data_ptr() - base) // 2:][:v.numel()] for v in views]
    if seed != 1958:                             # other bf16 values, same masters
        flat2, _ = wl.device_params(W, seed=seed)
        flat.copy_(flat2)
        del flat2
    plan = esopt.Plan(views)
    plan.set_master(masters)
    return plan, flat, mflat, views, masters


def test_seventy_generations_into_masters_and_replay_from_updates(tmp_path):
    W = wl.WORKLOADS["dense-27b"]
    rng = np.random.default_rng(1959)
    plan, flat, mflat, views, masters = _plan(W, 1958)
    pick = {0: "embedding", 1: "q", 7: "down", 8: "norm", len(W.shapes) - 1: "head"}
    samples = []
    for t in sorted(pick):
        n = W.numels[t]
        idx = np.unique(np.concatenate([[0, n - 1], rng.integers(0, n, 1022)])).astype(np.int64)
        samples.append((t, idx, torch.from_numpy(idx).cuda()))

    def sample():
        torch.cuda.synchronize()
        return ([masters[t].index_select(0, i).cpu().numpy() for t, _, i in samples],
                [to_host(views[t].reshape(-1).index_select(0, i)) for t, _, i in samples])

    records, reps = [], []
    m_prev, _ = sample()
    for g in range(T):
        seeds = [int(s) for s in 20_000 * (g + 1) + np.arange(G)]
        rewards = rng.random(G).astype(np.float32)
        rec = run_generation(plan, seeds, [1] * G, SIGMA, ALPHA, lambda i: float(rewards[i]),
                             checksum=True)
        assert rec.flags & esopt.ES_UPDATE_MASTER
        records.append(rec)
        m_now, b_now = sample()
        r32 = np.array(rec.rewards, np.float32)
        z, _ = oracle.zscore(r32)
        d, w = oracle.member_weights(seeds, [1] * G, z, oracle.update_coefficient(ALPHA, SIGMA, G))
        live = [(sd, wd) for sd, wd in zip(d, w) if wd != 0.0]
        for (t, idx, _), m0, m1, b1 in zip(samples, m_prev, m_now, b_now):
            el = idx.astype(np.uint64)
            exp, _, _ = oracle.update_master(m0, t, seeds, [1] * G, r32, ALPHA, SIGMA, elems=el)
            reps.append(master_report(m1, exp, master_tolerance(exp, live, t, el)))
            np.testing.assert_array_equal(b1, oracle.f64_to_bf16_rne(m1.astype(np.float64)))
        m_prev = m_now
    bad = sum(r["bad"] for r in reps)
    n = sum(r["n"] for r in reps)
    exact = sum(r["exact"] * r["n"] for r in reps) / n
    worst = max(r["max_err_over_tol"] for r in reps)
    print(f"{T} updates into masters on {n // T} sampled elements: exact {exact:.4f}, "
          f"largest error {worst:.3f} of the bound, beyond it {bad}")
    assert_master_parity({"bad": bad}, "paper-length run into masters")
    final_m, final_b = m_prev, sample()[1]
    plan.close()
    del plan, flat, mflat, views, masters
    torch.cuda.empty_cache()

    save_log(tmp_path / "run.json", records, meta={"workload": W.name, "masters": True})
    recs, _ = load_log(tmp_path / "run.json")
    plan2, flat2, mflat2, views2, masters2 = _plan(W, 77)      # other bf16 values
    replay(plan2, recs)                  # updates only; raises at the first checksum mismatch
    for (t, _, i), m, b in zip(samples, final_m, final_b):
        torch.cuda.synchronize()
        np.testing.assert_array_equal(masters2[t].index_select(0, i).cpu().numpy(), m)
        np.testing.assert_array_equal(to_host(views2[t].reshape(-1).index_select(0, i)), b)
    plan2.close()
