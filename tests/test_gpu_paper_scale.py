"""A run of the paper's length on the 27B-shaped set: G = 8 one-sided members,
70 updates, sigma 1.5e-3, alpha 2.5e-4 (the 27B setting of Appendix D.4),
synthetic rewards.  Every pass of every generation is checked on sampled
elements against the oracle applied to the GPU's own state before that pass
(so a legitimate 1-ulp tie of one pass is not carried into the next pass's
expected values), pooled at the parity bar.  The run is then rebuilt from its
JSON seed log on freshly generated starting parameters with the fused passes
(swaps, and the last revert inside the update), and every generation's
recorded checksum is verified: the reconstruction protocol of Section 3 and
Appendix D.6 at full scale."""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_17310_amd import esopt, workloads as wl
from paper_2608_17310_amd.generation import GenerationRecord, load_log, replay, save_log
from parity import assert_parity, perturb_delta, report, to_host, update_delta

pytestmark = pytest.mark.gpu

G, T, SIGMA, ALPHA = 8, 70, 1.5e-3, 2.5e-4


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)


def _samples(W, rng):
    """(tensor index, local indices) of sampled elements: 512 from each of a
    few tensors of every kind (embedding, attention, MLP, norm, head), the
    first and last elements included."""
    names = {0: "embedding", 1: "q", 2: "k", 5: "gate", 7: "down", 8: "norm",
             len(W.shapes) - 2: "final norm", len(W.shapes) - 1: "head"}
    out = []
    for t in sorted(names):
        n = W.numels[t]
        idx = np.unique(np.concatenate([[0, n - 1], rng.integers(0, n, 510)])).astype(np.int64)
        out.append((t, idx))
    return out


class Sampler:
    def __init__(self, views, samples):
        self.parts = [(t, idx, views[t].reshape(-1), torch.from_numpy(idx).cuda())
                      for t, idx in samples]

    def bits(self):
        torch.cuda.synchronize()
        return [to_host(v.index_select(0, i)) for _, _, v, i in self.parts]


def test_seventy_generations_match_the_oracle_and_replay_from_the_log(tmp_path):
    W = wl.WORKLOADS["dense-27b"]
    rng = np.random.default_rng(1958)
    flat, views = wl.device_params(W)
    plan = esopt.Plan(views)
    sm = Sampler(views, _samples(W, rng))
    els = [idx.astype(np.uint64) for _, idx, _, _ in sm.parts]
    tids = [t for t, _, _, _ in sm.parts]
    got, exp, base, delta = [], [], [], []

    def check(before, after, fn, dfn):
        for x0, x1, t, el in zip(before, after, tids, els):
            got.append(x1)
            exp.append(fn(x0, t, el))
            base.append(x0)
            delta.append(dfn(t, el))

    records = []
    for g in range(T):
        seeds = [int(s) for s in 10_000 * (g + 1) + np.arange(G)]
        signs = [1] * G
        rewards = rng.random(G).astype(np.float32)
        x = sm.bits()
        plan.perturb(seeds[0], 1, SIGMA)
        y = sm.bits()
        check(x, y, lambda b, t, el: oracle.perturb(b, seeds[0], t, 1, SIGMA, elems=el),
              lambda t, el: perturb_delta(seeds[0], t, 1, SIGMA, el))
        for i in range(G - 1):
            plan.swap(seeds[i], 1, seeds[i + 1], 1, SIGMA)
            x, y = y, sm.bits()
            check(x, y,
                  lambda b, t, el: oracle.swap(b, t, seeds[i], 1, SIGMA, seeds[i + 1], 1, SIGMA,
                                               elems=el),
                  lambda t, el: (perturb_delta(seeds[i], t, -1, SIGMA, el)
                                 + perturb_delta(seeds[i + 1], t, 1, SIGMA, el)))
        plan.restore(seeds[-1], 1, SIGMA)
        x, y = y, sm.bits()
        check(x, y, lambda b, t, el: oracle.restore(b, seeds[-1], t, 1, SIGMA, elems=el),
              lambda t, el: perturb_delta(seeds[-1], t, -1, SIGMA, el))
        plan.update(seeds, signs, torch.from_numpy(rewards).cuda(), ALPHA, sigma=SIGMA)
        x, y = y, sm.bits()
        check(x, y,
              lambda b, t, el: oracle.update(b, t, seeds, signs, rewards, ALPHA, SIGMA,
                                             elems=el)[0],
              lambda t, el: update_delta(t, seeds, signs, rewards, ALPHA, SIGMA, 0, el))
        records.append(GenerationRecord(seeds, signs, [float(r) for r in rewards], SIGMA, ALPHA,
                                        fused_swap=True, checksum=plan.checksum()))
    final = [to_host(v.reshape(-1)[:: 1 << 16]) for v in views]
    rep = report(np.concatenate(got), np.concatenate(exp), np.concatenate(base),
                 np.concatenate(delta))
    print(f"{T} generations x {G + 2} passes on {sum(e.size for e in els)} sampled elements:",
          rep)
    assert_parity(rep, "paper-length run")
    plan.close()
    del flat, views, plan
    torch.cuda.empty_cache()

    # rebuild from the log, with the fused passes, verifying every checksum
    save_log(tmp_path / "run.json", records, meta={"workload": W.name})
    recs, meta = load_log(tmp_path / "run.json")
    assert meta["workload"] == W.name and len(recs) == T
    flat2, views2 = wl.device_params(W)
    with esopt.Plan(views2) as p:
        replay(p, recs)                  # raises ReplayMismatch at the first differing generation
        assert p.checksum() == records[-1].checksum
    for v, f in zip(views2, final):
        np.testing.assert_array_equal(to_host(v.reshape(-1)[:: 1 << 16]), f)
