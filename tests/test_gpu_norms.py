"""RMSNorm weights at 1.0, as in a trained model (the 4B-shaped set's 73
norm vectors of 2560): perturb and restore through the C ABI element by
element against the oracle, and the fractions the bf16 grid fixes around 1.0
(the perturbation rounds away on 97.5 % of elements; the revert lands one
step below 1 on 2.5 %) against the closed forms of tests/test_oracle_es.py."""
import math

import numpy as np
import pytest
import torch
from scipy import stats

import oracle
from paper_2608_17310_amd import esopt, workloads as wl
from parity import assert_parity, perturb_delta, report, to_host

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)


def test_unit_norm_vectors_match_oracle_and_closed_forms():
    W = wl.WORKLOADS["dense-4b"]
    vec = [i for i, s in enumerate(W.shapes) if len(s) == 1]
    assert len(vec) == 73
    views = [torch.ones(W.numels[i], dtype=torch.bfloat16, device="cuda") for i in vec]
    one = to_host(views[0][:1])[0]
    s = float(np.float32(1e-3))
    lo, hi = 2.0 ** -9 / s, 2.0 ** -8 / s
    with esopt.Plan(views, tensor_ids=vec) as p:
        p.perturb(31, 1, 1e-3)
        torch.cuda.synchronize()
        pert = [to_host(v) for v in views]
        p.restore(31, 1, 1e-3)
        torch.cuda.synchronize()
        back = [to_host(v) for v in views]
    checks = {"perturb": ([], [], [], []), "restore": ([], [], [], [])}
    for i, x1, x2 in zip(vec, pert, back):
        el = np.arange(x1.size, dtype=np.uint64)
        x0 = np.full(x1.size, one, np.uint16)
        for name, got, base, exp, d in (
                ("perturb", x1, x0, oracle.perturb(x0, 31, i, 1, 1e-3, elems=el),
                 perturb_delta(31, i, 1, 1e-3, el)),
                ("restore", x2, x1, oracle.restore(x1, 31, i, 1, 1e-3, elems=el),
                 perturb_delta(31, i, -1, 1e-3, el))):
            for lst, v in zip(checks[name], (got, exp, base, d)):
                lst.append(v)
    for name, lists in checks.items():
        rep = report(*[np.concatenate(x) for x in lists])
        print("unit norms:", name, rep)
        assert_parity(rep, name)
    x1, x2 = np.concatenate(pert), np.concatenate(back)
    n = x1.size
    for frac, expect in [(np.mean(x1 == one), stats.norm.cdf(hi) - stats.norm.cdf(-lo)),
                         (np.mean(x2 != one), stats.norm.cdf(hi) - stats.norm.cdf(lo))]:
        se = math.sqrt(expect * (1 - expect) / n)
        print(f"fraction {frac:.5f} against {expect:.5f} (5 s.e. {5 * se:.5f})")
        assert abs(frac - expect) < 5 * se
    assert np.all(oracle.bf16_to_f64(x2[x2 != one]) == 1 - 2.0 ** -8)
