"""A plan at the maximum tensor count (ES_MAX_TENSORS = 2^20): views of 0 to
8 elements each, every one a tail tile of its own.  Perturb and update leave
the same bits as the same tensors planned in reverse order (the noise depends
only on each tensor's id and element index), sampled tensors match the
oracle, and the bytes between the views are untouched."""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_17310_amd import esopt, workloads as wl
from parity import assert_parity, perturb_delta, report, to_device, to_host, update_delta

pytestmark = pytest.mark.gpu

MAX_TENSORS = 1 << 20


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)


def test_plan_at_the_maximum_tensor_count():
    rng = np.random.default_rng(90)
    sizes = rng.integers(0, 9, MAX_TENSORS)
    starts = np.arange(MAX_TENSORS) * 10 + rng.integers(0, 2, MAX_TENSORS)   # some unaligned
    bits = wl.random_bf16_bits(MAX_TENSORS * 10 + 8, 91)
    ids = rng.permutation(1 << 24)[:MAX_TENSORS]
    r = torch.tensor([0.3, 0.8, 0.1, 0.6], device="cuda")
    outs, mid = [], None
    for order in (1, -1):
        buf = to_device(bits)
        views = [buf[s:s + n] for s, n in zip(starts, sizes)]
        with esopt.Plan(views[::order], tensor_ids=list(ids[::order])) as p:
            assert p.numel == int(sizes.sum())
            p.perturb(12, -1, 1e-3)
            if order == 1:
                torch.cuda.synchronize()
                mid = to_host(buf)
            p.update([1, 2, 2, 3], [1, 1, -1, 1], r, 5e-4)
        torch.cuda.synchronize()
        outs.append(to_host(buf))
        del views
    np.testing.assert_array_equal(outs[0], outs[1])
    gaps = np.ones(bits.size, bool)
    for s, n in zip(starts, sizes):
        gaps[s:s + n] = False
    np.testing.assert_array_equal(outs[0][gaps], bits[gaps])
    # sampled tensors, each pass against the oracle applied to the GPU's
    # state before it
    reps = {"perturb": ([], [], [], []), "update": ([], [], [], [])}
    rr = r.cpu().numpy()
    for k in rng.choice(MAX_TENSORS, 400, replace=False):
        s, n, t = int(starts[k]), int(sizes[k]), int(ids[k])
        if n == 0:
            continue
        el = np.arange(n, dtype=np.uint64)
        x0, x1, x2 = bits[s:s + n], mid[s:s + n], outs[0][s:s + n]
        for name, got, exp, base, d in (
                ("perturb", x1, oracle.perturb(x0, 12, t, -1, 1e-3, elems=el), x0,
                 perturb_delta(12, t, -1, 1e-3, el)),
                ("update", x2, oracle.update(x1, t, [1, 2, 2, 3], [1, 1, -1, 1], rr, 5e-4, 1e-3,
                                             elems=el)[0], x1,
                 update_delta(t, [1, 2, 2, 3], [1, 1, -1, 1], rr, 5e-4, 1e-3, 0, el))):
            for lst, v in zip(reps[name], (got, exp, base, d)):
                lst.append(v)
    for name, lists in reps.items():
        rep = report(*[np.concatenate(v) for v in lists])
        print("2^20 tensors, sampled:", name, rep)
        assert_parity(rep, name)


def test_quantized_plan_at_the_maximum_tensor_count():
    """The same for an int8 plan: 2^20 views of 0 to 40 codes sharing one
    scale, each a tail tile of its own (the table lookup per tile at its
    largest), order-independent codes, untouched gaps, sampled oracle parity
    of the perturbation."""
    from test_gpu_quant import _perturb_expect
    from parity import assert_qparity, qreport
    rng = np.random.default_rng(92)
    sizes = rng.integers(0, 41, MAX_TENSORS)
    starts = np.arange(MAX_TENSORS) * 48 + rng.integers(0, 3, MAX_TENSORS)
    codes = rng.integers(-127, 128, MAX_TENSORS * 48 + 8).astype(np.int8)
    ids = rng.permutation(1 << 24)[:MAX_TENSORS]
    scale = np.array([6e-4], np.float32)
    r = torch.tensor([0.3, 0.8, 0.1], device="cuda")
    outs, mid = [], None
    for order in (1, -1):
        buf = torch.from_numpy(codes).cuda()
        views = [buf[s:s + n] for s, n in zip(starts, sizes)]
        sdev = torch.from_numpy(scale).cuda()
        with esopt.QPlan(views[::order], [sdev] * MAX_TENSORS, [0] * MAX_TENSORS,
                         tensor_ids=list(ids[::order])) as p:
            assert p.numel == int(sizes.sum())
            p.perturb(13, 1, 1e-3)
            if order == 1:
                torch.cuda.synchronize()
                mid = buf.cpu().numpy()
            p.update([1, 2, 3], [1, -1, 1], r, 5e-4, round_seed=4)
        torch.cuda.synchronize()
        outs.append(buf.cpu().numpy())
        del views
    np.testing.assert_array_equal(outs[0], outs[1])
    gaps = np.ones(codes.size, bool)
    for s0, n in zip(starts, sizes):
        gaps[s0:s0 + n] = False
    np.testing.assert_array_equal(outs[0][gaps], codes[gaps])
    got, q_in, v, tol, ok = [], [], [], [], []
    for k in rng.choice(MAX_TENSORS, 400, replace=False):
        s0, n, t = int(starts[k]), int(sizes[k]), int(ids[k])
        if n == 0:
            continue
        d, o, tl = _perturb_expect(scale, 0, 13, t, 1, 1e-3, np.arange(n, dtype=np.uint64))
        for lst, x in zip((got, q_in, v, tol, ok), (mid[s0:s0 + n], codes[s0:s0 + n], d, tl, o)):
            lst.append(x)
    rep = qreport(*[np.concatenate(x) for x in (got, q_in, v, tol, ok)])
    print("2^20 int8 tensors, sampled perturb:", rep)
    assert_qparity(rep, "int8 perturb at 2^20 tensors")

