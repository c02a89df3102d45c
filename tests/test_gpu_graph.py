"""The passes can be captured into a HIP graph and replayed: each call only
launches kernels on the given stream (no host synchronisation, no memset
nodes, member tables passed as kernel arguments).  The graph is replayed
several times with eager work and synchronisation between replays, and every
replay is checked against the same calls made eagerly on a twin."""
import numpy as np
import pytest
import torch

from paper_2608_17310_amd import esopt, workloads as wl
from parity import to_device, to_host

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)


def _calls(plan, rewards, z):
    plan.perturb(5, 1, 1e-3)
    plan.swap(5, 1, 6, -1, 1e-3)
    plan.restore(6, -1, 1e-3)
    plan.update([1, 2, 2, 3], [1, 1, -1, 1], rewards, 5e-4, z_out=z)
    plan.update([1, 2, 2, 3], [1, 1, -1, 1], rewards, 5e-4,
                flags=esopt.ES_UPDATE_STOCHASTIC_ROUND, round_seed=17)


def test_captured_generation_replays_like_eager_calls():
    bits = [wl.random_bf16_bits(n, 300 + i) for i, n in enumerate([1 << 18, 4097, 77])]
    live = [to_device(b) for b in bits]
    twin = [to_device(b) for b in bits]
    rewards = torch.tensor([0.3, 0.9, 0.1, 0.6], device="cuda")
    z_live = torch.zeros(4, device="cuda")
    z_twin = torch.zeros(4, device="cuda")
    plan = esopt.Plan(live)
    plan_twin = esopt.Plan(twin)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        _calls(plan, rewards, z_live)
    torch.cuda.synchronize()
    # capture ran nothing: the parameters are unchanged
    for b, t in zip(bits, live):
        np.testing.assert_array_equal(to_host(t), b)
    for rep in range(3):
        g.replay()
        torch.cuda.synchronize()
        _calls(plan_twin, rewards, z_twin)          # eager work between replays
        torch.cuda.synchronize()
        for a, b in zip(live, twin):
            np.testing.assert_array_equal(to_host(a), to_host(b))
        assert torch.equal(z_live, z_twin)
    assert not np.array_equal(to_host(live[0]), bits[0])
    plan.close()
    plan_twin.close()


def test_captured_int8_passes_replay_like_eager_calls():
    host = wl.host_qparams(wl.TINY)
    live = [torch.from_numpy(q).cuda() for q, _, _ in host]
    twin = [torch.from_numpy(q).cuda() for q, _, _ in host]
    scales = [torch.from_numpy(s).cuda() for _, s, _ in host]
    rows = [r for _, _, r in host]
    rewards = torch.tensor([0.3, 0.9, 0.1], device="cuda")
    plan = esopt.QPlan(live, scales, rows)
    plan_twin = esopt.QPlan(twin, scales, rows)

    def calls(p):
        p.perturb(4, 1, 1e-3)
        p.restore(4, 1, 1e-3)
        p.update([1, 2, 3], [1, 1, 1], rewards, 5e-3, round_seed=2)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        calls(plan)
    torch.cuda.synchronize()
    for rep in range(3):
        g.replay()
        torch.cuda.synchronize()
        calls(plan_twin)
        torch.cuda.synchronize()
        for a, b in zip(live, twin):
            assert torch.equal(a, b)
    plan.close()
    plan_twin.close()


def test_captured_block_passes_replay_like_eager_calls():
    """A plan holding a strided column block and a whole vector runs every
    pass as two launches (plain tiles, then the tiles with row maps); both
    are captured, and the checksum's two accumulating launches too."""
    a_bits = wl.random_bf16_bits(96 * 1024, 310)
    v_bits = wl.random_bf16_bits(5000, 311)

    def make():
        a = to_device(a_bits, (96, 1024))[:, 256:512].contiguous()
        v = to_device(v_bits)
        return [a, v], esopt.Plan(blocks=[esopt.Block(a, 1, 1024, 0, 256),
                                          esopt.Block(v, 2, 5000)])
    live, plan = make()
    twin, plan_twin = make()
    rewards = torch.tensor([0.3, 0.9, 0.1, 0.6], device="cuda")
    z_live = torch.zeros(4, device="cuda")
    z_twin = torch.zeros(4, device="cuda")
    c_live = torch.zeros(1, dtype=torch.int64, device="cuda")
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        _calls(plan, rewards, z_live)
        plan.checksum(out=c_live, stream=s)
    torch.cuda.synchronize()
    for rep in range(3):
        g.replay()
        torch.cuda.synchronize()
        _calls(plan_twin, rewards, z_twin)
        c_twin = plan_twin.checksum()
        torch.cuda.synchronize()
        for a, b in zip(live, twin):
            np.testing.assert_array_equal(to_host(a), to_host(b))
        assert torch.equal(z_live, z_twin)
        assert int(c_live.item()) & ((1 << 64) - 1) == c_twin
    plan.close()
    plan_twin.close()
