"""es_qswap: the revert of one member and the apply of the next in one pass
over int8 or E4M3 codes (Section 3; Appendix D.6 order), bit for bit the
codes of es_qrestore followed by es_qperturb: on tensors with invalid scales
and codes of -128, on fp8 codes of every byte value (not-a-number codes, -0,
+-448, subnormals), on shards and blocks, for an antithetic partner, with a
zero sigma on either side, and through the generation driver, whose log
replays with separate passes."""
import numpy as np
import pytest
import torch

from paper_2608_17310_amd import esopt
from paper_2608_17310_amd.generation import replay, run_generation
from test_gpu_fp8 import _codes as _f8codes
from test_gpu_quant import _device_views, _tensor_set

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)


def _host(t):
    return t.cpu().numpy().copy()


def _plans(fmt):
    """Two identical quantized plans (codes, scales, rows, ids of the int8
    test set, with fp8 codes of every byte value for "e4m3")."""
    codes, scales, rows, ids = _tensor_set()
    if fmt == "e4m3":
        codes = [_f8codes(c.size, 90 + i).view(np.int8) for i, c in enumerate(codes)]
    out = []
    for _ in range(2):
        _, views = _device_views(codes)
        if fmt == "e4m3":
            views = [v.view(torch.uint8) for v in views]
        sdev = [torch.from_numpy(s).cuda() for s in scales]
        out.append((esopt.QPlan(views, sdev, rows, tensor_ids=ids, format=fmt), views))
    return out


MOVES = [
    # (from seed, sign, sigma), (to seed, sign, sigma)
    ((5, 1, 1e-3), (6, 1, 1e-3)),
    ((7, 1, 1.5e-3), (7, -1, 1.5e-3)),            # antithetic partner: one key
    ((8, -1, 2e-3), (9, 1, 5e-4)),                # different radii
    ((10, 1, 0.0), (11, -1, 1e-3)),               # zero sigma: the perturb alone
    ((12, 1, 1e-3), (13, 1, 0.0)),                # zero sigma: the restore alone
    (((1 << 63) + 1, -1, 1e-3), (2, 1, 1e-3)),
]


@pytest.mark.parametrize("fmt", ["int8", "e4m3"])
def test_fused_equals_restore_then_perturb(fmt):
    (pa, va), (pb, vb) = _plans(fmt)
    for (sf, gf, xf), (st, gt, xt) in MOVES:
        pa.perturb(sf, gf, max(xf, 1e-3))          # a member applied first
        pb.perturb(sf, gf, max(xf, 1e-3))
        pa.swap(sf, gf, st, gt, xf, sigma_to=xt)
        pb.restore(sf, gf, xf)
        pb.perturb(st, gt, xt)
        torch.cuda.synchronize()
        for a, b in zip(va, vb):
            np.testing.assert_array_equal(_host(a), _host(b), err_msg=f"{fmt} {sf}->{st}")
    pa.swap(1, 1, 2, 1, 0.0)                      # both zero: nothing runs
    torch.cuda.synchronize()
    for a, b in zip(va, vb):
        np.testing.assert_array_equal(_host(a), _host(b))
    assert pa.checksum() == pb.checksum()
    with pytest.raises(esopt.EsError):
        pa.swap(1, 0, 2, 1, 1e-3)
    with pytest.raises(esopt.EsError):
        pa.swap(1, 1, 2, 1, 1e-3, sigma_to=float("nan"))
    pa.close()
    pb.close()


@pytest.mark.parametrize("fmt", ["int8", "e4m3"])
def test_fused_on_shards_and_blocks(fmt):
    rng = np.random.default_rng(91)
    rows, cols = 64, 1024
    codes = (rng.integers(-127, 128, rows * cols).astype(np.int8) if fmt == "int8"
             else _f8codes(rows * cols, 92).view(np.int8))
    scales = rng.uniform(2e-4, 1e-3, rows).astype(np.float32)
    dt = torch.int8 if fmt == "int8" else torch.uint8

    def plans():
        src = torch.from_numpy(codes.reshape(rows, cols)).cuda().view(dt)
        blk = src[:, 256:768].contiguous()
        shard = src[32:].reshape(-1).clone()
        s = torch.from_numpy(scales).cuda()
        return (esopt.QPlan(blocks=[esopt.QBlock(blk, s, 512, 3, cols, 0, 256)], format=fmt),
                esopt.QPlan([shard], [s[32:].contiguous()], [cols], tensor_ids=[4], format=fmt,
                            offsets=[32 * cols]), [blk, shard])
    a1, a2, va = plans()
    b1, b2, vb = plans()
    for p in (a1, a2, b1, b2):
        p.perturb(21, 1, 1e-3)
    for p in (a1, a2):
        p.swap(21, 1, 22, -1, 1e-3)
    for p in (b1, b2):
        p.restore(21, 1, 1e-3)
        p.perturb(22, -1, 1e-3)
    torch.cuda.synchronize()
    for a, b in zip(va, vb):
        np.testing.assert_array_equal(_host(a), _host(b))
    for p in (a1, a2, b1, b2):
        p.close()


@pytest.mark.parametrize("fmt", ["int8", "e4m3"])
def test_generation_driver_fuses_quantized_swaps(fmt):
    (pa, va), (pb, vb) = _plans(fmt)
    seeds, signs = [4, 4, 5, 6], [1, -1, 1, 1]
    scores = [0.3, 0.9, 0.1, 0.5]
    rec = run_generation(pa, seeds, signs, 1e-3, 5e-4, lambda i: scores[i], round_seed=3)
    assert rec.fused_swap
    for sd, sg in zip(seeds, signs):
        pb.perturb(sd, sg, 1e-3)
        pb.restore(sd, sg, 1e-3)
    pb.update(seeds, signs, torch.tensor(scores, dtype=torch.float32, device="cuda"), 5e-4,
              sigma=1e-3, round_seed=3)
    torch.cuda.synchronize()
    for a, b in zip(va, vb):
        np.testing.assert_array_equal(_host(a), _host(b))
    (pc, vc), _ = _plans(fmt)
    rec.fused_swap = False
    replay(pc, [rec])                               # separate passes, same codes
    torch.cuda.synchronize()
    for a, c in zip(va, vc):
        np.testing.assert_array_equal(_host(a), _host(c))
    for p in (pa, pb, pc):
        p.close()
