"""es_hbm_calibrate: the read pass folds every word into the sink (their
XOR), the write pass leaves the documented pattern, the in-place pass leaves
the buffer bit for bit unchanged -- with nontemporal and with ordinary
accesses -- and invalid buffers and modes are refused."""
import numpy as np
import pytest
import torch

from paper_2608_17310_amd import esopt

pytestmark = pytest.mark.gpu

TILE = 1 << 17                # bytes per tile: 1024 lanes x 8 words x 16 bytes


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)


def _buf(n_tiles, seed):
    rng = np.random.default_rng(seed)
    host = rng.integers(-2**31, 2**31, size=n_tiles * TILE // 4, dtype=np.int64).astype(np.int32)
    return host, torch.from_numpy(host).cuda()


POLICIES = [0, esopt.CALIBRATE_TEMPORAL]


@pytest.mark.parametrize("policy", POLICIES)
@pytest.mark.parametrize("n_tiles", [1, 300, 1000])      # fewer and more tiles than CUs
def test_read_folds_every_word_into_the_sink(n_tiles, policy):
    host, buf = _buf(n_tiles, n_tiles)
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    esopt.hbm_calibrate(buf, esopt.CALIBRATE_READ | policy, sink)
    torch.cuda.synchronize()
    exp = np.bitwise_xor.reduce(host.view(np.uint32))
    assert np.uint32(sink.cpu().numpy().view(np.uint32)[0]) == exp
    assert torch.equal(buf.cpu(), torch.from_numpy(host))


@pytest.mark.parametrize("policy", POLICIES)
@pytest.mark.parametrize("n_tiles", [1, 300])
def test_write_leaves_the_pattern_and_in_place_changes_nothing(n_tiles, policy):
    host, buf = _buf(n_tiles, 7 + n_tiles)
    esopt.hbm_calibrate(buf, esopt.CALIBRATE_READ_WRITE | policy)
    torch.cuda.synchronize()
    assert torch.equal(buf.cpu(), torch.from_numpy(host))
    esopt.hbm_calibrate(buf, esopt.CALIBRATE_WRITE | policy)
    torch.cuda.synchronize()
    got = buf.cpu().numpy().view(np.uint32).reshape(n_tiles, 8, 1024, 4)
    t, u, l = np.meshgrid(np.arange(n_tiles), np.arange(8), np.arange(1024), indexing="ij")
    exp = np.stack([t, u, l, np.zeros_like(t)], axis=-1).astype(np.uint32)
    np.testing.assert_array_equal(got, exp)


def test_invalid_buffers_are_refused():
    buf = torch.zeros(TILE // 4 + 4, dtype=torch.int32, device="cuda")
    with pytest.raises(esopt.EsError):
        esopt.hbm_calibrate(buf, esopt.CALIBRATE_WRITE)          # not whole tiles
    with pytest.raises(esopt.EsError):
        esopt.hbm_calibrate(buf[4:4 + TILE // 4], esopt.CALIBRATE_WRITE - 1)   # read: no sink
    for bad in (-1, 3, 7, 8):
        with pytest.raises(esopt.EsError):
            esopt.hbm_calibrate(buf[4:4 + TILE // 4], bad)
