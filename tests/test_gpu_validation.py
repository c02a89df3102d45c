"""Memory the device cannot use is refused before any launch: host pointers,
sizes past the end of an allocation, for plans and for the per-call device
arrays; mapped pinned host memory is accepted.  Nothing here launches a
kernel on bad memory: every case is rejected by the host-side checks."""
import ctypes

import numpy as np
import pytest
import torch

from paper_2608_17310_amd import esopt

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)


def _plan(*tensors):
    lib = esopt.load()
    arr = (esopt.EsTensor * len(tensors))(*tensors)
    h = ctypes.c_void_p()
    rc = lib.es_plan_create(arr, len(tensors), ctypes.byref(h))
    if rc == esopt.ES_OK:
        lib.es_plan_destroy(h)
    return rc


def test_plan_refuses_host_memory_and_overstated_sizes():
    E = esopt.ES_ERR_INVALID_ARG
    host = np.zeros(4096, dtype=np.uint16)
    assert _plan(esopt.EsTensor(host.ctypes.data, host.size, 0, 0)) == E
    assert "device can access" in esopt.last_error() or "device memory" in esopt.last_error()
    t = torch.zeros(1000, dtype=torch.bfloat16, device="cuda")
    assert _plan(esopt.EsTensor(t.data_ptr(), 1000, 0, 0)) == esopt.ES_OK
    assert _plan(esopt.EsTensor(t.data_ptr(), 1 << 30, 0, 0)) == E       # 2 GiB past a small block
    assert "past the end" in esopt.last_error()
    # the binding's Plan surfaces the error
    with pytest.raises(esopt.EsError):
        lib = esopt.load()
        arr = (esopt.EsTensor * 1)(esopt.EsTensor(host.ctypes.data, host.size, 0, 0))
        esopt._check(lib.es_plan_create(arr, 1, ctypes.byref(ctypes.c_void_p())), "es_plan_create")


def test_qplan_refuses_short_scales_and_host_scales():
    lib = esopt.load()
    E = esopt.ES_ERR_INVALID_ARG
    q = torch.zeros(1 << 24, dtype=torch.int8, device="cuda")
    sc = torch.ones(4, device="cuda")              # lives in a small (2 MiB) block
    h = ctypes.c_void_p()
    # rows of 8 codes need 2^21 scales (8 MiB): past the end of the block
    t = esopt.EsQTensor(q.data_ptr(), sc.data_ptr(), q.numel(), 8, 0)
    assert lib.es_qplan_create((esopt.EsQTensor * 1)(t), 1, ctypes.byref(h)) == E
    assert "scales" in esopt.last_error()
    t = esopt.EsQTensor(q.data_ptr(), sc.data_ptr(), q.numel(), 0, 0)    # one scale: fine
    assert lib.es_qplan_create((esopt.EsQTensor * 1)(t), 1, ctypes.byref(h)) == esopt.ES_OK
    lib.es_qplan_destroy(h)
    host = np.ones(4, np.float32)
    t = esopt.EsQTensor(q.data_ptr(), host.ctypes.data, q.numel(), 0, 0)
    assert lib.es_qplan_create((esopt.EsQTensor * 1)(t), 1, ctypes.byref(h)) == E


def test_update_arrays_are_checked_and_pinned_rewards_work():
    lib = esopt.load()
    w = torch.randn(1 << 16, device="cuda").to(torch.bfloat16)
    w2 = w.clone()
    w0 = w.clone()
    plan = esopt.Plan([w])
    plan2 = esopt.Plan([w2])
    seeds = (ctypes.c_uint64 * 3)(1, 2, 3)
    signs = (ctypes.c_int32 * 3)(1, 1, 1)
    opts = esopt.EsUpdateOpts(5e-4, 1e-3, 1e-8, 0, 0)
    host_r = np.array([0.1, 0.5, 0.9], np.float32)
    s = esopt._stream(None)
    E = esopt.ES_ERR_INVALID_ARG
    assert lib.es_update(plan.handle, seeds, signs, ctypes.c_void_p(host_r.ctypes.data), 3,
                         ctypes.byref(opts), None, None, s) == E
    r_dev = torch.from_numpy(host_r).cuda()
    host_z = np.zeros(3, np.float32)
    assert lib.es_update(plan.handle, seeds, signs, ctypes.c_void_p(r_dev.data_ptr()), 3,
                         ctypes.byref(opts), ctypes.c_void_p(host_z.ctypes.data), None, s) == E
    assert lib.es_zscore(ctypes.c_void_p(host_r.ctypes.data), 3, 1e-8,
                         ctypes.c_void_p(r_dev.data_ptr()), None, s) == E
    # nothing ran: the parameters are untouched
    torch.cuda.synchronize()
    assert torch.equal(w, w2)
    # rewards in pinned host memory are mapped for the device and accepted
    r_pin = torch.from_numpy(host_r).pin_memory()
    plan.update([1, 2, 3], [1, 1, 1], r_pin, 5e-4)
    plan2.update([1, 2, 3], [1, 1, 1], r_dev, 5e-4)
    torch.cuda.synchronize()
    assert torch.equal(w.view(torch.int16), w2.view(torch.int16))
    assert not torch.equal(w.view(torch.int16), w0.view(torch.int16))
    plan.close()
    plan2.close()
