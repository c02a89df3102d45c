"""A generation driven from C (tests/harness/c_generation.c) through the
public header and the HIP runtime alone: the perturbed tensors match the
oracle element by element, the radius and z-scores match the oracle's, the
final tensors are bit for bit those of the same calls made through the
Python binding, and the plan checksum the C program read back equals the
oracle's checksum of those tensors.  The same over binary32 masters
(es_plan_set_master, es_perturb_master, ES_UPDATE_MASTER): the members
applied from the masters against the oracle, the masters against the
oracle's update within the bar of the kernel's arithmetic, and masters and
bf16 values bit for bit those of the binding."""
import os
import shutil
import subprocess

import numpy as np
import pytest
import torch

import oracle
from paper_2608_17310_amd import esopt, workloads as wl
from parity import (assert_master_parity, assert_parity, master_report, master_tolerance,
                    perturb_delta, report, to_host)

pytestmark = pytest.mark.gpu

HERE = os.path.dirname(os.path.abspath(__file__))
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
N0, N1 = 300_007, 65_536 * 2 + 5          # several tiles each, ragged ends
SEEDS, REWARDS = [100, 101, 102, 103], [0.3, 0.9, 0.1, 0.6]


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)


def _build(tmp_path):
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("gcc not available")
    exe = str(tmp_path / "c_generation")
    libdir = os.path.dirname(esopt.LIB_PATH)
    subprocess.run([gcc, "-std=c99", "-Wall", "-Werror", "-D__HIP_PLATFORM_AMD__",
                    "-I", os.path.join(ROCM, "include"), "-I", os.path.join(HERE, "..", "include"),
                    os.path.join(HERE, "harness", "c_generation.c"),
                    "-L", libdir, "-l:" + os.path.basename(esopt.LIB_PATH),
                    "-L", os.path.join(ROCM, "lib"), "-lamdhip64",
                    "-Wl,-rpath," + libdir, "-Wl,-rpath," + os.path.join(ROCM, "lib"),
                    "-o", exe], check=True)
    return exe


def test_generation_from_c_matches_binding_and_oracle(tmp_path):
    exe = _build(tmp_path)
    x0 = wl.random_bf16_bits(N0 + N1, 300)
    x0.tofile(tmp_path / "in.bin")
    print("running", exe, N0, N1, flush=True)
    res = subprocess.run([exe, str(tmp_path / "in.bin"), str(tmp_path / "pert.bin"),
                          str(tmp_path / "final.bin"), str(N0), str(N1)],
                         capture_output=True, text=True, timeout=120)
    assert res.returncode == 0, res.stderr
    out = {l.split()[0]: l.split()[1:] for l in res.stdout.splitlines()}
    sigma = float(np.float32(out["sigma"][0]))        # 9 digits: the binary32 value
    assert sigma == float(np.float32(oracle.sigma_cosine(1e-3, 1e-4, 3, 100)))
    assert int(out["status"][0]) == 0
    z = np.array([float(v) for v in out["z"]])
    z_exp, st = oracle.zscore(REWARDS)
    assert st == 0
    np.testing.assert_allclose(z, z_exp, rtol=1e-6, atol=1e-6)

    # the first member applied, against the oracle
    pert = np.fromfile(tmp_path / "pert.bin", dtype=np.uint16)
    parts = [(slice(0, N0), 0), (slice(N0, N0 + N1), 5)]
    for sl, tid in parts:
        el = np.arange(sl.stop - sl.start, dtype=np.uint64)
        rep = report(pert[sl], oracle.perturb(x0[sl], SEEDS[0], tid, 1, sigma), x0[sl],
                     perturb_delta(SEEDS[0], tid, 1, sigma, el))
        print("C driver perturb, tensor", tid, rep)
        assert_parity(rep, f"C driver perturb {tid}")

    # the same calls through the binding
    final = np.fromfile(tmp_path / "final.bin", dtype=np.uint16)
    buf = torch.zeros(N0 + N1 + 1, dtype=torch.int16, device="cuda")
    buf.copy_(torch.from_numpy(np.concatenate([x0[:N0], np.zeros(1, np.uint16), x0[N0:]]).view(np.int16)).cuda())
    views = [buf[:N0].view(torch.bfloat16), buf[N0 + 1:].view(torch.bfloat16)]
    with esopt.Plan(views, tensor_ids=[0, 5]) as p:
        p.perturb(SEEDS[0], 1, sigma)
        for a, b in zip(SEEDS, SEEDS[1:]):
            p.swap(a, 1, b, 1, sigma)
        p.restore_update(SEEDS[-1], 1, sigma, SEEDS, [1] * 4,
                         torch.tensor(REWARDS, dtype=torch.float32, device="cuda"), 5e-4)
        assert p.checksum() == int(out["checksum"][0])
    torch.cuda.synchronize()
    np.testing.assert_array_equal(np.concatenate([to_host(v) for v in views]), final)
    assert int(out["checksum"][0]) == oracle.plan_checksum(
        [(final[sl], tid, 0) for sl, tid in parts])
    assert np.mean(final != x0) > 0.5


def test_generation_over_masters_from_c(tmp_path):
    exe = _build(tmp_path)
    x0 = wl.random_bf16_bits(N0 + N1, 301)
    x0.tofile(tmp_path / "in.bin")
    print("running", exe, N0, N1, "with masters", flush=True)
    res = subprocess.run([exe, str(tmp_path / "in.bin"), str(tmp_path / "pert.bin"),
                          str(tmp_path / "final.bin"), str(N0), str(N1),
                          str(tmp_path / "masters.bin")],
                         capture_output=True, text=True, timeout=120)
    assert res.returncode == 0, res.stderr
    out = {l.split()[0]: l.split()[1:] for l in res.stdout.splitlines()}
    sigma = float(np.float32(out["sigma"][0]))
    assert int(out["status"][0]) == 0
    m0 = (x0.astype(np.uint32) << 16).view(np.float32)       # the masters' start

    pert = np.fromfile(tmp_path / "pert.bin", dtype=np.uint16)
    parts = [(slice(0, N0), 0), (slice(N0, N0 + N1), 5)]
    for sl, tid in parts:
        el = np.arange(sl.stop - sl.start, dtype=np.uint64)
        rep = report(pert[sl], oracle.perturb_master(m0[sl], SEEDS[0], tid, 1, sigma), x0[sl],
                     perturb_delta(SEEDS[0], tid, 1, sigma, el))
        print("C driver perturb_master, tensor", tid, rep)
        assert_parity(rep, f"C driver perturb_master {tid}")

    masters = np.fromfile(tmp_path / "masters.bin", dtype=np.float32)
    z, _ = oracle.zscore(REWARDS)
    c = oracle.update_coefficient(5e-4, sigma, len(SEEDS), 0)
    d, w = oracle.member_weights(SEEDS, [1] * 4, z, c)
    live = [(sd, wd) for sd, wd in zip(d, w) if wd != 0.0]
    for sl, tid in parts:
        exp, _, st = oracle.update_master(m0[sl], tid, SEEDS, [1] * 4,
                                          np.array(REWARDS, np.float32), 5e-4, sigma)
        assert st == 0
        el = np.arange(sl.stop - sl.start, dtype=np.uint64)
        rep = master_report(masters[sl], exp, master_tolerance(exp, live, tid, el))
        print("C driver masters, tensor", tid, rep)
        assert_master_parity(rep, f"C driver masters {tid}")

    # the same calls through the binding
    final = np.fromfile(tmp_path / "final.bin", dtype=np.uint16)
    buf = torch.zeros(N0 + N1 + 1, dtype=torch.int16, device="cuda")
    buf.copy_(torch.from_numpy(np.concatenate([x0[:N0], np.zeros(1, np.uint16), x0[N0:]]).view(np.int16)).cuda())
    views = [buf[:N0].view(torch.bfloat16), buf[N0 + 1:].view(torch.bfloat16)]
    mdev = [torch.from_numpy(m0[sl].copy()).cuda() for sl, _ in parts]
    with esopt.Plan(views, tensor_ids=[0, 5]) as p:
        p.set_master(mdev)
        for sd in SEEDS:
            p.perturb_master(sd, 1, sigma)
        p.update(SEEDS, [1] * 4, torch.tensor(REWARDS, dtype=torch.float32, device="cuda"),
                 5e-4, flags=esopt.ES_UPDATE_MASTER)
        assert p.checksum() == int(out["checksum"][0])
    torch.cuda.synchronize()
    np.testing.assert_array_equal(np.concatenate([to_host(v) for v in views]), final)
    np.testing.assert_array_equal(np.concatenate([m.cpu().numpy() for m in mdev]).view(np.uint32),
                                  masters.view(np.uint32))
    assert np.mean(masters != m0) > 0.99
