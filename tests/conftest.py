"""Shared pytest configuration.

Markers:
  gpu -- needs an MI355X (gfx950) and the built HIP library; the CPU suite runs
         with -m "not gpu".
"""
import os
import shutil
import subprocess
import sys

import pytest

REPO = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if REPO not in sys.path:
    sys.path.insert(0, REPO)

HARNESS_DIR = os.path.join(REPO, "tests", "harness")
TORCH_INCLUDE = None


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X GPU and the built HIP library")


def _torch_include():
    import torch.utils.cpp_extension as ce
    return ce.include_paths()[0]


@pytest.fixture(scope="session")
def kat_harness(tmp_path_factory):
    """Compile the two independent Philox harnesses (PyTorch's and rocRAND's
    host engines) and return {name: callable(list of (seed, subsequence,
    quad)) -> list of 4-tuples of output words}."""
    out = tmp_path_factory.mktemp("kat")
    exes = {}
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ not available")
    torch_exe = str(out / "philox_torch_kat")
    subprocess.run([gxx, "-O1", "-std=c++17", "-I", _torch_include(),
                    os.path.join(HARNESS_DIR, "philox_torch_kat.cpp"), "-o", torch_exe],
                   check=True)
    exes["torch"] = torch_exe
    clang = "/opt/rocm/llvm/bin/clang++"
    if os.path.exists(clang) and os.path.exists("/opt/rocm/include/rocrand/rocrand_philox4x32_10.h"):
        rr_exe = str(out / "philox_rocrand_kat")
        subprocess.run([clang, "-x", "hip", "--cuda-host-only", "-O1", "-std=c++17",
                        "-I", "/opt/rocm/include",
                        os.path.join(HARNESS_DIR, "philox_rocrand_kat.cpp"), "-o", rr_exe],
                       check=True)
        exes["rocrand"] = rr_exe

    def make(exe):
        def run(rows):
            text = "".join("%d %d %d\n" % tuple(int(v) for v in r) for r in rows)
            res = subprocess.run([exe], input=text, capture_output=True, text=True, check=True)
            return [tuple(int(x) for x in line.split()) for line in res.stdout.splitlines()]
        return run

    return {k: make(v) for k, v in exes.items()}
