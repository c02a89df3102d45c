"""The library's host code under AddressSanitizer and UndefinedBehaviorSanitizer
(no GPU): tests/harness/host_sanitize.hip compiles the library source into one
program with both sanitizers on the host pass only, then checks the update's
population tables, the tiling of tensors, the int8 row divisor and every
argument check that fails before a device is touched, each against a plain
reference.  Any out-of-bounds access, use after free, overflow or other
undefined behaviour on those paths stops the program with a report."""
import os
import shutil
import subprocess

import pytest

REPO = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HARNESS = os.path.join(REPO, "tests", "harness", "host_sanitize.hip")


def _hipcc():
    for cand in (shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    pytest.skip("hipcc not available")


def test_host_code_under_address_and_undefined_behaviour_sanitizers(tmp_path):
    exe = str(tmp_path / "host_sanitize")
    cmd = [_hipcc(), "--offload-arch=gfx950", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
           "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=undefined",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", HARNESS, "-o", exe]
    res = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
    assert res.returncode == 0, res.stderr[-4000:]
    # the sanitizers' runtimes are in the program
    blob = open(exe, "rb").read()
    assert b"__asan_init" in blob and b"__ubsan_handle" in blob
    env = dict(os.environ,
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    run = subprocess.run([exe], capture_output=True, text=True, timeout=300, env=env)
    assert run.returncode == 0 and run.stdout.strip().endswith("ok"), (
        run.stdout[-4000:] + run.stderr[-4000:])
