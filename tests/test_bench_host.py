"""Host-side logic of bench.py that needs no GPU: the count of seeds whose
noise the update generates, and the refusal of more than one GPU."""
import json
import os
import subprocess
import sys

import numpy as np

import bench

REPO = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_live_seeds_counts_nonzero_merged_weights():
    seeds, signs = [1, 1, 2, 2, 3, 3], [1, -1, 1, -1, 1, -1]
    # antithetic pairs: a pair with equal rewards merges to zero weight
    assert bench.live_seeds(seeds, signs, np.float32([1, 0, 1, 1, 0, 1])) == 2
    assert bench.live_seeds(seeds, signs, np.float32([1, 1, 0, 0, 1, 1])) == 0
    # every reward equal: z-scores to zero, nothing is generated
    assert bench.live_seeds([1, 2, 3], [1, 1, 1], np.float32([0.5, 0.5, 0.5])) == 0
    # distinct single members: only one at exactly the mean drops out
    assert bench.live_seeds([4, 5, 6], [1, 1, 1], np.float32([0.0, 1.0, 2.0])) == 2
    assert bench.live_seeds([4, 5, 6], [1, 1, 1], np.float32([0.1, 0.7, 0.3])) == 3
    # a repeated seed with the same sign adds its weights
    assert bench.live_seeds([7, 7, 8], [1, 1, 1], np.float32([0.0, 1.0, 2.0])) == 2


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(REPO, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    msg = json.loads(r.stdout.strip().splitlines()[-1])
    assert "one GPU" in msg["error"]


def test_host_cpu_is_reported():
    h = bench.host_cpu()
    assert h["host_logical_cpus"] == os.cpu_count()
    assert h["cpu_model"] is None or isinstance(h["cpu_model"], str)
