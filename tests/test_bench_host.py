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


def test_sigma_follows_the_library_schedule_and_holds_after_it():
    import oracle
    from paper_2608_17310_amd import workloads as wl
    W = wl.DENSE_4B                                   # 1e-3 -> 1e-4 over T = 100
    assert bench.sigma_at(oracle.sigma_cosine, W, 0) == W.sigma0
    assert abs(bench.sigma_at(oracle.sigma_cosine, W, 50) - 5.5e-4) < 1e-15
    assert bench.sigma_at(oracle.sigma_cosine, W, W.T) == W.sigma_T
    assert bench.sigma_at(oracle.sigma_cosine, W, W.T + 7) == W.sigma_T
    W1 = wl.DENSE_27B                                 # constant sigma
    assert bench.sigma_at(oracle.sigma_cosine, W1, 13) == W1.sigma0


def test_cpu_workers_use_the_affinity_mask_up_to_the_cap():
    workers, avail = bench.cpu_workers()
    assert avail == len(os.sched_getaffinity(0))
    assert workers == min(avail, bench.CPU_WORKER_CAP)
    h = bench.host_cpu()
    assert h["cpus_available"] == avail and h["worker_cap"] == bench.CPU_WORKER_CAP


def _fake_profile(tmp, labels, extra, seq):
    """CSV files in the layout rocprofv3 writes for one trace run and three
    counter runs: `seq` is the dispatch sequence as (kernel name, ns,
    {counter: value}); the library's dispatches must follow the labels."""
    import csv
    for run in ("trace", "fetch", "write", "valu"):
        d = tmp / run / "host" / "1"
        d.mkdir(parents=True)
        with open(tmp / run / "labels.json", "w") as fh:
            json.dump({"launches": labels, **extra}, fh)
        if run == "trace":
            with open(d / "trace_kernel_trace.csv", "w", newline="") as fh:
                w = csv.writer(fh)
                w.writerow(["Dispatch_Id", "Kernel_Name", "Start_Timestamp", "End_Timestamp"])
                t = 1000
                for i, (name, ns, _) in enumerate(seq):
                    w.writerow([i + 1, name, t, t + ns])
                    t += ns + 10
            continue
        want = {"fetch": ["FETCH_SIZE"], "write": ["WRITE_SIZE"],
                "valu": list(bench.VALU_COUNTERS)}[run]
        with open(d / f"{run}_counter_collection.csv", "w", newline="") as fh:
            w = csv.writer(fh)
            w.writerow(["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value",
                        "Start_Timestamp", "End_Timestamp"])
            t = 1000
            for i, (name, ns, ctr) in enumerate(seq):
                for c in want:
                    w.writerow([i + 1, name, c, ctr.get(c, 0.0), t, t + ns])
                t += ns + 10


def test_summarize_joins_labels_with_dispatches(tmp_path):
    P = 1 << 20
    copy_kib = (1 << 30) / 1024
    lib = "void (anonymous namespace)::es_perturb_kernel<1024, 8, 1>((anonymous namespace)::DevTile const*)"
    upd = "void (anonymous namespace)::es_update_kernel<1024, 8, true, false>(int)"
    other = "void at::native::normal_kernel(float*)"
    copy = "__amd_rocclr_copyBuffer"
    # the perturb moves 2 B/param each way; the FETCH counter reads half of
    # what is fetched (the copy of 2^30 B fetches 2^29 counted bytes)
    pc = {"FETCH_SIZE": 2 * P / 2 / 1024, "WRITE_SIZE": 2 * P / 1024, "SQ_INSTS_VALU": 16 * P / 64,
          "GRBM_GUI_ACTIVE": 8 * 2.0 * 1000, "SQ_INSTS_VALU_TRANS_F32": P / 64}
    uc = {"FETCH_SIZE": 2 * P / 2 / 1024, "WRITE_SIZE": 2 * P / 1024,
          "SQ_INSTS_VALU": 4 * 14 * P / 64, "GRBM_GUI_ACTIVE": 8 * 2.4 * 5000}
    seq = [(other, 50, {}), (lib, 1000, pc), (other, 40, {}), (lib, 1000, pc), (upd, 5000, uc),
           (copy, 700, {"FETCH_SIZE": copy_kib / 2, "WRITE_SIZE": copy_kib})]
    labels = [
        {"label": "es_perturb", "group": "perturb", "params": P, "algorithmic_bytes": 4 * P,
         "normals": P, "members": None},
        {"label": "es_restore", "group": "perturb", "params": P, "algorithmic_bytes": 4 * P,
         "normals": P, "members": None},
        {"label": "es_update (N=4, nearest-even)", "group": "update", "params": P,
         "algorithmic_bytes": 4 * P, "normals": 4 * P, "members": None}]
    extra = {"workload": "tiny-1m", "params": P, "members": 4, "distinct_seeds": 4,
             "source_hash": bench._kernel_source_hash(), "pass_args": "--profile-pass"}
    _fake_profile(tmp_path / "prof", labels, extra, seq)
    out = tmp_path / "profiles"
    out.mkdir()
    bench.summarize(str(tmp_path / "prof"), profiles_dir=str(out))
    c = json.load(open(out / "counters.json"))
    assert abs(c["es_perturb"]["bytes_per_launch"] / (4 * P) - 1) < 1e-12
    assert abs(c["es_update"]["valu_insts_per_launch"] * 64 / P - 56) < 1e-9
    text = open(out / "es_perturb_tiny-1m.md").read()
    # 16 VALU instructions per parameter, one normal per parameter, 2.0 GHz
    assert "| es_perturb | `es_perturb_kernel<1024, 8, 1>` | 1 | 1000 |" in text
    assert "| 16.00 | 16.00 | 1.00 |" in text and "| 2.000 |" in text
    assert "es_update_tiny-1m.md" in os.listdir(out)
    # a label without its dispatch is an error, not a silent shift
    bad = tmp_path / "bad"
    _fake_profile(bad, labels, extra, seq[:4] + seq[5:])
    import pytest
    with pytest.raises(RuntimeError):
        bench.summarize(str(bad), profiles_dir=str(out))
