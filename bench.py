"""Benchmark of the ES parameter path on one MI355X.

One step is one ES generation's parameter-space work (arXiv 2608.17310,
Section 3; Appendix D.6): for each of the N members, es_perturb (theta +=
s sigma_t eps_i) and es_restore (theta -= s sigma_t eps_i) over the whole
parameter set, then one fused es_update (z-score of the N rewards, merged
member weights, theta += sum_d w_d eps_d) over the whole set.  Model
evaluation between perturb and restore is outside this path and not run.

Inputs are synthetic and resident in HBM before timing: a transformer-shaped
bf16 parameter set with N(0, 0.02) values and a precomputed reward vector per
step.  Throughput `value` counts parameter passes: each step makes 2N
perturb/restore passes and one N-member update pass over P parameters, so
value = (2N + 1) P / step time.  Per-kernel figures come from HIP events
recorded on the launch stream around every launch inside the timed region.

    python bench.py [--steps K] [--warmup W] [--workload dense-27b]
"""
import argparse
import gc
import json
import math
import multiprocessing as mp
import os
import sys
import time

import numpy as np

REPO = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, REPO)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, public spec
VALU_PEAK_TINST = 256 * 64 * 2.4e9 / 1e12   # 39.3 T lane-instructions/s (256 CU x 64 lanes x 2.4 GHz)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="dense-27b")
    ap.add_argument("--members", type=int, default=None, help="override N (distinct seeds)")
    ap.add_argument("--no-swap-walk", action="store_true",
                    help="do not time the same generations with fused swaps")
    ap.add_argument("--sweep-members", default=None, metavar="N1,N2,...",
                    help="large-population sweep of the fused update on the 4B-shaped set "
                         "(one JSON line per N)")
    ap.add_argument("--int8", action="store_true",
                    help="the int8 path: codes with per-row scales, es_qperturb / es_qrestore / "
                         "es_qupdate")
    ap.add_argument("--fp8", action="store_true",
                    help="the fp8 path: E4M3 codes with per-row scales (es_qplan_create_format)")
    ap.add_argument("--stochastic-round", action="store_true",
                    help="round the update stochastically (ES_UPDATE_STOCHASTIC_ROUND)")
    ap.add_argument("--master", action="store_true",
                    help="binary32 masters of every parameter (es_plan_set_master); the update "
                         "goes into them and rewrites the bf16 values (ES_UPDATE_MASTER)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="target CPU time of the oracle baseline sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--profile-pass", action="store_true",
                    help="launch every kernel once per label for rocprofv3 (with --sweep-members: "
                         "one update per N)")
    ap.add_argument("--labels-dir", default=None,
                    help="where a profile pass writes labels.json")
    ap.add_argument("--profile-repeat", type=int, default=3,
                    help="launches per label in a profile pass")
    ap.add_argument("--counters-json", default=os.path.join(REPO, "profiles", "counters.json"),
                    help="per-launch counter values measured with rocprofv3 (see --summarize)")
    ap.add_argument("--summarize-trace", default=None, metavar="TRACE_DIR",
                    help="turn a kernel trace of the bench command into profiles/")
    ap.add_argument("--summarize", default=None, metavar="OUT_DIR",
                    help="turn the rocprofv3 runs of a profile pass (OUT_DIR/trace, fetch, write, "
                         "valu) into profiles/")

    return ap.parse_args()


def step_seeds(W, t, n_members):
    """Seeds of generation t: a fresh seed per distinct member seed."""
    base = W.seeds if n_members is None else tuple(range(n_members))
    return [int(s) + 1_000_003 * (t + 1) for s in base]


def live_seeds(seeds, signs, rewards):
    """Distinct seeds whose noise the update generates: those whose merged
    weight, proportional to the sum of sign_i (R_i - mean R) over the seed's
    members, is nonzero (none when every reward is equal).  The kernel skips
    the others, so they count no normals.  Reporting only."""
    r = np.asarray(rewards, np.float64)
    if np.all(r == r[0]):
        return 0
    mu = r.mean()
    acc = {}
    for s, sg, x in zip(seeds, signs, r):
        acc[s] = acc.get(s, 0.0) + sg * (x - mu)
    return sum(1 for v in acc.values() if v != 0.0)


def sigma_at(sigma_cosine, W, t):
    """sigma_t of generation t on the cosine schedule of Section 3.1, from the
    library's es_sigma_cosine (the GPU leg) or the oracle's (the CPU leg);
    generations past the schedule's last update keep sigma_T."""
    return sigma_cosine(W.sigma0, W.sigma_T, min(t, W.T), W.T)


CPU_WORKER_CAP = 16    # CPU share of one GPU slot on a shared host


def cpu_workers():
    """Worker processes of the CPU leg: every CPU this process may run on
    (its affinity mask), capped at CPU_WORKER_CAP.  Returns (workers,
    available CPUs)."""
    try:
        avail = len(os.sched_getaffinity(0))
    except AttributeError:
        avail = os.cpu_count() or 1
    return max(1, min(avail, CPU_WORKER_CAP)), avail


# ---------------------------------------------------------------- CPU leg --

def _oracle_chunk(args):
    """The oracle's work of one step on a sample of one tensor's elements."""
    import oracle
    theta, tid, elems, seeds, signs, rewards, alpha, sigma = args
    t0 = time.perf_counter()
    for s, sg in zip(seeds, signs):
        p = oracle.perturb(theta, s, tid, sg, sigma, elems=elems)
        theta = oracle.restore(p, s, tid, sg, sigma, elems=elems)
    theta, _ = oracle.update(theta, tid, seeds, signs, rewards, alpha, sigma, elems=elems)
    return time.perf_counter() - t0


def cpu_baseline(W, seeds, signs, rewards, sigma, theta_samples, workers, budget_s):
    """Time the oracle (as it stands) on a bounded element sample; returns the
    rate in parameter passes per second and a description of the sample."""
    n = len(seeds)
    # calibrate: one small chunk on one core
    t_small = _oracle_chunk((theta_samples[0][1][:4096], theta_samples[0][0],
                             theta_samples[0][2][:4096], seeds, signs, rewards, W.alpha, sigma))
    per_elem = t_small / 4096
    total = sum(len(x[1]) for x in theta_samples)
    target = int(budget_s * workers / per_elem)
    frac = min(1.0, target / total)
    jobs = []
    for tid, theta, elems in theta_samples:
        k = max(1, int(len(elems) * frac))
        jobs.append((theta[:k], tid, elems[:k], seeds, signs, rewards, W.alpha, sigma))
    n_elems = sum(len(j[2]) for j in jobs)
    t0 = time.perf_counter()
    with mp.get_context("fork").Pool(workers) as pool:
        pool.map(_oracle_chunk, jobs, chunksize=1)
    wall = time.perf_counter() - t0
    rate = (2 * n + 1) * n_elems / wall
    return {"value": rate, "unit": "params/s", "cores": workers, "kind": "oracle",
            **host_cpu(),
            "full_step_s_extrapolated": round((2 * n + 1) * W.n_params / rate, 1),
            "sample": f"{n_elems} elements sampled across {len(jobs)} tensors of {W.name}, "
                      f"one full step (N={n}: {2 * n} perturb/restore + 1 update) in fp64 "
                      f"NumPy over {workers} worker processes, {wall:.1f} s wall"}


def flat_ceilings(esopt, stream, gib=16):
    """Read-only, write-only and in-place rates of the device's memory over a
    flat buffer (es_hbm_calibrate: the perturb's tile shape and launch),
    medians of three passes each; the in-place rate counts read and written
    bytes, like the passes' algorithmic rates."""
    import torch
    cal = torch.empty(gib << 30, dtype=torch.uint8, device="cuda")
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    out = {"buffer_bytes": cal.numel()}
    for name, mode, factor in (("read_GBps", esopt.CALIBRATE_READ, 1),
                               ("write_GBps", esopt.CALIBRATE_WRITE, 1),
                               ("in_place_GBps", esopt.CALIBRATE_READ_WRITE, 2)):
        esopt.hbm_calibrate(cal, mode, sink)
        ts = []
        for _ in range(3):
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            esopt.hbm_calibrate(cal, mode, sink)
            e1.record(stream)
            e1.synchronize()
            ts.append(e0.elapsed_time(e1))
        out[name] = round(factor * cal.numel() / (float(np.median(ts)) / 1e3) / 1e9, 1)
    del cal
    torch.cuda.empty_cache()
    return out


def host_cpu():
    """The host's CPU model (from /proc/cpuinfo), its logical CPU count, the
    CPUs this process may use and the cap on worker processes."""
    model = None
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"cpu_model": model, "host_logical_cpus": os.cpu_count(),
            "cpus_available": cpu_workers()[1], "worker_cap": CPU_WORKER_CAP}


def host_samples(W, per_tensor=1 << 16):
    """A bounded element sample of every tensor of W: random element indices
    and N(0, 0.02) bf16 values drawn on the host (the oracle's cost does not
    depend on the values)."""
    from paper_2608_17310_amd import workloads as wl
    rng = np.random.default_rng(0)
    out = []
    for tid, n in enumerate(W.numels):
        idx = np.unique(rng.integers(0, n, size=min(n, per_tensor))).astype(np.uint64)
        out.append((tid, wl.random_bf16_bits(idx.size, 1000 + tid), idx))
    return out


def _oracle_qchunk(args):
    """The oracle's work of one int8 or fp8 step on a sample of one tensor's
    codes."""
    import oracle
    q, scales, row, tid, elems, seeds, signs, rewards, alpha, sigma, fmt = args
    if fmt == "e4m3":
        perturb, restore, update = oracle.f8perturb, oracle.f8restore, oracle.f8update
    else:
        perturb, restore, update = oracle.qperturb, oracle.qrestore, oracle.qupdate
    t0 = time.perf_counter()
    for s, sg in zip(seeds, signs):
        p = perturb(q, scales, row, s, tid, sg, sigma, elems=elems)
        q = restore(p, scales, row, s, tid, sg, sigma, elems=elems)
    q, _ = update(q, scales, row, tid, seeds, signs, rewards, alpha, sigma, elems=elems,
                  round_seed=1)
    return time.perf_counter() - t0


def cpu_baseline_int8(W, seeds, signs, rewards, sigma, workers, budget_s, per_tensor=1 << 14,
                      fmt="int8"):
    """The oracle's int8 (or fp8) step on a bounded sample: random codes and
    indices, per-row scales of the workload's shapes (values do not change
    the cost)."""
    from paper_2608_17310_amd import workloads as wl
    rng = np.random.default_rng(0)
    samples = []
    for tid, (n, shape) in enumerate(zip(W.numels, W.shapes)):
        row = wl.row_of(shape)
        idx = np.unique(rng.integers(0, n, size=min(n, per_tensor))).astype(np.uint64)
        if fmt == "e4m3":
            scales = rng.uniform(1.5e-4, 3e-4, 1 if row == 0 else n // row).astype(np.float32)
            codes = rng.integers(0, 0x7E, size=idx.size).astype(np.uint8) | \
                (rng.integers(0, 2, size=idx.size).astype(np.uint8) << 7)
        else:
            scales = rng.uniform(3e-4, 1e-3, 1 if row == 0 else n // row).astype(np.float32)
            codes = rng.integers(-127, 128, size=idx.size).astype(np.int8)
        samples.append((codes, scales, row, tid, idx))
    n = len(seeds)
    c0 = samples[0]
    t_small = _oracle_qchunk((c0[0][:1024], c0[1], c0[2], c0[3], c0[4][:1024], seeds, signs,
                              rewards, W.alpha, sigma, fmt))
    per_elem = t_small / 1024
    total = sum(x[4].size for x in samples)
    frac = min(1.0, int(budget_s * workers / per_elem) / total)
    jobs = []
    for codes, scales, row, tid, idx in samples:
        k = max(1, int(idx.size * frac))
        jobs.append((codes[:k], scales, row, tid, idx[:k], seeds, signs, rewards, W.alpha, sigma,
                     fmt))
    n_elems = sum(j[4].size for j in jobs)
    t0 = time.perf_counter()
    with mp.get_context("fork").Pool(workers) as pool:
        pool.map(_oracle_qchunk, jobs, chunksize=1)
    wall = time.perf_counter() - t0
    rate = (2 * n + 1) * n_elems / wall
    return {"value": rate, "unit": "params/s", "cores": workers, "kind": "oracle",
            **host_cpu(),
            "full_step_s_extrapolated": round((2 * n + 1) * W.n_params / rate, 1),
            "sample": f"{n_elems} {fmt} codes sampled across {len(jobs)} tensors of {W.name}, "
                      f"one full {fmt} step (N={n}: {2 * n} perturb/restore + 1 update) in fp64 "
                      f"NumPy over {workers} worker processes, {wall:.1f} s wall"}


# ---------------------------------------------------------------- GPU leg --

def run_sweep(args):
    """The fused update alone on the 4B-shaped set for each population size N
    (distinct seeds, rewards N(0,1)): where the update turns from HBM-bound
    (4 B per parameter whatever N) to VALU-bound (N normals per parameter)."""
    import torch
    from paper_2608_17310_amd import esopt, workloads as wl
    torch.cuda.set_device(0)
    ns = [int(x) for x in args.sweep_members.split(",")]
    W = wl.DENSE_4B
    flat, views = wl.device_params(W)
    plan = esopt.Plan(views)
    P = plan.numel
    stream = torch.cuda.current_stream()

    def median_ms(fn):
        fn()
        ts = []
        for _ in range(max(args.steps, 1)):
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            fn()
            e1.record(stream)
            e1.synchronize()
            ts.append(e0.elapsed_time(e1))
        return float(np.median(ts))

    if args.profile_pass:
        log = ProfileLog(args.labels_dir)
        R = args.profile_repeat
        log.add("warm-up in-place copy", "warmup", P, 4 * P, 0, plan.stream_pass, members=-1)
        log.add("es_stream_pass (in-place copy over the plan's tiles)", "ceiling", P, 4 * P, 0,
                plan.stream_pass, members=0, repeat=R)
        for n in ns:
            Wn = wl.sweep_workload(n)
            r = torch.from_numpy(wl.rewards(Wn)).cuda()
            flags = esopt.ES_REWARDS_ARE_WEIGHTS if n == 1 else 0
            log.add(f"es_update (N={n})", "update", P, 4 * P, n * P, plan.update, list(Wn.seeds),
                    list(Wn.signs), r, Wn.alpha, flags=flags, members=n, repeat=R)
        torch.cuda.synchronize()
        plan.close()
        del flat, views
        torch.cuda.empty_cache()
        calibration_copy(torch)
        torch.cuda.synchronize()
        log.write({"sweep": True, "workload": W.name, "params": P,
                   "source_hash": _kernel_source_hash(),
                   "pass_args": f"--sweep-members {args.sweep_members} --profile-pass"})
        print(json.dumps({"profile_pass": W.name + " sweep", "launches": len(log.rows)}))
        return
    # the practical HBM floor of any pass over these tiles: the in-place copy
    stream_t = median_ms(plan.stream_pass) / 1e3
    for n in ns:
        Wn = wl.sweep_workload(n)
        r = torch.from_numpy(wl.rewards(Wn)).cuda()
        seeds = list(Wn.seeds)
        # one member z-scores to zero (no update): use its reward as the weight
        flags = esopt.ES_REWARDS_ARE_WEIGHTS if n == 1 else 0
        plan.update(seeds, list(Wn.signs), r, Wn.alpha, flags=flags)
        ts = []
        for _ in range(max(args.steps, 1)):
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            plan.update(seeds, list(Wn.signs), r, Wn.alpha, flags=flags)
            e1.record(stream)
            e1.synchronize()
            ts.append(e0.elapsed_time(e1) / 1e3)
        t = float(np.median(ts))
        hbm_t = 4 * P / (HBM_PEAK_GBS * 1e9)
        print(json.dumps({"sweep": "fused es_update", "workload": W.name, "params": P, "members": n,
                          "ms": round(t * 1e3, 3), "params_per_s": P / t,
                          "normals_per_s": n * P / t,
                          "GBps_algorithmic": round(4 * P / t / 1e9, 1),
                          "hbm_time_at_peak_ms": round(hbm_t * 1e3, 3),
                          "stream_pass_ms": round(stream_t * 1e3, 3),
                          # within 1.5x of the in-place copy of the same memory: HBM-bound
                          "bound": "hbm" if t < 1.5 * stream_t else "valu"}), flush=True)
    plan.close()


def run_quantized(args):
    """The int8 (or, with --fp8, the E4M3) step on the workload's shapes:
    N x (es_qperturb + es_qrestore) + es_qupdate over codes with per-row
    scales, inputs resident in HBM."""
    import torch
    from paper_2608_17310_amd import esopt, workloads as wl
    fmt = "e4m3" if args.fp8 else "int8"
    tag = "fp8" if args.fp8 else "int8"
    W = wl.WORKLOADS[args.workload]
    n_members = args.members
    signs = list(W.signs) if n_members is None else [1] * n_members
    N = len(signs)
    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        cpu = cpu_baseline_int8(W, step_seeds(W, args.warmup, n_members), signs,
                                wl.rewards(W, args.warmup, n=N),
                                sigma_at(oracle.sigma_cosine, W, args.warmup),
                                cpu_workers()[0], args.cpu_seconds, fmt=fmt)
    if not torch.cuda.is_available():
        print(json.dumps({"error": "no GPU"}))
        sys.exit(1)
    torch.cuda.set_device(0)
    flat, views, scales, rows = (wl.device_f8params if args.fp8 else wl.device_qparams)(W)
    plan = esopt.QPlan(views, scales, rows, format=fmt)
    P = plan.numel
    stream = torch.cuda.current_stream()
    total_steps = args.warmup + args.steps
    rewards_np = np.stack([wl.rewards(W, t, n=N) for t in range(total_steps)])
    rewards_all = torch.from_numpy(rewards_np).cuda()
    torch.cuda.synchronize()
    log = EventLog(torch, stream)

    def run_step(t, record, swap=False):
        seeds = step_seeds(W, t, n_members)
        sigma = sigma_at(esopt.sigma_cosine, W, t)
        if swap:
            log.call("es_qperturb", record, plan.perturb, seeds[0], signs[0], sigma)
            for i in range(N - 1):
                log.call("es_qswap", record, plan.swap, seeds[i], signs[i], seeds[i + 1],
                         signs[i + 1], sigma)
            log.call("es_qrestore", record, plan.restore, seeds[-1], signs[-1], sigma)
        else:
            for sd, sg in zip(seeds, signs):
                log.call("es_qperturb", record, plan.perturb, sd, sg, sigma)
                log.call("es_qrestore", record, plan.restore, sd, sg, sigma)
        log.call("es_qupdate", record, plan.update, seeds, signs, rewards_all[t], W.alpha,
                 sigma=sigma, round_seed=1000 + t)

    for t in range(args.warmup):
        run_step(t, record=False)
    ms_step, wall = timed_region(torch, stream, args.steps,
                                 lambda i: run_step(args.warmup + i, record=True))
    per = log.ms()
    t_pert = median_s(per["es_qperturb"] + per["es_qrestore"])
    t_upd = median_s(per["es_qupdate"])
    # the same generations with the members moved by fused swaps (es_qperturb,
    # N - 1 es_qswap, es_qrestore, es_qupdate), timed in the same run after
    # one untimed generation
    swap = None
    if not args.no_swap_walk and N > 1:
        log.ev = []
        run_step(args.warmup, record=False, swap=True)
        ms_swap, wall_swap = timed_region(
            torch, stream, args.steps, lambda i: run_step(args.warmup + i, record=True, swap=True))
        per_sw = log.ms()
        swap = {"ms_step": ms_swap, "wall": wall_swap, "t_swap": median_s(per_sw["es_qswap"]),
                "calls": len(per_sw["es_qswap"])}
    value = (2 * N + 1) * P / (ms_step / 1e3)
    n_distinct = len(dict.fromkeys(step_seeds(W, 0, n_members)))
    n_live = float(np.mean([live_seeds(step_seeds(W, t, n_members), signs, rewards_np[t])
                            for t in range(args.warmup, total_steps)]))
    label = f"{W.name}-{tag}"
    c_pert = _counters_for(args.counters_json, f"es_{'f8' if args.fp8 else 'q'}perturb", label)
    c_upd = _counters_for(args.counters_json, f"es_{'f8' if args.fp8 else 'q'}update", label)
    c_swap = _counters_for(args.counters_json, f"es_{'f8' if args.fp8 else 'q'}swap", label)

    def alu_roofline(c, t, kernel, extra):
        r = {"bound": "alu", "unit": "T lane-instr/s", "peak": round(VALU_PEAK_TINST, 2),
             "achieved": None, "frac": None, "kernel": kernel,
             "traffic": c["bytes_per_launch"] if c else None,
             "algorithmic_bytes_per_launch": 2 * P,
             "achieved_GBps_algorithmic": round(2 * P / t / 1e9, 1)}
        if c and extra:
            ach = c["valu_insts_per_launch"] * 64 / t / 1e12
            r.update(achieved=round(ach, 2), frac=round(ach / VALU_PEAK_TINST, 4))
        return r
    same_config = N == len(W.seeds) and n_members is None
    out = {
        "metric": f"params/s of the {tag} ES step (es_qperturb/es_qrestore and fused "
                  f"es_qupdate, N members)",
        "value": value, "unit": "params/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_step, 3), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "param_dtype": "e4m3" if args.fp8 else "int8",
        "data": "synthetic",
        "config": {"workload": label, "params": P, "tensors": len(views), "members": N,
                   "param_bytes": P + 4 * sum(int(x.numel()) for x in scales),
                   "plan_device_bytes": plan.device_bytes,
                   "distinct_seeds": n_distinct, "sigma0": W.sigma0, "alpha": W.alpha,
                   "scales": "one binary32 scale per row of the last dimension, one per vector"
                             + (" (absmax / 448)" if args.fp8 else " (absmax / 127)"),
                   "counting": "value = (2N+1) P / step time: 2N perturb/restore passes and one "
                               "fused N-member update pass per step"},
        "roofline": alu_roofline(c_pert, t_pert, f"es_qpass_kernel, {fmt} "
                                 "(es_qperturb / es_qrestore)", True),
        "roofline_update": alu_roofline(c_upd, t_upd, f"es_qpass_kernel, {fmt} (es_qupdate)",
                                        same_config),
        "per_kernel": {
            "es_qperturb": {"ms": round(t_pert * 1e3, 3), "params_per_s": P / t_pert,
                            "GBps_algorithmic": round(2 * P / t_pert / 1e9, 1)},
            "es_qupdate": {"ms": round(t_upd * 1e3, 3), "params_per_s": P / t_upd,
                           "normals_per_s": n_live * P / t_upd,
                           "distinct_seeds": n_distinct, "live_seeds": round(n_live, 3)}},
        "timing": "per-kernel figures are medians of HIP event pairs on the launch stream",
        "wall_s_timed": round(wall, 3),
        "cpu_baseline": cpu,
    }
    if swap is not None:
        t_sw = swap["t_swap"]
        out["per_kernel"]["es_qswap"] = {"ms": round(t_sw * 1e3, 3), "params_per_s": P / t_sw,
                                         "normals_per_s": 2 * P / t_sw, "calls": swap["calls"],
                                         "ms_over_perturb_restore": round(t_sw / (2 * t_pert), 4)}
        out["ms_per_step_swap"] = round(swap["ms_step"], 3)
        out["swap_walk"] = {
            "member_moves": "es_qperturb, N-1 fused es_qswap, es_qrestore, then es_qupdate",
            "ms_per_step": round(swap["ms_step"], 3),
            "speedup_vs_perturb_restore": round(ms_step / swap["ms_step"], 4),
            "wall_s_timed": round(swap["wall"], 3),
            "roofline": alu_roofline(c_swap, t_sw, f"es_qpass_kernel, {fmt} (es_qswap)", True)}
    print(json.dumps(out))
    plan.close()


class EventLog:
    """HIP events recorded on the launch stream around each timed launch;
    per-kind durations are reported as medians."""

    def __init__(self, torch, stream):
        self.torch, self.stream, self.ev = torch, stream, []

    def call(self, kind, record, fn, *a, **kw):
        if not record:
            return fn(*a, **kw)
        e0 = self.torch.cuda.Event(enable_timing=True)
        e1 = self.torch.cuda.Event(enable_timing=True)
        e0.record(self.stream)
        out = fn(*a, **kw)
        e1.record(self.stream)
        self.ev.append((kind, e0, e1))
        return out

    def ms(self):
        per = {}
        for kind, a, b in self.ev:
            per.setdefault(kind, []).append(a.elapsed_time(b))
        return per


def median_s(xs_ms):
    return float(np.median(xs_ms)) / 1e3


def timed_region(torch, stream, steps, fn):
    """Run fn(i) for i < steps between two events on the launch stream, with
    the host's garbage collector off (a 35 ms collector pause was once seen
    inside a short step); returns (ms per step, wall seconds)."""
    torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    gc.collect()
    gc.disable()
    t_wall0 = time.perf_counter()
    start.record(stream)
    for i in range(steps):
        fn(i)
    end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_wall0
    gc.enable()
    return start.elapsed_time(end) / steps, wall


def master_views(torch, flat, views):
    """Binary32 masters of a flat bf16 parameter buffer's tensors: one float32
    buffer holding the values (4 bytes per parameter: 91 GB for the 27B-shaped
    set, which one MI355X's 288 GB holds beside the bf16 copy), viewed at the
    same offsets (each view 16-byte aligned, as the bf16 views are)."""
    mflat = flat.float()
    base = flat.data_ptr()
    out = []
    for v in views:
        off = (v.data_ptr() - base) // 2
        out.append(mflat[off:off + v.numel()])
    return mflat, out


def main():
    args = parse()
    if args.summarize:
        summarize(args.summarize)
        return
    if args.summarize_trace:
        summarize_bench_trace(args.summarize_trace, workload=args.workload, master=args.master)
        return
    if args.gpus != 1:
        print(json.dumps({"error": "the ES parameter path runs on one GPU; --gpus above 1 is "
                                   "not supported (population parallelism across GPUs is not "
                                   "implemented)"}))
        sys.exit(2)
    if args.sweep_members:
        return run_sweep(args)
    if args.profile_pass:
        return run_profile_pass(args)
    if args.int8 or args.fp8:
        return run_quantized(args)
    import torch
    from paper_2608_17310_amd import workloads as wl

    W = wl.WORKLOADS[args.workload]
    n_members = args.members
    signs = list(W.signs) if n_members is None else [1] * n_members
    N = len(signs)
    cpu = None
    if not args.no_cpu_baseline:
        # before the GPU (or the HIP library) is touched: worker processes
        # fork from a clean parent; sigma from the oracle's schedule
        import oracle
        workers, _ = cpu_workers()
        cpu = cpu_baseline(W, step_seeds(W, args.warmup, n_members), signs,
                           wl.rewards(W, args.warmup, n=N),
                           sigma_at(oracle.sigma_cosine, W, args.warmup),
                           host_samples(W), workers, args.cpu_seconds)

    from paper_2608_17310_amd import esopt
    if not torch.cuda.is_available():
        print(json.dumps({"error": "no GPU"}))
        sys.exit(1)
    torch.cuda.set_device(0)
    flat, views = wl.device_params(W)
    plan = esopt.Plan(views)
    P = plan.numel
    stream = torch.cuda.current_stream()
    total_steps = args.warmup + args.steps
    rewards_np = np.stack([wl.rewards(W, t, n=N) for t in range(total_steps)])
    rewards_all = torch.from_numpy(rewards_np).cuda()
    torch.cuda.synchronize()

    log = EventLog(torch, stream)
    update_flags = esopt.ES_UPDATE_STOCHASTIC_ROUND if args.stochastic_round else 0
    if args.master:
        if args.stochastic_round:
            raise SystemExit("--master rounds the bf16 copy to nearest-even: no --stochastic-round")
        mflat, masters = master_views(torch, flat, views)
        plan.set_master(masters)
        update_flags = esopt.ES_UPDATE_MASTER

    def run_step(t, record, swap):
        """One generation's parameter work: every member applied and reverted
        (separate passes, then the fused update; or perturb, N - 1 fused swaps,
        and the last member's revert fused into the update)."""
        seeds = step_seeds(W, t, n_members)
        sigma = sigma_at(esopt.sigma_cosine, W, t)
        if swap:
            log.call("es_perturb", record, plan.perturb, seeds[0], signs[0], sigma)
            for i in range(N - 1):
                log.call("es_swap", record, plan.swap, seeds[i], signs[i], seeds[i + 1],
                         signs[i + 1], sigma)
            if args.master:                 # the update rewrites the bf16 values
                log.call("es_update", record, plan.update, seeds, signs, rewards_all[t],
                         W.alpha, sigma=sigma, flags=update_flags)
                return
            log.call("es_restore_update", record, plan.restore_update, seeds[-1], signs[-1],
                     sigma, seeds, signs, rewards_all[t], W.alpha, sigma=sigma,
                     flags=update_flags, round_seed=1000 + t)
            return
        elif args.master:                   # every member applied from the masters
            for sd, sg in zip(seeds, signs):
                log.call("es_perturb_master", record, plan.perturb_master, sd, sg, sigma)
        else:
            for sd, sg in zip(seeds, signs):
                log.call("es_perturb", record, plan.perturb, sd, sg, sigma)
                log.call("es_restore", record, plan.restore, sd, sg, sigma)
        log.call("es_update", record, plan.update, seeds, signs, rewards_all[t], W.alpha,
                 sigma=sigma, flags=update_flags, round_seed=1000 + t)

    for t in range(args.warmup):
        run_step(t, record=False, swap=False)
    ms_step, wall = timed_region(torch, stream, args.steps,
                                 lambda i: run_step(args.warmup + i, record=True, swap=False))
    per = log.ms()
    if args.master:
        # the perturb roofline stays es_perturb's, timed separately below
        t_pmaster = median_s(per["es_perturb_master"])
        for _ in range(3):
            log.call("es_perturb", True, plan.perturb, 1, 1, W.sigma0)
            log.call("es_restore", True, plan.restore, 1, 1, W.sigma0)
        torch.cuda.synchronize()
        per = log.ms()
    t_pert = median_s(per["es_perturb"] + per["es_restore"])
    t_upd = median_s(per["es_update"])
    passes = N + 1 if args.master else 2 * N + 1
    value = passes * P / (ms_step / 1e3)
    n_distinct = len(dict.fromkeys(step_seeds(W, 0, n_members)))
    n_live = float(np.mean([live_seeds(step_seeds(W, t, n_members), signs, rewards_np[t])
                            for t in range(args.warmup, total_steps)]))

    # the same generations with the members moved by fused swaps (perturb,
    # N - 1 swaps, the last revert and the update in one pass), timed in the
    # same run after one untimed generation
    swap = None
    if not args.no_swap_walk and N > 1:
        log.ev = []
        run_step(args.warmup, record=False, swap=True)
        ms_swap, wall_swap = timed_region(
            torch, stream, args.steps, lambda i: run_step(args.warmup + i, record=True, swap=True))
        per_sw = log.ms()
        swap = {"ms_step": ms_swap, "wall": wall_swap, "t_swap": median_s(per_sw["es_swap"]),
                "calls": len(per_sw["es_swap"]),
                "t_restore_update": (None if args.master
                                     else median_s(per_sw["es_restore_update"]))}

    # the practical in-place streaming ceiling over the same memory: the same
    # tiles and launch, loads and stores only, not pipelined (es_stream_pass),
    # timed after the steps; then the flat-buffer read / write / in-place rates
    plan.stream_pass()
    log.ev = []
    for _ in range(5):
        log.call("es_stream_pass", True, plan.stream_pass)
    torch.cuda.synchronize()
    t_stream = median_s(log.ms()["es_stream_pass"])
    ceiling_gbs = 4 * P / t_stream / 1e9
    flat_rates = flat_ceilings(esopt, stream)
    c_pert = _counters_for(args.counters_json, "es_perturb", W.name)
    c_upd = _counters_for(args.counters_json,
                          "es_update_master" if args.master else "es_update", W.name)
    c_swap = _counters_for(args.counters_json, "es_swap", W.name)
    perturb_gbs = 4 * P / t_pert / 1e9
    roofline = {"bound": "hbm", "achieved": round(perturb_gbs, 1), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(perturb_gbs / HBM_PEAK_GBS, 4),
                "traffic": c_pert["bytes_per_launch"] if c_pert else None,
                "kernel": "es_perturb_kernel (es_perturb / es_restore)",
                "algorithmic_bytes_per_launch": 4 * P,
                "ceiling": {"GBps": round(ceiling_gbs, 1),
                            "frac_of_ceiling": round(perturb_gbs / ceiling_gbs, 4),
                            "kernel": "es_stream_kernel: in-place copy of every parameter, same "
                                      "tiles (es_stream_pass)"},
                "flat_buffer_ceilings": flat_rates}

    def valu_roofline(c, t, kernel, comparable):
        """A VALU-bound kernel against the VALU issue peak: instructions per
        launch from counters (same workload and kernel sources), duration
        live."""
        r = {"bound": "alu", "unit": "T lane-instr/s", "peak": round(VALU_PEAK_TINST, 2),
             "achieved": None, "frac": None, "kernel": kernel,
             "traffic": c["bytes_per_launch"] if c else None}
        if c and comparable:
            ach = c["valu_insts_per_launch"] * 64 / t / 1e12
            r.update(achieved=round(ach, 2), frac=round(ach / VALU_PEAK_TINST, 4))
        return r
    default_pop = N == len(W.seeds) and n_members is None
    upd_bytes = 10 * P if args.master else 4 * P    # masters: 4 read + 4 written, bf16 2 written
    update = {"ms": round(t_upd * 1e3, 3), "params_per_s": P / t_upd,
              "GBps_algorithmic": round(upd_bytes / t_upd / 1e9, 1),
              "normals_per_s": n_live * P / t_upd, "distinct_seeds": n_distinct,
              "live_seeds": round(n_live, 3)}
    per_kernel = {
        "es_perturb": {"ms": round(t_pert * 1e3, 3), "params_per_s": P / t_pert,
                       "GBps_algorithmic": round(perturb_gbs, 1),
                       "frac_hbm_peak": round(perturb_gbs / HBM_PEAK_GBS, 4)},
        "es_update": update,
        "es_stream_pass": {"ms": round(t_stream * 1e3, 3), "GBps": round(ceiling_gbs, 1)},
    }
    if args.master:
        c_pm = _counters_for(args.counters_json, "es_perturb_master", W.name)
        per_kernel["es_perturb_master"] = {
            "ms": round(t_pmaster * 1e3, 3), "params_per_s": P / t_pmaster,
            "GBps_algorithmic": round(6 * P / t_pmaster / 1e9, 1),
            "frac_hbm_peak": round(6 * P / t_pmaster / 1e9 / HBM_PEAK_GBS, 4),
            "algorithmic_bytes_per_launch": 6 * P,
            "traffic": c_pm["bytes_per_launch"] if c_pm else None}
    out = {
        "metric": "params/s and achieved HBM GB/s for es_perturb and fused es_update (N members)",
        "value": value,
        "unit": "params/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_step, 3),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32", "param_dtype": "bf16", "data": "synthetic",
        "config": {"workload": W.name, "params": P, "tensors": len(views), "members": N,
                   "param_bytes": 2 * P, "plan_device_bytes": plan.device_bytes,
                   "distinct_seeds": n_distinct, "sigma0": W.sigma0, "alpha": W.alpha,
                   "update_rounding": ("binary32 masters, bf16 copy nearest-even"
                                       if args.master else
                                       "stochastic" if args.stochastic_round else "nearest-even"),
                   "member_moves": ("es_perturb_master (each member applied from the "
                                    "masters; no revert)" if args.master else
                                    "es_perturb/es_restore"),
                   "counting": ("value = (N+1) P / step time: N passes applying a member from "
                                "the masters (no revert) and one N-member update into binary32 "
                                "masters" if args.master else
                                "value = (2N+1) P / step time: 2N perturb/restore passes "
                                "and one fused N-member update pass per step")},
        "roofline": roofline,
        "roofline_update": valu_roofline(c_upd, t_upd, "es_update_kernel (fused N-member update)",
                                         default_pop and not args.stochastic_round),
        "per_kernel": per_kernel,
        "timing": "per-kernel figures are medians of HIP event pairs on the launch stream",
        "wall_s_timed": round(wall, 3),
    }
    if swap is not None:
        t_sw = swap["t_swap"]
        per_kernel["es_swap"] = {"ms": round(t_sw * 1e3, 3), "params_per_s": P / t_sw,
                                 "GBps_algorithmic": round(4 * P / t_sw / 1e9, 1),
                                 "normals_per_s": 2 * P / t_sw, "calls": swap["calls"]}
        out["ms_per_step_swap"] = round(swap["ms_step"], 3)
        if swap["t_restore_update"] is not None:
            per_kernel["es_restore_update"] = {
                "ms": round(swap["t_restore_update"] * 1e3, 3),
                "ms_over_update": round(swap["t_restore_update"] / t_upd, 4)}
        out["swap_walk"] = {
            "member_moves": ("es_perturb, N-1 fused es_swap, then the update into the masters "
                             "(no last revert)" if args.master else
                             "es_perturb, N-1 fused es_swap, then the last revert and the update "
                             "in one pass (es_restore_update)"),
            "ms_per_step": round(swap["ms_step"], 3),
            "speedup_vs_perturb_restore": round(ms_step / swap["ms_step"], 4),
            "wall_s_timed": round(swap["wall"], 3),
            "roofline": valu_roofline(c_swap, t_sw, "es_perturb_kernel<..., 2> (es_swap, two keys)",
                                      True)}
    if cpu is not None:
        out["cpu_baseline"] = cpu
    plan.close()
    print(json.dumps(out))


# ------------------------------------------------------------ profiling --
#
# A profile pass launches each of the library's kernels once per label (no
# timing of its own) and writes the labels, in launch order, to
# <dir>/labels.json.  rocprofv3 runs the same pass several times -- a kernel
# trace and one run per counter set -- and --summarize matches the k-th
# dispatch of a library kernel in each run's CSV to the k-th label.

LIBRARY_KERNELS = ("es_perturb_kernel", "es_update_kernel", "es_apply_master_kernel",
                   "es_stream_kernel", "es_calibrate_kernel", "es_qpass_kernel",
                   "es_checksum_kernel", "es_qchecksum_kernel")
COUNTER_SETS = {
    "fetch": "FETCH_SIZE",
    "write": "WRITE_SIZE",
    "valu": "SQ_INSTS_VALU SQ_ACTIVE_INST_VALU SQ_INSTS_VALU_TRANS_F32 SQ_WAVES SQ_BUSY_CYCLES "
            "GRBM_GUI_ACTIVE",
}
CALIBRATION_COPY_BYTES = 1 << 30
# counters are collected for the library's kernels and the calibration copy only
COUNTER_KERNEL_REGEX = "es_[a-z0-9_]*kernel|copyBuffer"


def profile_commands(pass_args):
    """The rocprofv3 runs behind a summary (<out>: an output directory)."""
    cmds = [f"rocprofv3 --kernel-trace --stats -f csv -d <out>/trace -o trace -- python3 bench.py "
            f"{pass_args} --labels-dir <out>/trace"]
    for run, counters in COUNTER_SETS.items():
        cmds.append(f"timeout -s KILL 300 rocprofv3 --pmc {counters} --kernel-include-regex "
                    f"'{COUNTER_KERNEL_REGEX}' -f csv -d <out>/{run} -o {run} "
                    f"-- python3 bench.py {pass_args} --labels-dir <out>/{run}")
    return cmds


class ProfileLog:
    """Labels of the library-kernel launches of a profile pass, in order."""

    def __init__(self, out_dir):
        self.out_dir, self.rows = out_dir, []

    def add(self, label, group, params, bytes_, normals, fn, *a, members=None, repeat=1, **kw):
        """Launch fn (exactly one library kernel) `repeat` times under
        `label`; bytes_ is the algorithmic memory traffic, normals the
        Gaussian draws per launch."""
        for _ in range(repeat):
            fn(*a, **kw)
            self.rows.append({"label": label, "group": group, "params": params,
                              "algorithmic_bytes": bytes_, "normals": normals,
                              "members": members})

    def write(self, extra):
        if self.out_dir:
            os.makedirs(self.out_dir, exist_ok=True)
            with open(os.path.join(self.out_dir, "labels.json"), "w") as fh:
                json.dump({"launches": self.rows, **extra}, fh, indent=1)


def calibration_copy(torch):
    """The device copy whose FETCH_SIZE / WRITE_SIZE readings scale the
    counters to bytes (a plain copy of known size)."""
    calib = torch.empty(CALIBRATION_COPY_BYTES, dtype=torch.uint8, device="cuda")
    torch.empty_like(calib).copy_(calib)


def run_profile_pass(args):
    """Every kernel of the step once on the workload (bf16 passes, the same
    passes over the matrices as column blocks, the int8 and fp8 passes on the
    same shapes), the in-place stream over the plan, the six flat-buffer
    calibration passes and the calibration copy."""
    import torch
    from paper_2608_17310_amd import esopt, workloads as wl
    torch.cuda.set_device(0)
    W = wl.WORKLOADS[args.workload]
    log = ProfileLog(args.labels_dir)
    seeds, signs = step_seeds(W, 0, None), list(W.signs)
    N = len(seeds)
    rewards = torch.from_numpy(wl.rewards(W, 0, n=N)).cuda()
    flat, views = wl.device_params(W)
    plan = esopt.Plan(views)
    P = plan.numel
    nd = len(dict.fromkeys(seeds))
    s0 = W.sigma0
    R = args.profile_repeat
    other = seeds[1] if N > 1 else seeds[0] + 1
    # a first pass over freshly written parameters runs slower: warm up (its
    # launches are labelled and left out of the summaries)
    log.add("warm-up perturb", "warmup", P, 4 * P, P, plan.perturb, seeds[0], signs[0], s0)
    log.add("warm-up restore", "warmup", P, 4 * P, P, plan.restore, seeds[0], signs[0], s0)
    for _ in range(R):         # alternating, so the parameters stay where they were
        log.add("es_perturb", "perturb", P, 4 * P, P, plan.perturb, seeds[0], signs[0], s0)
        log.add("es_restore", "perturb", P, 4 * P, P, plan.restore, seeds[0], signs[0], s0)
    for _ in range(R):
        log.add("es_swap (two keys)", "swap", P, 4 * P, 2 * P, plan.swap, seeds[0], 1, other, 1,
                s0)
        log.add("es_swap (two keys)", "swap", P, 4 * P, 2 * P, plan.swap, other, 1, seeds[0], 1,
                s0)
    log.add("es_swap (one key, antithetic)", "swap", P, 4 * P, P, plan.swap, seeds[0], 1,
            seeds[0], -1, s0, repeat=2 * R)
    log.add(f"es_update (N={N}, nearest-even)", "update", P, 4 * P, nd * P, plan.update, seeds,
            signs, rewards, W.alpha, sigma=s0, repeat=R)
    log.add(f"es_update (N={N}, stochastic rounding)", "update", P, 4 * P, nd * P, plan.update,
            seeds, signs, rewards, W.alpha, sigma=s0, flags=esopt.ES_UPDATE_STOCHASTIC_ROUND,
            round_seed=1, repeat=R)
    log.add(f"es_restore_update (N={N}, nearest-even; the last member reverted in the pass)",
            "update", P, 4 * P, nd * P, plan.restore_update, seeds[-1], signs[-1], s0, seeds,
            signs, rewards, W.alpha, sigma=s0, repeat=R)
    mflat, masters = master_views(torch, flat, views)
    plan.set_master(masters)
    log.add(f"es_update (N={N}, binary32 masters)", "update", P, 10 * P, nd * P, plan.update,
            seeds, signs, rewards, W.alpha, sigma=s0, flags=esopt.ES_UPDATE_MASTER, repeat=R)
    log.add("es_perturb_master (a member from binary32 masters)", "perturb", P, 6 * P, P,
            plan.perturb_master, seeds[0], signs[0], s0, repeat=R)
    torch.cuda.synchronize()
    plan.set_master(None)
    del mflat, masters
    torch.cuda.empty_cache()
    log.add("es_stream_pass (in-place copy over the plan's tiles)", "ceiling", P, 4 * P, 0,
            plan.stream_pass, repeat=R)
    out = torch.zeros(1, dtype=torch.int64, device="cuda")
    log.add("es_plan_checksum", "checksum", P, 2 * P, 0, plan.checksum, out, repeat=R)
    torch.cuda.synchronize()
    plan.close()
    # the same matrices as column blocks (es_plan_create_blocks): each 2-D
    # tensor's memory read as 8 consecutive [rows, cols / 8] blocks, block k
    # holding columns k cols / 8 .. of the tensor, so every pass takes the
    # strided launch with its row maps over the same bytes
    blocks = []
    for i, v in enumerate(views):
        if v.dim() != 2:
            continue
        r_, c_ = v.shape
        w = c_ // 8
        flat_v = v.reshape(-1)
        blocks += [esopt.Block(flat_v[k * r_ * w:(k + 1) * r_ * w].view(r_, w), 8 * i + k, c_, 0,
                               k * w) for k in range(8)]
    bplan = esopt.Plan(blocks=blocks)
    PB = bplan.numel
    # the first launches of a new plan and kernel run cold (left out of the
    # summaries, as above)
    log.add("warm-up perturb (column blocks)", "warmup", PB, 4 * PB, PB, bplan.perturb, seeds[0],
            signs[0], s0)
    log.add("warm-up restore (column blocks)", "warmup", PB, 4 * PB, PB, bplan.restore, seeds[0],
            signs[0], s0)
    for _ in range(R):
        log.add("es_perturb (column blocks)", "blocks", PB, 4 * PB, PB, bplan.perturb, seeds[0],
                signs[0], s0)
        log.add("es_restore (column blocks)", "blocks", PB, 4 * PB, PB, bplan.restore, seeds[0],
                signs[0], s0)
    log.add(f"es_update (N={N}, nearest-even, column blocks)", "blocks", PB, 4 * PB, nd * PB,
            bplan.update, seeds, signs, rewards, W.alpha, sigma=s0, repeat=R)
    log.add("es_stream_pass (column blocks)", "blocks", PB, 4 * PB, 0, bplan.stream_pass,
            repeat=R)
    torch.cuda.synchronize()
    bplan.close()
    del flat, views, blocks
    torch.cuda.empty_cache()

    qflat, qviews, scales, rows = wl.device_qparams(W)
    qplan = esopt.QPlan(qviews, scales, rows)
    QP = qplan.numel
    for _ in range(R):
        log.add("es_qperturb", "int8", QP, 2 * QP, QP, qplan.perturb, seeds[0], signs[0], s0)
        log.add("es_qswap", "int8", QP, 2 * QP, 2 * QP, qplan.swap, seeds[0], signs[0],
                seeds[1], signs[1], s0)
        log.add("es_qrestore", "int8", QP, 2 * QP, QP, qplan.restore, seeds[1], signs[1], s0)
    log.add(f"es_qupdate (N={N})", "int8", QP, 2 * QP, nd * QP, qplan.update, seeds, signs,
            rewards, W.alpha, sigma=s0, round_seed=1, repeat=R)
    torch.cuda.synchronize()
    qplan.close()
    del qflat, qviews, scales
    torch.cuda.empty_cache()

    fflat, fviews, fscales, frows = wl.device_f8params(W)
    fplan = esopt.QPlan(fviews, fscales, frows, format="e4m3")
    for _ in range(R):
        log.add("es_f8perturb", "fp8", QP, 2 * QP, QP, fplan.perturb, seeds[0], signs[0], s0)
        log.add("es_f8swap", "fp8", QP, 2 * QP, 2 * QP, fplan.swap, seeds[0], signs[0],
                seeds[1], signs[1], s0)
        log.add("es_f8restore", "fp8", QP, 2 * QP, QP, fplan.restore, seeds[1], signs[1], s0)
    log.add(f"es_f8update (N={N})", "fp8", QP, 2 * QP, nd * QP, fplan.update, seeds, signs,
            rewards, W.alpha, sigma=s0, round_seed=1, repeat=R)
    torch.cuda.synchronize()
    fplan.close()
    del fflat, fviews, fscales
    torch.cuda.empty_cache()

    cal = torch.empty(16 << 30, dtype=torch.uint8, device="cuda")
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    B = cal.numel()
    for pol, pname in ((0, "nontemporal"), (esopt.CALIBRATE_TEMPORAL, "ordinary")):
        for mode, mname, factor in ((esopt.CALIBRATE_READ, "read", 1),
                                    (esopt.CALIBRATE_WRITE, "write", 1),
                                    (esopt.CALIBRATE_READ_WRITE, "in-place", 2)):
            log.add(f"es_hbm_calibrate {mname}, {pname} accesses (16 GiB)", "ceiling", 0,
                    factor * B, 0, esopt.hbm_calibrate, cal, mode | pol, sink, repeat=R)
    torch.cuda.synchronize()
    del cal
    torch.cuda.empty_cache()
    calibration_copy(torch)
    torch.cuda.synchronize()
    log.write({"workload": W.name, "params": P, "members": N, "distinct_seeds": nd,
               "source_hash": _kernel_source_hash(),
               "pass_args": "--profile-pass" + ("" if args.workload == "dense-27b"
                                                 else f" --workload {args.workload}")})
    print(json.dumps({"profile_pass": W.name, "launches": len(log.rows)}))


def _library_dispatches(rows, name_key, id_key):
    """Library-kernel dispatches of one run in dispatch order, one entry per
    dispatch: (dispatch id, kernel name, row or rows)."""
    by_id = {}
    for r in rows:
        name = r[name_key]
        if any(k in name for k in LIBRARY_KERNELS):
            by_id.setdefault(int(r[id_key]), (name, []))[1].append(r)
    return [(i, by_id[i][0], by_id[i][1]) for i in sorted(by_id)]


def _read_csv(d, suffix):
    """The rows of the one *suffix (or *suffix.gz) file under d."""
    import csv
    import glob
    import gzip
    files = (glob.glob(os.path.join(d, "**", f"*{suffix}"), recursive=True)
             + glob.glob(os.path.join(d, "**", f"*{suffix}.gz"), recursive=True))
    if not files:
        raise FileNotFoundError(f"no *{suffix} under {d}")
    path = max(files, key=os.path.getmtime)          # the latest run's file
    opener = gzip.open if path.endswith(".gz") else open
    with opener(path, "rt", newline="") as fh:
        return list(csv.DictReader(fh))


def _labels(d):
    with open(os.path.join(d, "labels.json")) as fh:
        return json.load(fh)


def _match(labels, dispatches, what):
    if len(labels["launches"]) != len(dispatches):
        raise RuntimeError(f"{what}: {len(labels['launches'])} labelled launches but "
                           f"{len(dispatches)} library-kernel dispatches")
    return list(zip(labels["launches"], dispatches))


def summarize(out_dir, profiles_dir=os.path.join(REPO, "profiles")):
    """Turn the trace and counter runs of one profile pass (out_dir/trace,
    out_dir/fetch, out_dir/write, out_dir/valu) into summaries and
    counters.json entries under profiles_dir."""
    lab = _labels(os.path.join(out_dir, "trace"))
    if "sweep" in lab:
        return summarize_sweep(out_dir, lab, profiles_dir)
    per = _per_label(out_dir)
    src = lab["source_hash"]
    if src != _kernel_source_hash():
        raise RuntimeError("profile taken on other kernel sources than the working tree's")
    wname, P = lab["workload"], lab["params"]
    cmds = profile_commands(lab["pass_args"])
    header = ["Commands (from the repository root on an MI355X machine, after "
              "`cd /tmp && export TMPDIR=/tmp`; `<out>` is an output directory; then "
              f"`python3 bench.py --summarize <out>`):", ""] + [f"* `{c}`" for c in cmds] + [
        "", f"Kernel-sources hash: `{src}`", "", CALIBRATION_NOTE.format(**per["_calibration"]), ""]
    groups = {
        "perturb": ("es_perturb", f"es_perturb / es_restore on {wname} ({P:,} bf16 parameters)"),
        "swap": ("es_swap", f"es_swap on {wname} ({P:,} bf16 parameters)"),
        "update": ("es_update", f"es_update on {wname} ({P:,} bf16 parameters, "
                                f"N = {lab['members']}, {lab['distinct_seeds']} distinct seeds)"),
        "int8": ("es_qpass", f"int8 passes on {wname}-int8 (the same shapes as int8 codes with "
                             f"per-row scales)"),
        "fp8": ("es_qpass", f"fp8 passes on {wname}-fp8 (the same shapes as E4M3 codes with "
                            f"per-row scales)"),
        "ceiling": ("hbm_ceilings", f"HBM ceilings: the in-place stream over the {wname} plan and "
                                    f"the flat-buffer calibration passes"),
        "checksum": ("es_plan_checksum", f"es_plan_checksum on {wname}"),
        "blocks": ("es_blocks", f"Column blocks of {wname}'s matrices (es_plan_create_blocks: "
                                f"each matrix as 8 blocks of rows x cols/8, the strided launch "
                                f"with row maps)"),
    }
    counters_path = os.path.join(profiles_dir, "counters.json")
    counters = json.load(open(counters_path)) if os.path.exists(counters_path) else {}
    keys = {"es_perturb": "es_perturb", f"es_update (N={lab['members']}, nearest-even)": "es_update",
            "es_swap (two keys)": "es_swap", "es_qperturb": "es_qperturb",
            f"es_qupdate (N={lab['members']})": "es_qupdate", "es_f8perturb": "es_f8perturb",
            f"es_f8update (N={lab['members']})": "es_f8update", "es_qswap": "es_qswap",
            "es_f8swap": "es_f8swap",
            f"es_update (N={lab['members']}, binary32 masters)": "es_update_master",
            "es_perturb_master (a member from binary32 masters)": "es_perturb_master"}
    for group, (stem, title) in groups.items():
        rows = [r for r in per["_rows"] if r["group"] == group]
        if not rows:
            continue
        lines = [f"# {title}", ""] + header + _table(rows)
        suffix = {"int8": "-int8", "fp8": "-fp8"}.get(group, "")
        fname = f"{stem}_{wname}{suffix}.md"
        with open(os.path.join(profiles_dir, fname), "w") as fh:
            fh.write("\n".join(lines) + "\n")
        for r in rows:
            k = keys.get(r["label"])
            if k:
                counters[k] = {"source_hash": src,
                               "workload": wname + suffix,
                               "params": r["params"], "bytes_per_launch": r["fetch"] + r["write"],
                               "fetch_bytes": r["fetch"], "write_bytes": r["write"],
                               "valu_insts_per_launch": r["SQ_INSTS_VALU"], "avg_ns": r["ns"],
                               "counters": {c: r[c] for c in VALU_COUNTERS}}
    with open(counters_path, "w") as fh:
        json.dump(counters, fh, indent=1)
    print(json.dumps({k: v["bytes_per_launch"] for k, v in counters.items()}))


VALU_COUNTERS = ("SQ_INSTS_VALU", "SQ_ACTIVE_INST_VALU", "SQ_INSTS_VALU_TRANS_F32", "SQ_WAVES",
                 "SQ_BUSY_CYCLES", "GRBM_GUI_ACTIVE")
CALIBRATION_NOTE = ("Counter calibration: a plain {copy_bytes} B device copy read {f_copy:.0f} B by "
                    "FETCH_SIZE and {w_copy:.0f} B by WRITE_SIZE (KiB counters x 1024), so fetched "
                    "bytes are FETCH_SIZE x 1024 x {f_scale:.3f} and written bytes WRITE_SIZE x "
                    "1024 x {w_scale:.3f}.  Durations are the kernel trace's; the shader clock is "
                    "GRBM_GUI_ACTIVE / 8 XCDs over the duration of the same dispatch in the counter "
                    "run; VALU issue is SQ_INSTS_VALU x 64 lanes over the trace duration against "
                    "39.32 T lane-instructions/s (256 CUs x 64 lanes x 2.4 GHz), and per cycle "
                    "against one wave instruction per CU per cycle at the measured clock.")


def _per_label(out_dir):
    """Join the four runs on the labels: per labelled launch the trace
    duration, scaled fetch / write bytes and the VALU counters."""
    res = {}
    trace_lab = _labels(os.path.join(out_dir, "trace"))
    tr = _library_dispatches(_read_csv(os.path.join(out_dir, "trace"), "kernel_trace.csv"),
                             "Kernel_Name", "Dispatch_Id")
    runs = {}
    for run in COUNTER_SETS:
        d = os.path.join(out_dir, run)
        rows = _read_csv(d, "counter_collection.csv")
        runs[run] = (_labels(d), _library_dispatches(rows, "Kernel_Name", "Dispatch_Id"), rows)
    # calibration from the largest device copy of the fetch / write runs
    def copy_max(rows, counter):
        return max(float(r["Counter_Value"]) for r in rows
                   if "copyBuffer" in r["Kernel_Name"] and r["Counter_Name"] == counter) * 1024
    f_copy = copy_max(runs["fetch"][2], "FETCH_SIZE")
    w_copy = copy_max(runs["write"][2], "WRITE_SIZE")
    cal = {"copy_bytes": CALIBRATION_COPY_BYTES, "f_copy": f_copy, "w_copy": w_copy,
           "f_scale": CALIBRATION_COPY_BYTES / f_copy, "w_scale": CALIBRATION_COPY_BYTES / w_copy}
    out = []
    agg = {}
    for l, (i, name, r) in _match(trace_lab, tr, "trace"):
        ns = int(r[0]["End_Timestamp"]) - int(r[0]["Start_Timestamp"])
        agg.setdefault(l["label"], {**l, "kernel": name, "ns_list": []})["ns_list"].append(ns)
    for run, (labs, disp, _) in runs.items():
        for l, (i, name, rs) in _match(labs, disp, run):
            e = agg[l["label"]]
            for r in rs:
                e.setdefault(r["Counter_Name"] + "_list", []).append(float(r["Counter_Value"]))
            if run == "valu":
                e.setdefault("valu_ns_list", []).append(
                    int(rs[0]["End_Timestamp"]) - int(rs[0]["Start_Timestamp"]))
    for label, e in agg.items():
        e["ns"] = float(np.mean(e["ns_list"]))
        e["fetch"] = float(np.mean(e["FETCH_SIZE_list"])) * 1024 * cal["f_scale"]
        e["write"] = float(np.mean(e["WRITE_SIZE_list"])) * 1024 * cal["w_scale"]
        for c in VALU_COUNTERS:
            e[c] = float(np.mean(e[c + "_list"]))
        e["valu_ns"] = float(np.mean(e["valu_ns_list"]))
        out.append(e)
    res["_rows"] = out
    res["_calibration"] = cal
    return res


def _table(rows):
    lines = ["| launch | kernel | calls | trace ns | algorithmic GB/s | fetched B | written B | "
             "counted / algorithmic bytes | B per param | VALU instr per param | per normal | "
             "of which transcendental (per param) | VALU issue (of 39.32 T/s) | shader clock GHz | "
             "VALU issue per CU-cycle at that clock |",
             "|---|---|---|---|---|---|---|---|---|---|---|---|---|---|---|"]
    for e in rows:
        P, ns = e["params"], e["ns"]
        vi = e["SQ_INSTS_VALU"]
        clock = e["GRBM_GUI_ACTIVE"] / 8 / e["valu_ns"]
        kname = _short_name(e["kernel"])
        tot = e["fetch"] + e["write"]
        lines.append(
            f"| {e['label']} | `{kname}` | {len(e['ns_list'])} | {ns:.0f} | "
            f"{e['algorithmic_bytes'] / ns:.1f} | {e['fetch']:.4e} | {e['write']:.4e} | "
            f"{tot / e['algorithmic_bytes']:.4f} | "
            + (f"{tot / P:.3f} | {vi * 64 / P:.2f} | " if P else "— | — | ")
            + (f"{vi * 64 / e['normals']:.2f} | " if e["normals"] else "— | ")
            + (f"{e['SQ_INSTS_VALU_TRANS_F32'] * 64 / P:.2f} | " if P else "— | ")
            + f"{vi * 64 / (ns * 1e-9) / 1e12 / VALU_PEAK_TINST:.3f} | {clock:.3f} | "
            f"{vi / (256 * e['GRBM_GUI_ACTIVE'] / 8):.3f} |")
    lines += ["", "Raw counters per launch (means over the launches of each label):", ""]
    for e in rows:
        lines.append(f"* {e['label']}: " + ", ".join(f"{c} {e[c]:.4e}" for c in VALU_COUNTERS)
                     + f"; counter-run duration {e['valu_ns']:.0f} ns")
    return lines


def summarize_sweep(out_dir, lab, profiles_dir):
    """profiles/es_update_<workload>-sweep.md from a sweep profile pass."""
    per = _per_label(out_dir)
    src = lab["source_hash"]
    if src != _kernel_source_hash():
        raise RuntimeError("profile taken on other kernel sources than the working tree's")
    cmds = profile_commands(lab["pass_args"])
    rows = sorted((e for e in per["_rows"] if e["group"] != "warmup"), key=lambda e: e["members"])
    lines = [f"# Fused es_update population sweep on {lab['workload']} ({lab['params']:,} bf16 "
             f"parameters, rewards N(0,1), distinct seeds)", "",
             "Commands (from the repository root on an MI355X machine, after "
             "`cd /tmp && export TMPDIR=/tmp`; `<out>` is an output directory; then "
             "`python3 bench.py --summarize <out>`):", ""] + [f"* `{c}`" for c in cmds] + [
        "", f"Kernel-sources hash: `{src}`", "", CALIBRATION_NOTE.format(**per["_calibration"]), "",
        "| N | trace ms | algorithmic TB/s | B per param (counted) | VALU instr per param | "
        "VALU instr per normal | VALU issue (of 39.32 T/s) | shader clock GHz | VALU issue per "
        "CU-cycle | bound |",
        "|---|---|---|---|---|---|---|---|---|---|"]
    stream = [e for e in rows if e["group"] == "ceiling"]
    t_stream = stream[0]["ns"] if stream else None
    for e in rows:
        if e["group"] != "update":
            continue
        P, ns, vi = e["params"], e["ns"], e["SQ_INSTS_VALU"]
        clock = e["GRBM_GUI_ACTIVE"] / 8 / e["valu_ns"]
        issue = vi * 64 / (ns * 1e-9) / 1e12 / VALU_PEAK_TINST
        bound = "hbm" if t_stream and ns < 1.5 * t_stream else "valu"
        lines.append(f"| {e['members']} | {ns / 1e6:.3f} | {4 * P / ns / 1e3:.3f} | "
                     f"{(e['fetch'] + e['write']) / P:.3f} | {vi * 64 / P:.1f} | "
                     f"{vi * 64 / e['normals']:.2f} | {issue:.3f} | {clock:.3f} | "
                     f"{vi / (256 * e['GRBM_GUI_ACTIVE'] / 8):.3f} | {bound} |")
    if stream:
        s = stream[0]
        lines += ["", f"In-place copy of the same memory (es_stream_pass): {s['ns'] / 1e6:.3f} ms, "
                      f"{4 * s['params'] / s['ns'] / 1e3:.3f} TB/s, "
                      f"{(s['fetch'] + s['write']) / s['params']:.3f} B per param counted; "
                      "'bound' is hbm where the update takes under 1.5x this time."]
    lines += [""] + _table(rows)[-len(rows) - 3:]
    path = os.path.join(profiles_dir, f"es_update_{lab['workload']}-sweep.md")
    with open(path, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print(path)


def _short_name(name, width=90):
    """A kernel's name without return type, anonymous namespace and
    argument list, cut to `width` characters."""
    n = name.replace("(anonymous namespace)::", "")
    if n.startswith("void "):
        n = n[5:]
    n = n.split("(")[0]
    return n if len(n) <= width else n[:width - 3] + "..."


BENCH_TRACE_COMMAND = ("rocprofv3 --kernel-trace --stats -f csv -d <out> -o bench -- python3 "
                       "bench.py --steps 2 --warmup 1 --no-cpu-baseline")


def summarize_bench_trace(trace_dir, profiles_dir=os.path.join(REPO, "profiles"),
                          workload="dense-27b", master=False):
    """profiles/bench_kernel_stats_<workload>.md: the --stats table of a
    kernel trace of the default bench command (every kernel the timed step,
    the swap walk and the ceiling passes launch); with master, of the
    command with --master (..._<workload>-master.md)."""
    stats = _read_csv(trace_dir, "kernel_stats.csv")
    cmd = BENCH_TRACE_COMMAND + (" --master" if master else "")
    what = "the benchmark command" + (" with binary32 masters" if master else "")
    lines = [f"# Kernel statistics of {what} on {workload}", "",
             "Command (from the repository root on an MI355X machine, after "
             "`cd /tmp && export TMPDIR=/tmp`; `<out>` is an output directory; then "
             f"`python3 bench.py --summarize-trace <out>{' --master' if master else ''}`):", "",
             f"* `{cmd}`", "", f"Kernel-sources hash: `{_kernel_source_hash()}`",
             "", "| kernel | calls | average ns | min ns | max ns | share of GPU time |",
             "|---|---|---|---|---|---|"]
    for r in stats:
        name = _short_name(r["Name"])
        lines.append(f"| `{name}` | {r['Calls']} | {float(r['AverageNs']):.0f} | {r['MinNs']} | "
                     f"{r['MaxNs']} | {float(r['Percentage']):.2f} % |")
    path = os.path.join(profiles_dir,
                        f"bench_kernel_stats_{workload}{'-master' if master else ''}.md")
    with open(path, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print(path)


def _counters_for(path, kind, label):
    """The counter entry of a kernel if it was taken on these kernel sources
    and this workload, else None."""
    if not os.path.exists(path):
        return None
    e = json.load(open(path)).get(kind)
    if isinstance(e, dict) and e.get("source_hash") == _kernel_source_hash() and e.get("workload") == label:
        return e
    return None


def _kernel_source_hash():
    """Hash of the device code the counters describe: the device headers and
    the device section of esopt.hip (host-side edits leave the kernels, and so
    the counters, unchanged)."""
    import hashlib
    csrc = os.path.join(REPO, "paper_2608_17310_amd", "csrc")
    h = hashlib.sha256()
    for f in sorted(x for x in os.listdir(csrc) if x.endswith(".hpp")):
        h.update(open(os.path.join(csrc, f), "rb").read())
    src = open(os.path.join(csrc, "esopt.hip"), "rb").read()
    start, end = src.index(b"// Device code"), src.index(b"// Host side")
    h.update(src[start:end])
    return h.hexdigest()[:16]


if __name__ == "__main__":
    main()
