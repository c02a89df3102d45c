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
    ap.add_argument("--swap", action="store_true",
                    help="move between members with the fused es_swap (N+1 passes per step)")
    ap.add_argument("--sweep-members", default=None, metavar="N1,N2,...",
                    help="large-population sweep of the fused update on the 4B-shaped set "
                         "(one JSON line per N)")
    ap.add_argument("--int8", action="store_true",
                    help="the int8 path: codes with per-row scales, es_qperturb / es_qrestore / "
                         "es_qupdate")
    ap.add_argument("--stochastic-round", action="store_true",
                    help="round the update stochastically (ES_UPDATE_STOCHASTIC_ROUND)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="target CPU time of the oracle baseline sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--profile-pass", action="store_true",
                    help="run one perturb, one update and a calibration copy, for rocprofv3")
    ap.add_argument("--counters-json", default=os.path.join(REPO, "profiles", "counters.json"),
                    help="per-launch counter values measured with rocprofv3 (see --summarize)")
    ap.add_argument("--summarize", nargs=4, metavar=("TRACE_DIR", "FETCH_DIR", "WRITE_DIR", "VALU_DIR"),
                    help="turn rocprofv3 CSV output of the profiling runs into profiles/")
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


def sigma_at(W, t):
    if W.sigma0 == W.sigma_T:
        return W.sigma0
    return W.sigma_T + (W.sigma0 - W.sigma_T) * (1 + math.cos(math.pi * (t % W.T) / W.T)) / 2


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
    """The host's CPU model (from /proc/cpuinfo) and logical CPU count."""
    model = None
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"cpu_model": model, "host_logical_cpus": os.cpu_count()}


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
    """The oracle's work of one int8 step on a sample of one tensor's codes."""
    import oracle
    q, scales, row, tid, elems, seeds, signs, rewards, alpha, sigma = args
    t0 = time.perf_counter()
    for s, sg in zip(seeds, signs):
        p = oracle.qperturb(q, scales, row, s, tid, sg, sigma, elems=elems)
        q = oracle.qrestore(p, scales, row, s, tid, sg, sigma, elems=elems)
    q, _ = oracle.qupdate(q, scales, row, tid, seeds, signs, rewards, alpha, sigma, elems=elems,
                          round_seed=1)
    return time.perf_counter() - t0


def cpu_baseline_int8(W, seeds, signs, rewards, sigma, workers, budget_s, per_tensor=1 << 14):
    """The oracle's int8 step on a bounded sample: random codes and indices,
    per-row scales of the workload's shapes (values do not change the cost)."""
    from paper_2608_17310_amd import workloads as wl
    rng = np.random.default_rng(0)
    samples = []
    for tid, (n, shape) in enumerate(zip(W.numels, W.shapes)):
        row = wl.row_of(shape)
        idx = np.unique(rng.integers(0, n, size=min(n, per_tensor))).astype(np.uint64)
        scales = rng.uniform(3e-4, 1e-3, 1 if row == 0 else n // row).astype(np.float32)
        codes = rng.integers(-127, 128, size=idx.size).astype(np.int8)
        samples.append((codes, scales, row, tid, idx))
    n = len(seeds)
    c0 = samples[0]
    t_small = _oracle_qchunk((c0[0][:1024], c0[1], c0[2], c0[3], c0[4][:1024], seeds, signs,
                              rewards, W.alpha, sigma))
    per_elem = t_small / 1024
    total = sum(x[4].size for x in samples)
    frac = min(1.0, int(budget_s * workers / per_elem) / total)
    jobs = []
    for codes, scales, row, tid, idx in samples:
        k = max(1, int(idx.size * frac))
        jobs.append((codes[:k], scales, row, tid, idx[:k], seeds, signs, rewards, W.alpha, sigma))
    n_elems = sum(j[4].size for j in jobs)
    t0 = time.perf_counter()
    with mp.get_context("fork").Pool(workers) as pool:
        pool.map(_oracle_qchunk, jobs, chunksize=1)
    wall = time.perf_counter() - t0
    rate = (2 * n + 1) * n_elems / wall
    return {"value": rate, "unit": "params/s", "cores": workers, "kind": "oracle",
            **host_cpu(),
            "full_step_s_extrapolated": round((2 * n + 1) * W.n_params / rate, 1),
            "sample": f"{n_elems} int8 codes sampled across {len(jobs)} tensors of {W.name}, one "
                      f"full int8 step (N={n}: {2 * n} perturb/restore + 1 update) in fp64 NumPy "
                      f"over {workers} worker processes, {wall:.1f} s wall"}


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


def run_int8(args):
    """The int8 step on the workload's shapes: N x (es_qperturb + es_qrestore)
    + es_qupdate over codes with per-row scales, inputs resident in HBM."""
    import torch
    from paper_2608_17310_amd import esopt, workloads as wl
    W = wl.WORKLOADS[args.workload]
    n_members = args.members
    signs = list(W.signs) if n_members is None else [1] * n_members
    N = len(signs)
    cpu = None
    if not args.no_cpu_baseline and not args.profile_pass:
        cpu = cpu_baseline_int8(W, step_seeds(W, args.warmup, n_members), signs,
                                wl.rewards(W, args.warmup, n=N), sigma_at(W, args.warmup),
                                min(16, os.cpu_count() or 1), args.cpu_seconds)
    if not torch.cuda.is_available():
        print(json.dumps({"error": "no GPU"}))
        sys.exit(1)
    torch.cuda.set_device(0)
    flat, views, scales, rows = wl.device_qparams(W)
    plan = esopt.QPlan(views, scales, rows)
    P = plan.numel
    stream = torch.cuda.current_stream()
    total_steps = args.warmup + args.steps
    rewards_np = np.stack([wl.rewards(W, t, n=N) for t in range(total_steps)])
    rewards_all = torch.from_numpy(rewards_np).cuda()
    torch.cuda.synchronize()
    if args.profile_pass:
        seeds = step_seeds(W, 0, n_members)
        plan.perturb(seeds[0], signs[0], W.sigma0)
        plan.restore(seeds[0], signs[0], W.sigma0)
        plan.update(seeds, signs, rewards_all[0], W.alpha, sigma=W.sigma0, round_seed=1)
        calib = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")     # 1 GiB copy
        torch.empty_like(calib).copy_(calib)
        torch.cuda.synchronize()
        print(json.dumps({"profile_pass": W.name + "-int8", "params": P, "members": N,
                          "calibration_copy_bytes": 1 << 30}))
        return
    ev = []

    def timed(kind, record, fn, *a, **kw):
        if record:
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            fn(*a, **kw)
            e1.record(stream)
            ev.append((kind, e0, e1))
        else:
            fn(*a, **kw)

    def run_step(t, record):
        seeds = step_seeds(W, t, n_members)
        sigma = sigma_at(W, t)
        for sd, sg in zip(seeds, signs):
            timed("es_qperturb", record, plan.perturb, sd, sg, sigma)
            timed("es_qrestore", record, plan.restore, sd, sg, sigma)
        timed("es_qupdate", record, plan.update, seeds, signs, rewards_all[t], W.alpha,
              sigma=sigma, round_seed=1000 + t)

    for t in range(args.warmup):
        run_step(t, record=False)
    torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    # no garbage-collector pause inside the timed region (one measured 35 ms
    # on a small set, where the GPU waits on the host)
    gc.collect()
    gc.disable()
    t_wall0 = time.perf_counter()
    start.record(stream)
    for t in range(args.warmup, total_steps):
        run_step(t, record=True)
    end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_wall0
    gc.enable()
    ms_step = start.elapsed_time(end) / args.steps
    per = {}
    for kind, a, b in ev:
        per.setdefault(kind, []).append(a.elapsed_time(b))
    t_pert = float(np.mean(per["es_qperturb"] + per["es_qrestore"])) / 1e3
    t_upd = float(np.mean(per["es_qupdate"])) / 1e3
    value = (2 * N + 1) * P / (ms_step / 1e3)
    n_distinct = len(dict.fromkeys(step_seeds(W, 0, n_members)))
    n_live = float(np.mean([live_seeds(step_seeds(W, t, n_members), signs, rewards_np[t])
                            for t in range(args.warmup, total_steps)]))
    label = W.name + "-int8"
    c_pert = _counters_for(args.counters_json, "es_qperturb", label)
    c_upd = _counters_for(args.counters_json, "es_qupdate", label)

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
        "metric": "params/s of the int8 ES step (es_qperturb/es_qrestore and fused es_qupdate, "
                  "N members)",
        "value": value, "unit": "params/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_step, 3), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32", "param_dtype": "int8",
        "data": "synthetic",
        "config": {"workload": label, "params": P, "tensors": len(views), "members": N,
                   "param_bytes": P + 4 * sum(int(x.numel()) for x in scales),
                   "plan_device_bytes": plan.device_bytes,
                   "distinct_seeds": n_distinct, "sigma0": W.sigma0, "alpha": W.alpha,
                   "scales": "one binary32 scale per row of the last dimension, one per vector",
                   "counting": "value = (2N+1) P / step time: 2N perturb/restore passes and one "
                               "fused N-member update pass per step"},
        "roofline": alu_roofline(c_pert, t_pert, "es_qpass_kernel (es_qperturb / es_qrestore)", True),
        "roofline_update": alu_roofline(c_upd, t_upd, "es_qpass_kernel (es_qupdate)", same_config),
        "per_kernel": {
            "es_qperturb": {"ms": round(t_pert * 1e3, 3), "params_per_s": P / t_pert,
                            "GBps_algorithmic": round(2 * P / t_pert / 1e9, 1)},
            "es_qupdate": {"ms": round(t_upd * 1e3, 3), "params_per_s": P / t_upd,
                           "normals_per_s": n_live * P / t_upd,
                           "distinct_seeds": n_distinct, "live_seeds": round(n_live, 3)}},
        "wall_s_timed": round(wall, 3),
        "cpu_baseline": cpu,
    }
    print(json.dumps(out))
    plan.close()


def main():
    args = parse()
    if args.summarize:
        summarize(*args.summarize, workload=args.workload, int8=args.int8)
        return
    if args.gpus != 1:
        print(json.dumps({"error": "the ES parameter path runs on one GPU; --gpus above 1 is "
                                   "not supported (population parallelism across GPUs is not "
                                   "implemented)"}))
        sys.exit(2)
    if args.sweep_members:
        return run_sweep(args)
    if args.int8:
        return run_int8(args)
    import torch
    from paper_2608_17310_amd import esopt, workloads as wl

    W = wl.WORKLOADS[args.workload]
    n_members = args.members
    signs = list(W.signs) if n_members is None else [1] * n_members
    N = len(signs)
    cpu = None
    if not args.no_cpu_baseline and not args.profile_pass:
        # before the GPU is touched: worker processes fork from a clean parent
        cpu = cpu_baseline(W, step_seeds(W, args.warmup, n_members), signs,
                           wl.rewards(W, args.warmup, n=N), sigma_at(W, args.warmup),
                           host_samples(W), min(16, os.cpu_count() or 1), args.cpu_seconds)

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

    if args.profile_pass:
        seeds = step_seeds(W, 0, n_members)
        plan.perturb(seeds[0], signs[0], W.sigma0)
        plan.restore(seeds[0], signs[0], W.sigma0)
        plan.update(seeds, signs, rewards_all[0], W.alpha, sigma=W.sigma0)
        calib = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")     # 1 GiB copy
        calib2 = torch.empty_like(calib)
        calib2.copy_(calib)
        torch.cuda.synchronize()
        print(json.dumps({"profile_pass": W.name, "params": P, "members": N,
                          "calibration_copy_bytes": 1 << 30}))
        return

    ev = []   # (kind, start, end) event pairs inside the timed region
    update_flags = esopt.ES_UPDATE_STOCHASTIC_ROUND if args.stochastic_round else 0

    def timed_call(kind, record, fn, *a):
        if record:
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            fn(*a)
            e1.record(stream)
            ev.append((kind, e0, e1))
        else:
            fn(*a)

    def run_step(t, record):
        seeds = step_seeds(W, t, n_members)
        sigma = sigma_at(W, t)
        if args.swap:
            timed_call("es_perturb", record, plan.perturb, seeds[0], signs[0], sigma)
            for i in range(N - 1):
                timed_call("es_swap", record, plan.swap, seeds[i], signs[i], seeds[i + 1],
                           signs[i + 1], sigma)
            timed_call("es_restore", record, plan.restore, seeds[-1], signs[-1], sigma)
        else:
            for s, sg in zip(seeds, signs):
                timed_call("es_perturb", record, plan.perturb, s, sg, sigma)
                timed_call("es_restore", record, plan.restore, s, sg, sigma)
        if record:
            a = torch.cuda.Event(enable_timing=True)
            b = torch.cuda.Event(enable_timing=True)
            a.record(stream)
        plan.update(seeds, signs, rewards_all[t], W.alpha, sigma=sigma, flags=update_flags,
                    round_seed=1000 + t)
        if record:
            b.record(stream)
            ev.append(("es_update", a, b))

    for t in range(args.warmup):
        run_step(t, record=False)
    torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    # no garbage-collector pause inside the timed region (one measured 35 ms
    # on a small set, where the GPU waits on the host)
    gc.collect()
    gc.disable()
    t_wall0 = time.perf_counter()
    start.record(stream)
    for t in range(args.warmup, total_steps):
        run_step(t, record=True)
    end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_wall0
    gc.enable()
    ms_total = start.elapsed_time(end)
    ms_step = ms_total / args.steps
    per = {}
    for kind, a, b in ev:
        per.setdefault(kind, []).append(a.elapsed_time(b))
    t_pert = float(np.mean(per["es_perturb"] + per["es_restore"])) / 1e3
    t_upd = float(np.mean(per["es_update"])) / 1e3
    passes = (N + 2) if args.swap else (2 * N + 1)
    value = passes * P / (ms_step / 1e3)
    n_distinct = len(dict.fromkeys(step_seeds(W, 0, n_members)))
    n_live = float(np.mean([live_seeds(step_seeds(W, t, n_members), signs, rewards_np[t])
                            for t in range(args.warmup, total_steps)]))

    # the practical in-place streaming ceiling over the same memory: the same
    # tiles and launch, loads and stores only, not pipelined (es_stream_pass),
    # timed after the step
    plan.stream_pass()
    ts = []
    for _ in range(3):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        plan.stream_pass()
        e1.record(stream)
        e1.synchronize()
        ts.append(e0.elapsed_time(e1))
    ceiling_gbs = 4 * P / (float(np.median(ts)) / 1e3) / 1e9
    flat_rates = flat_ceilings(esopt, stream)
    c_pert = _counters_for(args.counters_json, "es_perturb", W.name)
    c_upd = _counters_for(args.counters_json, "es_update", W.name)
    traffic = c_pert["bytes_per_launch"] if c_pert else None
    perturb_gbs = 4 * P / t_pert / 1e9
    roofline = {"bound": "hbm", "achieved": round(perturb_gbs, 1), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(perturb_gbs / HBM_PEAK_GBS, 4),
                "traffic": traffic, "kernel": "es_perturb_kernel (es_perturb / es_restore)",
                "algorithmic_bytes_per_launch": 4 * P,
                "ceiling": {"GBps": round(ceiling_gbs, 1),
                            "frac_of_ceiling": round(perturb_gbs / ceiling_gbs, 4),
                            "kernel": "es_stream_kernel: in-place copy of every parameter, same tiles (es_stream_pass)"},
                "flat_buffer_ceilings": flat_rates}
    update = {"ms": round(t_upd * 1e3, 3), "params_per_s": P / t_upd,
              "GBps_algorithmic": round(4 * P / t_upd / 1e9, 1),
              "normals_per_s": n_live * P / t_upd, "distinct_seeds": n_distinct,
              "live_seeds": round(n_live, 3)}
    # The update is VALU-bound: its roofline is the VALU issue rate.  The
    # instruction count per launch is a counter measurement (SQ_INSTS_VALU,
    # same workload and kernel sources); the duration is live.
    roofline_update = {"bound": "alu", "unit": "T lane-instr/s", "peak": round(VALU_PEAK_TINST, 2),
                       "achieved": None, "frac": None,
                       "kernel": "es_update_kernel (fused N-member update)",
                       "traffic": c_upd["bytes_per_launch"] if c_upd else None}
    if c_upd and N == len(W.seeds) and n_members is None and not args.stochastic_round:
        ach = c_upd["valu_insts_per_launch"] * 64 / t_upd / 1e12
        roofline_update.update(achieved=round(ach, 2), frac=round(ach / VALU_PEAK_TINST, 4))
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
                   "member_moves": "es_swap" if args.swap else "es_perturb/es_restore",
                   "update_rounding": "stochastic" if args.stochastic_round else "nearest-even",
                   "counting": ("value = (N+2) P / step time: perturb, N-1 fused swaps, restore "
                                "and one fused N-member update pass per step") if args.swap else
                               ("value = (2N+1) P / step time: 2N perturb/restore passes "
                                "and one fused N-member update pass per step")},
        "roofline": roofline,
        "roofline_update": roofline_update,
        "per_kernel": {
            "es_perturb": {"ms": round(t_pert * 1e3, 3), "params_per_s": P / t_pert,
                           "GBps_algorithmic": round(perturb_gbs, 1),
                           "frac_hbm_peak": round(perturb_gbs / HBM_PEAK_GBS, 4)},
            "es_update": update,
            **({"es_swap": {"ms": round(float(np.mean(per["es_swap"])), 3),
                            "params_per_s": P / (float(np.mean(per["es_swap"])) / 1e3),
                            "GBps_algorithmic": round(4 * P / (float(np.mean(per["es_swap"])) / 1e3) / 1e9, 1)}}
               if "es_swap" in per else {}),
        },
        "wall_s_timed": round(wall, 3),
    }
    if cpu is not None:
        out["cpu_baseline"] = cpu
    plan.close()
    print(json.dumps(out))


# ------------------------------------------------------------ profiling --

PROFILE_COMMANDS = {
    "trace": "rocprofv3 --kernel-trace --stats -f csv -d <out>/trace -o trace -- "
             "python3 bench.py --steps 2 --warmup 1 --no-cpu-baseline",
    "fetch": "rocprofv3 --pmc FETCH_SIZE -f csv -d <out>/fetch -o fetch -- "
             "python3 bench.py --profile-pass",
    "write": "rocprofv3 --pmc WRITE_SIZE -f csv -d <out>/write -o write -- "
             "python3 bench.py --profile-pass",
    "valu": "rocprofv3 --pmc SQ_INSTS_VALU SQ_ACTIVE_INST_VALU SQ_INSTS_VALU_TRANS_F32 SQ_WAVES "
            "SQ_BUSY_CYCLES GRBM_GUI_ACTIVE -f csv -d <out>/valu -o valu -- "
            "python3 bench.py --profile-pass",
}


def _kind(name):
    if "es_qpass_kernel" in name:
        if "true, false>" in name:
            return "es_qupdate"
        if "false, true>" in name:
            return "es_qrestore"
        return "es_qperturb"
    if "es_perturb_kernel" in name:
        return "es_perturb"
    if "es_update_kernel" in name:
        return "es_update"
    if "copyBuffer" in name:
        return "copy"
    return None


def _counter_rows(d):
    import csv
    import glob
    f = glob.glob(os.path.join(d, "*counter_collection.csv"))[0]
    out = {}
    for r in csv.DictReader(open(f)):
        k = _kind(r["Kernel_Name"])
        if k:
            out.setdefault((k, r["Counter_Name"]), []).append(float(r["Counter_Value"]))
    return out


def summarize(trace_dir, fetch_dir, write_dir, valu_dir, workload, int8=False):
    """Write profiles/<kernel>_<workload>.md and merge the kernels' entries
    into profiles/counters.json from the CSV output of the four rocprofv3 runs
    in PROFILE_COMMANDS (with --int8 added for the int8 path)."""
    import csv
    import glob
    stats = list(csv.DictReader(open(glob.glob(os.path.join(trace_dir, "*kernel_stats.csv"))[0])))
    fetch, write, valu = _counter_rows(fetch_dir), _counter_rows(write_dir), _counter_rows(valu_dir)
    # calibration: the largest copyBuffer dispatch of the profile pass is the 1 GiB device copy
    copy_bytes = 1 << 30
    f_copy = max(fetch[("copy", "FETCH_SIZE")]) * 1024
    w_copy = max(write[("copy", "WRITE_SIZE")]) * 1024
    f_scale, w_scale = copy_bytes / f_copy, copy_bytes / w_copy
    from paper_2608_17310_amd import workloads as wl
    P = wl.WORKLOADS[workload].n_params
    label = workload + ("-int8" if int8 else "")
    bytes_per_param = 2 if int8 else 4
    dtype = "int8" if int8 else "bf16"
    path = os.path.join(REPO, "profiles", "counters.json")
    counters = json.load(open(path)) if os.path.exists(path) else {}
    counters = {k: v for k, v in counters.items() if isinstance(v, dict) and "source_hash" in v}
    suffix = " --int8" if int8 else ""
    commands = [c.replace("bench.py --", "bench.py" + suffix + " --") for c in PROFILE_COMMANDS.values()]
    for kind in (("es_qperturb", "es_qupdate") if int8 else ("es_perturb", "es_update")):
        st = [r for r in stats if _kind(r["Name"]) == kind][0]
        fb = float(np.mean(fetch[(kind, "FETCH_SIZE")])) * 1024 * f_scale
        wb = float(np.mean(write[(kind, "WRITE_SIZE")])) * 1024 * w_scale
        v = {c: float(np.mean(valu[(kind, c)])) for c in
             ("SQ_INSTS_VALU", "SQ_ACTIVE_INST_VALU", "SQ_INSTS_VALU_TRANS_F32", "SQ_WAVES",
              "SQ_BUSY_CYCLES", "GRBM_GUI_ACTIVE")}
        counters[kind] = {"source_hash": _kernel_source_hash(), "workload": label, "params": P,
                          "calibration": {"copy_bytes": copy_bytes, "fetch_scale": f_scale,
                                          "write_scale": w_scale},
                          "bytes_per_launch": fb + wb, "fetch_bytes": fb, "write_bytes": wb,
                          "valu_insts_per_launch": v["SQ_INSTS_VALU"], "counters": v,
                          "avg_ns": float(st["AverageNs"]), "calls": int(st["Calls"])}
        lines = [
            f"# {kind} on {label} ({P:,} {dtype} parameters)",
            "",
            "Commands (run from the repository root on an MI355X machine, `cd /tmp && export TMPDIR=/tmp` first; "
            "`<out>` is an output directory):",
            "",
        ] + [f"* `{c}`" for c in commands] + [
            "",
            f"Kernel-sources hash: `{_kernel_source_hash()}`",
            "",
            "## Kernel trace (--stats)",
            "",
            "| kernel | calls | average ns | min ns | max ns |",
            "|---|---|---|---|---|",
            f"| `{st['Name'][:90]}` | {st['Calls']} | {float(st['AverageNs']):.0f} | {st['MinNs']} | {st['MaxNs']} |",
            "",
            "## HBM traffic per launch (FETCH_SIZE / WRITE_SIZE, KiB counters scaled by a 1 GiB copy)",
            "",
            f"* calibration copy of {copy_bytes} B read {f_copy:.0f} B by FETCH_SIZE and {w_copy:.0f} B by "
            f"WRITE_SIZE: scale factors {f_scale:.3f} and {w_scale:.3f}",
            f"* fetched {fb:.4e} B, written {wb:.4e} B, total {fb + wb:.4e} B = {(fb + wb) / P:.3f} B per "
            f"parameter (algorithmic: {bytes_per_param})",
            "",
            "## VALU counters per launch",
            "",
        ] + [f"* {k}: {val:.4e}" for k, val in v.items()] + [
            f"* VALU instructions per parameter: {v['SQ_INSTS_VALU'] * 64 / P:.2f} (wave instructions x 64 lanes / P)",
            f"* of which transcendental: {v['SQ_INSTS_VALU_TRANS_F32'] * 64 / P:.2f}",
            f"* VALU lane-instruction rate: {v['SQ_INSTS_VALU'] * 64 / (float(st['AverageNs']) * 1e-9) / 1e12:.2f} "
            f"T/s of {VALU_PEAK_TINST:.1f} T/s peak",
            "",
        ]
        with open(os.path.join(REPO, "profiles", f"{kind}_{label}.md"), "w") as fh:
            fh.write("\n".join(lines))
    with open(path, "w") as fh:
        json.dump(counters, fh, indent=1)
    print(json.dumps({k: v["bytes_per_launch"] for k, v in counters.items()}))


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
    """Hash of the device code the counters describe: the noise, int8 and
    table-search headers and the device section of esopt.hip (host-side edits
    leave the kernels, and so the counters, unchanged)."""
    import hashlib
    csrc = os.path.join(REPO, "paper_2608_17310_amd", "csrc")
    h = hashlib.sha256()
    for f in ("es_noise.hpp", "es_quant.hpp", "es_table.hpp"):
        h.update(open(os.path.join(csrc, f), "rb").read())
    src = open(os.path.join(csrc, "esopt.hip"), "rb").read()
    start, end = src.index(b"// Device code"), src.index(b"// Host side")
    h.update(src[start:end])
    return h.hexdigest()[:16]


if __name__ == "__main__":
    main()
