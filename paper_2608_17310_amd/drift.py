"""How far in-place bf16 perturb/restore walks move the parameters.

Section 3 and Appendix D.6 of arXiv 2608.17310 apply theta + sigma eps_i in
place, evaluate, and revert by subtracting the regenerated perturbation.  With
bf16 storage the revert cannot be exact: round-to-nearest is many-to-one, so
some elements come back one bf16 step away from where they started.  This
tool measures that drift on a parameter set with no update at all: each
generation walks N members (perturb, revert; or perturb, N-1 fused swaps,
revert), and after selected generations it reports, against the starting
parameters, the fraction of elements changed, the RMS drift in units of
sigma and of the starting value's bf16 spacing, the largest drift in
spacings, and whether magnitudes shrink or grow on average (spacings are
those of the larger of the start and end values, so a start of exactly 0 is
measured on the grid where it ended).  For scale it
also prints the RMS of one update step, alpha / sqrt(G) for z-scored rewards.

    python -m paper_2608_17310_amd.drift --workload dense-4b --generations 70 --members 8

With --norms-one the norm vectors hold 1.0, as in a trained model, instead of
N(0, 0.02), and each checkpoint adds a row over those vectors alone: 1.0 is a
binade boundary of bf16 (the grid steps by 2^-7 above it and 2^-8 below), so
an element whose perturbation rounds away can come back one step below 1.

With --format int8 or --format e4m3 the same walk runs on the quantized
codes of the set (per-row scales; es_qperturb / es_qrestore), and the drift
is measured on the dequantized values s * v(c), in units of sigma and of the
format's own grid spacing at the larger of the start and end values (one
quantum for int8; 2^(e-3) scale units on the binade [2^e, 2^(e+1)) of E4M3,
2^-9 below 2^-6).

Every pass runs in the library's kernels; the statistics are PyTorch
reductions on the device.  One JSON line per (walk, checkpoint).
"""

import argparse
import json
import math
import sys

import torch

from . import esopt, workloads as wl
from .generation import _walk

CHECKPOINTS = (1, 2, 5, 10, 20, 35, 50, 70, 100, 200)


def _bf16_spacing(x):
    """bf16 spacing at |x| (float32 tensor): 2^(e-7) for |x| in [2^e, 2^(e+1)),
    floored at the subnormal spacing 2^-133."""
    _, e = torch.frexp(x.abs())
    lead = torch.clamp(e.to(torch.int32) - 1, min=-126)
    lead = torch.where(x == 0, torch.full_like(lead, -126), lead)
    return torch.ldexp(torch.ones_like(x), (lead - 7).to(torch.float32))


def drift_stats(views, start, sigma):
    n = 0
    changed = 0
    sq = 0.0
    ulps_sum = 0.0
    ulps_max = 0.0
    over_one = 0
    mag = 0.0
    for v, s in zip(views, start):
        a = v.reshape(-1).float()
        b = s.reshape(-1).float()
        d = a - b
        n += a.numel()
        changed += int((v.reshape(-1).view(torch.int16) != s.reshape(-1).view(torch.int16)).sum())
        sq += float((d.double() ** 2).sum())
        u = d.abs() / _bf16_spacing(torch.maximum(a.abs(), b.abs()))
        ulps_sum += float(u.double().sum())
        ulps_max = max(ulps_max, float(u.max()))
        over_one += int((u > 1.0).sum())
        mag += float((a.abs() - b.abs()).double().sum())
    return {
        "changed": changed / n,
        "rms_over_sigma": math.sqrt(sq / n) / sigma,
        "mean_spacings": ulps_sum / n,
        "max_spacings": ulps_max,
        "beyond_one_spacing": over_one / n,
        "mean_magnitude_change_over_sigma": mag / n / sigma,
    }


def _code_values(codes, fmt):
    """Code values v(c) (float32 tensor) of int8 or E4M3 codes."""
    if fmt == "int8":
        return codes.reshape(-1).float()
    return codes.reshape(-1).view(torch.float8_e4m3fn).float()


def _grid_spacing(m, fmt):
    """Grid spacing of the format at magnitude m >= 0 (code units)."""
    if fmt == "int8":
        return torch.ones_like(m)
    _, e = torch.frexp(m)
    ke = torch.clamp(e.to(torch.int32) - 4, min=-9)
    ke = torch.where(m == 0, torch.full_like(ke, -9), ke)
    return torch.ldexp(torch.ones_like(m), ke.to(torch.float32))


def qdrift_stats(views, start, scales, rows, sigma, fmt):
    """drift_stats for quantized codes, on the dequantized values."""
    n = changed = over_one = 0
    sq = ulps_sum = ulps_max = mag = 0.0
    for v, s0, sc, row in zip(views, start, scales, rows):
        a = _code_values(v, fmt)
        b = _code_values(s0, fmt)
        scale = sc.float().repeat_interleave(row)[:a.numel()] if row else sc.float().expand(
            a.numel())
        d = (a - b) * scale
        n += a.numel()
        changed += int((v.reshape(-1).view(torch.uint8) != s0.reshape(-1).view(torch.uint8)).sum())
        sq += float((d.double() ** 2).sum())
        u = (a - b).abs() / _grid_spacing(torch.maximum(a.abs(), b.abs()), fmt)
        ulps_sum += float(u.double().sum())
        ulps_max = max(ulps_max, float(u.max()))
        over_one += int((u > 1.0).sum())
        mag += float(((a.abs() - b.abs()) * scale).double().sum())
    return {
        "changed": changed / n,
        "rms_over_sigma": math.sqrt(sq / n) / sigma,
        "mean_spacings": ulps_sum / n,
        "max_spacings": ulps_max,
        "beyond_one_spacing": over_one / n,
        "mean_magnitude_change_over_sigma": mag / n / sigma,
    }


def quantized_main(args, W):
    fmt = args.format
    make = wl.device_f8params if fmt == "e4m3" else wl.device_qparams
    flat, views, scales, rows = make(W)
    start_flat = flat.clone()
    offs, _ = wl.flat_layout(W.numels, align=256)
    start = [start_flat[o:o + n] for o, n in zip(offs, W.numels)]
    print(json.dumps({"workload": W.name, "format": fmt, "params": W.n_params,
                      "members": args.members, "sigma": args.sigma,
                      "update_step_rms": args.alpha / math.sqrt(args.members)}), flush=True)
    plan = esopt.QPlan(views, scales, rows, format=fmt)
    for g in range(1, args.generations + 1):
        for i in range(args.members):
            seed = 1_000_003 * g + i
            plan.perturb(seed, 1, args.sigma)
            plan.restore(seed, 1, args.sigma)
        if g in CHECKPOINTS or g == args.generations:
            torch.cuda.synchronize()
            row = {"walk": "restore", "format": fmt, "generation": g,
                   "roundings": g * 2 * args.members}
            row.update(qdrift_stats(views, start, scales, rows, args.sigma, fmt))
            print(json.dumps(row), flush=True)
    plan.close()
    return 0


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--workload", default="dense-4b", choices=sorted(wl.WORKLOADS))
    ap.add_argument("--generations", type=int, default=70)
    ap.add_argument("--members", type=int, default=8)
    ap.add_argument("--sigma", type=float, default=1e-3)
    ap.add_argument("--alpha", type=float, default=5e-4)
    ap.add_argument("--walks", default="restore,swap")
    ap.add_argument("--format", default="bf16", choices=("bf16", "int8", "e4m3"))
    ap.add_argument("--norms-one", action="store_true",
                    help="norm vectors at 1.0 (bf16 only), with a row over them alone")
    args = ap.parse_args(argv)
    W = wl.WORKLOADS[args.workload]
    if args.norms_one and args.format != "bf16":
        ap.error("--norms-one applies to bf16 parameters")
    torch.cuda.set_device(0)
    if args.format != "bf16":
        return quantized_main(args, W)
    flat, views = wl.device_params(W, norm_value=1.0 if args.norms_one else None)
    start_flat = flat.clone()
    offs, _ = wl.flat_layout(W.numels)
    start = [start_flat[o:o + n] for o, n in zip(offs, W.numels)]
    vec = [i for i, shp in enumerate(W.shapes) if len(shp) == 1]
    print(json.dumps({"workload": W.name, "params": W.n_params, "members": args.members,
                      "sigma": args.sigma, "update_step_rms": args.alpha / math.sqrt(args.members),
                      "norms": 1.0 if args.norms_one else "N(0, 0.02)"}),
          flush=True)
    for walk in args.walks.split(","):
        flat.copy_(start_flat)
        plan = esopt.Plan(views)
        for g in range(1, args.generations + 1):
            seeds = [1_000_003 * g + i for i in range(args.members)]
            _walk(plan, seeds, [1] * args.members, args.sigma, walk == "swap",
                  lambda i: None, None)
            if g in CHECKPOINTS or g == args.generations:
                torch.cuda.synchronize()
                row = {"walk": walk, "generation": g,
                       "roundings": g * (2 * args.members if walk == "restore" else args.members + 1)}
                row.update(drift_stats(views, start, args.sigma))
                print(json.dumps(row), flush=True)
                if args.norms_one:
                    row = {"walk": walk, "generation": g, "subset": "norm vectors"}
                    row.update(drift_stats([views[i] for i in vec], [start[i] for i in vec],
                                           args.sigma))
                    print(json.dumps(row), flush=True)
        plan.close()
    return 0


if __name__ == "__main__":
    sys.exit(main())
