"""One ES generation over a plan, and its deterministic replay.

Host orchestration of the library calls (every step runs in the HIP kernels):
Section 3 and Appendix D.6 of arXiv 2608.17310 apply theta + sigma_t eps_i
for candidate i, evaluate it, revert the perturbation, and after the whole
population apply the z-scored, reward-weighted update with each eps_i
regenerated from its seed; Section 3.1 sets sigma_t on a cosine schedule.

With fused_swap the revert of member i and the apply of member i+1 are one
pass (es_swap), and the last member's revert is made in the update's pass
(es_restore_update), so a generation of N members makes N passes over the
parameters instead of 2N, plus the update; the bits are those of the
separate passes.  The same driver runs the quantized paths (esopt.QPlan, int8
or E4M3 codes), whose swaps are fused too (es_qswap); their last member is
reverted in a pass of its own.  A bf16 plan with binary32 masters
(Plan.set_master) applies each member from the masters (es_perturb_master:
no revert, and each candidate's weights independent of the ones before it)
and updates the masters (ES_UPDATE_MASTER), which rewrites the bf16 values;
its replay needs only the updates.

Only seeds, signs, rewards and scalars (and the stochastic-rounding seed) are
recorded; because every kernel is deterministic, replaying the records from
the same starting parameters rebuilds the parameters bit for bit (the paper reconstructs its final models
from the recorded update sequence the same way, Appendix D.2 and D.4).  A record
can also carry the parameters' 64-bit checksum after its update, which replay
checks.
"""

import json
from dataclasses import asdict, dataclass, fields
from typing import Callable, List, Optional

import torch

from . import esopt


@dataclass
class GenerationRecord:
    seeds: List[int]
    signs: List[int]
    rewards: List[float]            # binary32 values, as passed to es_update
    sigma: float
    alpha: float
    flags: int = 0
    zscore_eps: float = 1e-8
    fused_swap: bool = True
    round_seed: int = 0             # key of the update's stochastic rounding
    checksum: Optional[int] = None  # es_plan_checksum after the update, if recorded


LOG_FORMAT = "es-generation-log/1"


def save_log(path, records, meta=None):
    """Write generation records as a JSON seed log: with the starting
    parameters it is everything replay() needs (Appendix D.2 and D.4 rebuild
    the final models the same way).  Rewards are binary32 values, which JSON
    round-trips exactly as decimal doubles."""
    doc = {"format": LOG_FORMAT, "meta": dict(meta or {}),
           "generations": [asdict(r) for r in records]}
    with open(path, "w") as fh:
        json.dump(doc, fh, indent=1)


def load_log(path):
    """Read a seed log written by save_log; returns (records, meta)."""
    with open(path) as fh:
        doc = json.load(fh)
    if doc.get("format") != LOG_FORMAT:
        raise ValueError(f"{path}: not an {LOG_FORMAT} file")
    names = {f.name for f in fields(GenerationRecord)}
    recs = []
    for g in doc["generations"]:
        unknown = set(g) - names
        if unknown:
            raise ValueError(f"{path}: unknown record fields {sorted(unknown)}")
        recs.append(GenerationRecord(**g))
    return recs, doc["meta"]


def sigma_schedule(sigma0, sigma_T, T):
    """sigma_t for the T updates t = 0 .. T-1 (Section 3.1; es_sigma_cosine)."""
    return [esopt.sigma_cosine(sigma0, sigma_T, t, T) for t in range(T)]


def antithetic_seeds(base_seed, n_pairs):
    """Seeds and signs of n_pairs antithetic pairs: (s, +1), (s, -1), ..."""
    seeds = [int(base_seed) + p for p in range(n_pairs) for _ in (0, 1)]
    signs = [sg for _ in range(n_pairs) for sg in (1, -1)]
    return seeds, signs


def _fuses_last_revert(plan, fused_swap):
    """Whether the walk leaves the last member applied for the update to
    revert in its own pass (es_restore_update)."""
    return fused_swap and hasattr(plan, "restore_update")


def _walk(plan, seeds, signs, sigma, fused_swap, visit, stream, revert_last=True):
    """Apply member 0, visit it, move to member 1, ... and revert the last
    (unless revert_last is false: the update then reverts it).  A plan with
    masters applies every member from them (es_perturb_master) and reverts
    nothing.
    When the passes run on a stream other than PyTorch's current one, each
    visit is ordered after its member's pass and the next pass after the
    visit's work on the current stream, so an evaluation that reads the
    parameters there sees exactly member i applied."""
    n = len(seeds)
    fused_swap = fused_swap and hasattr(plan, "swap")
    s = _torch_stream(stream, plan.device)
    cur = torch.cuda.current_stream(plan.device)
    side = s.cuda_stream != cur.cuda_stream
    # with masters every member is applied from them: nothing to revert
    master = getattr(plan, "has_master", False)
    if master:
        plan.perturb_master(seeds[0], signs[0], sigma, stream=s)
    else:
        plan.perturb(seeds[0], signs[0], sigma, stream=s)
    for i in range(n):
        if side:
            cur.wait_stream(s)
        visit(i)
        if side:
            s.wait_stream(cur)
        if master:
            if i + 1 < n:
                plan.perturb_master(seeds[i + 1], signs[i + 1], sigma, stream=s)
        elif i + 1 < n and fused_swap:
            plan.swap(seeds[i], signs[i], seeds[i + 1], signs[i + 1], sigma, stream=s)
        elif i + 1 < n:
            plan.restore(seeds[i], signs[i], sigma, stream=s)
            plan.perturb(seeds[i + 1], signs[i + 1], sigma, stream=s)
        elif revert_last:
            plan.restore(seeds[i], signs[i], sigma, stream=s)


def run_generation(plan, seeds, signs, sigma, alpha, evaluate: Callable[[int], float],
                   flags=0, zscore_eps=1e-8, fused_swap=True, stream=None, round_seed=0,
                   checksum=False):
    """Run one generation; evaluate(i) scores the parameters while member i is
    applied and returns a float.  Its GPU work goes on PyTorch's current
    stream (or is finished when it returns); the passes go on `stream`.  With ES_UPDATE_STOCHASTIC_ROUND in flags the
    update is rounded with the draws of round_seed (use a new one per
    generation).  With checksum, the parameters' checksum after the update
    is recorded, so that replay() can verify the rebuilt parameters.  Returns the GenerationRecord."""
    if len(seeds) != len(signs) or not seeds:
        raise ValueError("seeds and signs must be non-empty and of equal length")
    if checksum and not hasattr(plan, "checksum"):
        raise ValueError("this plan has no checksum")
    rewards = []
    master = getattr(plan, "has_master", False)
    if master:
        flags |= esopt.ES_UPDATE_MASTER
    fuse = not master and _fuses_last_revert(plan, fused_swap)
    # with masters the update rewrites the bf16 values: nothing to revert last
    _walk(plan, seeds, signs, sigma, fused_swap, lambda i: rewards.append(float(evaluate(i))),
          stream, revert_last=not fuse and not master)
    rec = GenerationRecord(list(map(int, seeds)), list(map(int, signs)),
                           [float(torch.tensor(r, dtype=torch.float32)) for r in rewards],
                           float(sigma), float(alpha), int(flags), float(zscore_eps), fused_swap,
                           int(round_seed))
    apply_update(plan, rec, stream, revert_last=fuse)
    if checksum:
        rec.checksum = plan.checksum(stream=stream)
    return rec


def _torch_stream(stream, device):
    if stream is None:
        return torch.cuda.current_stream(device)
    if isinstance(stream, torch.cuda.Stream):
        return stream
    return torch.cuda.ExternalStream(int(stream), device=device)


def apply_update(plan, rec: GenerationRecord, stream=None, revert_last=False):
    """The record's update; with revert_last, the last member (left applied
    by the walk) is reverted in the same pass (es_restore_update)."""
    # the rewards are staged on the stream the update runs on, so PyTorch's
    # caching allocator does not hand their memory out again before the
    # update has read it
    s = _torch_stream(stream, plan.device)
    with torch.cuda.stream(s):
        r = torch.tensor(rec.rewards, dtype=torch.float32, device=plan.device)
        kw = dict(sigma=rec.sigma, zscore_eps=rec.zscore_eps, flags=rec.flags, stream=s,
                  round_seed=rec.round_seed)
        if revert_last:
            plan.restore_update(rec.seeds[-1], rec.signs[-1], rec.sigma, rec.seeds, rec.signs,
                                r, rec.alpha, **kw)
        else:
            plan.update(rec.seeds, rec.signs, r, rec.alpha, **kw)


class ReplayMismatch(RuntimeError):
    """A replayed generation's parameters differ from the recorded checksum."""


def replay(plan, records, with_perturbations=True, stream=None, verify=True):
    """Re-apply recorded generations.  With with_perturbations (default) the
    perturb / swap / restore passes are replayed too, which reproduces the
    live run bit for bit (their bf16 rounding residues included); without,
    only the updates are applied.  Records of updates into masters
    (ES_UPDATE_MASTER) replay their update alone in either case: it rewrites
    the bf16 values from the masters, which the walk does not touch.  With
    verify (default), every record that carries a checksum is checked after
    its update (replays with perturbations, or of master records: otherwise
    the bits differ by design), raising ReplayMismatch at the first
    generation that differs."""
    for g, rec in enumerate(records):
        # an update into masters does not depend on the bf16 values it
        # rewrites, so the walk is not replayed for it
        master = bool(rec.flags & esopt.ES_UPDATE_MASTER)
        walk = with_perturbations and not master
        fuse = walk and _fuses_last_revert(plan, rec.fused_swap)
        if walk:
            _walk(plan, rec.seeds, rec.signs, rec.sigma, rec.fused_swap, lambda i: None, stream,
                  revert_last=not fuse)
        apply_update(plan, rec, stream, revert_last=fuse)
        if verify and (with_perturbations or master) and rec.checksum is not None:
            got = plan.checksum(stream=stream)
            if got != rec.checksum:
                raise ReplayMismatch(f"generation {g}: checksum {got:#018x}, "
                                     f"recorded {rec.checksum:#018x}")
