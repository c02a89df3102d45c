"""Seeded synthetic inputs for the ES parameter path.

This module only describes and materialises inputs: transformer-shaped lists
of bf16 parameter tensors with N(0, 0.02) values, member seeds and signs,
reward vectors, and the scalar hyperparameters of each workload.  It holds
none of the method's arithmetic and imports nothing else from this package, so
both the GPU path's tests and the CPU oracle's tests can draw identical inputs
from it.  bf16 values are produced by PyTorch's own binary32 -> bf16
conversion (host) or by PyTorch's device normal_ (large sets).

Shapes follow the dense decoder families the paper fine-tunes (Qwen3.5-4B and
-27B, LLaMA-3.1-8B; Section 4 onwards and the model list of the appendix):
per layer q, k, v, o projections, SwiGLU gate/up/down and two RMSNorm
vectors, plus embeddings and a final norm.  Hyperparameters (sigma, alpha,
population size) follow the paper's cross-setting hyperparameter table
(Appendix D.6): sigma_0 ~ 1e-3, alpha ~ 5e-4, 8-32 directions per update.
"""

from dataclasses import dataclass, field
from typing import Tuple

import numpy as np

WEIGHT_STD = 0.02


@dataclass(frozen=True)
class Workload:
    name: str
    description: str
    shapes: Tuple[Tuple[int, ...], ...]
    seeds: Tuple[int, ...]
    signs: Tuple[int, ...]
    alpha: float
    sigma0: float
    sigma_T: float
    T: int
    reward_kind: str            # "uniform", "bernoulli0.4" or "normal"
    reward_seed: int
    host_generated: bool = False
    extra: dict = field(default_factory=dict, compare=False)

    @property
    def n_members(self):
        return len(self.seeds)

    @property
    def numels(self):
        return [int(np.prod(s)) for s in self.shapes]

    @property
    def n_params(self):
        return sum(self.numels)

    @property
    def n_distinct(self):
        return len(dict.fromkeys(self.seeds))


def decoder_shapes(layers, hidden, inter, q_dim, kv_dim, vocab, tied):
    """Parameter shapes of a dense decoder: embeddings first, then per layer
    (q, k, v, o, gate, up, down, input norm, post-attention norm), then the
    final norm and (untied) output head."""
    shapes = [(vocab, hidden)]
    for _ in range(layers):
        shapes += [(q_dim, hidden), (kv_dim, hidden), (kv_dim, hidden),
                   (hidden, q_dim), (inter, hidden), (inter, hidden),
                   (hidden, inter), (hidden,), (hidden,)]
    shapes.append((hidden,))
    if not tied:
        shapes.append((vocab, hidden))
    return tuple(shapes)


def _antithetic(n_pairs):
    seeds = tuple(s for s in range(n_pairs) for _ in (0, 1))
    signs = tuple(sg for _ in range(n_pairs) for sg in (1, -1))
    return seeds, signs


TINY = Workload(
    name="tiny-1m",
    description="4 bf16 tensors, 1,016,832 params; N=4 seeds 0..3, sign +1",
    shapes=((256, 1024), (1024, 256), (1024,), (256, 1920)),
    seeds=(0, 1, 2, 3), signs=(1, 1, 1, 1),
    alpha=5e-4, sigma0=1e-3, sigma_T=1e-3, T=1,
    reward_kind="uniform", reward_seed=7, host_generated=True)

_s8, _g8 = _antithetic(4)
DENSE_0P5B = Workload(
    name="dense-0.5b",
    description="24 layers, hidden 1024, intermediate 3072, vocab 151936 tied; "
                "N=8 as 4 antithetic pairs",
    shapes=decoder_shapes(24, 1024, 3072, 1024, 1024, 151936, tied=True),
    seeds=_s8, signs=_g8,
    alpha=5e-4, sigma0=1e-3, sigma_T=1e-3, T=1,
    reward_kind="bernoulli0.4", reward_seed=11)

_s16, _g16 = _antithetic(8)
DENSE_4B = Workload(
    name="dense-4b",
    description="36 layers, hidden 2560, intermediate 9728, 32q/8kv heads x128, "
                "vocab 151936 tied; N=16 as 8 antithetic pairs; sigma cosine "
                "1e-3 -> 1e-4 over 100 steps",
    shapes=decoder_shapes(36, 2560, 9728, 4096, 1024, 151936, tied=True),
    seeds=_s16, signs=_g16,
    alpha=5e-4, sigma0=1e-3, sigma_T=1e-4, T=100,
    reward_kind="uniform", reward_seed=13)

DENSE_27B = Workload(
    name="dense-27b",
    description="64 layers, hidden 5120, intermediate 17408, 40q/8kv heads x128, "
                "vocab 151936 untied (22.70 G params, 45.4 GB bf16); N=32 "
                "distinct seeds, sign +1",
    shapes=decoder_shapes(64, 5120, 17408, 5120, 1024, 151936, tied=False),
    seeds=tuple(range(32)), signs=(1,) * 32,
    alpha=5e-4, sigma0=1e-3, sigma_T=1e-3, T=1,
    reward_kind="uniform", reward_seed=17)

DENSE_27B_EQ = Workload(
    name="dense-27b-77l",
    description="as dense-27b with 77 layers (26.99 G params, 53.98 GB bf16)",
    shapes=decoder_shapes(77, 5120, 17408, 5120, 1024, 151936, tied=False),
    seeds=tuple(range(32)), signs=(1,) * 32,
    alpha=5e-4, sigma0=1e-3, sigma_T=1e-3, T=1,
    reward_kind="uniform", reward_seed=17)


def sweep_workload(n_members):
    """Large-population update on the 4B-shaped set, rewards N(0,1)."""
    return Workload(
        name=f"dense-4b-sweep-n{n_members}",
        description=f"4B-shaped set, fused update with N={n_members} distinct seeds",
        shapes=DENSE_4B.shapes,
        seeds=tuple(range(n_members)), signs=(1,) * n_members,
        alpha=5e-4, sigma0=1e-3, sigma_T=1e-3, T=1,
        reward_kind="normal", reward_seed=19)


WORKLOADS = {w.name: w for w in (TINY, DENSE_0P5B, DENSE_4B, DENSE_27B, DENSE_27B_EQ)}


def rewards(wl, step=0, n=None):
    """Reward vector (binary32) of one generation: drawn from
    default_rng(reward_seed) at step 0 and default_rng([reward_seed, step])
    after that."""
    n = wl.n_members if n is None else n
    rng = np.random.default_rng(wl.reward_seed if step == 0 else [wl.reward_seed, step])
    if wl.reward_kind == "uniform":
        r = rng.random(n)
    elif wl.reward_kind == "bernoulli0.4":
        r = (rng.random(n) < 0.4).astype(np.float64)
    elif wl.reward_kind == "normal":
        r = rng.standard_normal(n)
    else:
        raise ValueError(wl.reward_kind)
    return r.astype(np.float32)


def host_tensor_values(shape, tensor_index, stream=0):
    """fp32 N(0, 0.02) values of one host-generated tensor, seeded by
    (stream, tensor_index)."""
    rng = np.random.default_rng([stream, tensor_index])
    return (rng.standard_normal(int(np.prod(shape))) * WEIGHT_STD).astype(np.float32)


def to_bf16_bits(values_f32):
    """bf16 bit patterns (uint16) of binary32 values, via PyTorch's RNE cast."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(values_f32, dtype=np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16).copy()


def host_params(wl, stream=0):
    """Host-generated bf16 bit arrays (one flat uint16 array per tensor)."""
    return [to_bf16_bits(host_tensor_values(s, i, stream))
            for i, s in enumerate(wl.shapes)]


def random_bf16_bits(n, seed, std=WEIGHT_STD):
    """n N(0, std) bf16 values (bits) from a seed; for ad-hoc test tensors."""
    rng = np.random.default_rng(seed)
    return to_bf16_bits((rng.standard_normal(n) * std).astype(np.float32))


ALIGN_ELEMS = 128   # 256-byte alignment of every tensor inside a flat buffer


def flat_layout(numels, align=ALIGN_ELEMS):
    """Offsets of tensors packed into one buffer, each aligned to `align`
    elements; returns (offsets, total_elements)."""
    offs, cur = [], 0
    for n in numels:
        offs.append(cur)
        cur += (n + align - 1) // align * align
    return offs, cur


def device_params(wl, device="cuda", seed=1234, norm_value=None):
    """Materialise the parameter set on a device as views into one flat bf16
    buffer, values N(0, 0.02) from PyTorch's seeded device generator.  With
    norm_value, the vectors (RMSNorm weights) hold that value instead (1.0 as
    in a trained model; the matrices are the same as without it).
    Returns (flat_buffer, [tensor views])."""
    import torch
    offs, total = flat_layout(wl.numels)
    flat = torch.empty(total, dtype=torch.bfloat16, device=device)
    gen = torch.Generator(device=device)
    gen.manual_seed(seed)
    views = []
    for off, n, shape in zip(offs, wl.numels, wl.shapes):
        v = flat[off:off + n]
        v.normal_(0.0, WEIGHT_STD, generator=gen)
        if norm_value is not None and len(shape) == 1:
            v.fill_(norm_value)
        views.append(v.view(shape))
    return flat, views


# ------------------------------------------------------------------ int8 sets --
# The int8 path's inputs: the same synthetic weights, N(0, 0.02), quantized
# symmetrically to int8 codes with one binary32 scale per row of the last
# dimension (absmax / 127; per output channel for a [out, in] matrix) and one
# scale per tensor for vectors.  This prepares inputs only.

def quantize_rows(w, row):
    """(codes int8, scales float32) of a float32 array quantized per `row`
    consecutive values (row == 0: one scale), symmetric absmax / 127; an
    all-zero row gets scale 1.  Works on numpy arrays and torch tensors."""
    import torch
    t = torch.as_tensor(w, dtype=torch.float32).reshape(-1)
    g = t.reshape(1, -1) if row == 0 else t.reshape(-1, row)
    amax = g.abs().amax(dim=1)
    s = torch.where(amax > 0, amax / 127.0, torch.ones_like(amax))
    q = torch.clamp(torch.round(g / s[:, None]), -127, 127).to(torch.int8).reshape(-1)
    return q, s.contiguous()


def row_of(shape):
    """Scale grouping used for a tensor of this shape: its last dimension for
    matrices (a multiple of 8 in every workload here), one scale for vectors."""
    return int(shape[-1]) if len(shape) >= 2 else 0


def host_qparams(wl, stream=0):
    """Host int8 codes, scales and rows of a workload (numpy)."""
    out = []
    for i, s in enumerate(wl.shapes):
        q, sc = quantize_rows(host_tensor_values(s, i, stream), row_of(s))
        out.append((q.numpy(), sc.numpy(), row_of(s)))
    return out


def device_qparams(wl, device="cuda", seed=1234):
    """The workload's weights drawn on the device (as device_params) and
    quantized per row into one flat int8 buffer (tensors 256-byte aligned).
    Returns (flat_codes, [code views], [scales], [rows])."""
    import torch
    offs, total = flat_layout(wl.numels, align=256)
    flat = torch.empty(total, dtype=torch.int8, device=device)
    gen = torch.Generator(device=device)
    gen.manual_seed(seed)
    views, scales, rows = [], [], []
    for off, n, shape in zip(offs, wl.numels, wl.shapes):
        w = torch.empty(n, dtype=torch.float32, device=device)
        w.normal_(0.0, WEIGHT_STD, generator=gen)
        row = row_of(shape)
        q, s = quantize_rows(w, row)
        del w
        v = flat[off:off + n]
        v.copy_(q)
        views.append(v)
        scales.append(s)
        rows.append(row)
    return flat, views, scales, rows


# ------------------------------------------------------------------ fp8 sets --
# The fp8 path's inputs: the same synthetic weights, N(0, 0.02), quantized to
# E4M3 codes (PyTorch's float8_e4m3fn, round to nearest) with one binary32
# scale per row of the last dimension chosen so the row's largest magnitude
# maps to 448, the format's largest value (absmax / 448), and one scale per
# tensor for vectors -- a per-channel fp8 checkpoint.  This prepares inputs
# only.

E4M3_MAX = 448.0


def quantize_rows_e4m3(w, row):
    """(codes as uint8 bytes of float8_e4m3fn, scales float32) of a float32
    array quantized per `row` consecutive values (row == 0: one scale),
    scale absmax / 448; an all-zero row gets scale 1."""
    import torch
    t = torch.as_tensor(w, dtype=torch.float32).reshape(-1)
    g = t.reshape(1, -1) if row == 0 else t.reshape(-1, row)
    amax = g.abs().amax(dim=1)
    s = torch.where(amax > 0, amax / E4M3_MAX, torch.ones_like(amax))
    c = (g / s[:, None]).clamp(-E4M3_MAX, E4M3_MAX).to(torch.float8_e4m3fn)
    return c.view(torch.uint8).reshape(-1), s.contiguous()


def host_f8params(wl, stream=0):
    """Host E4M3 code bytes, scales and rows of a workload (numpy)."""
    out = []
    for i, s in enumerate(wl.shapes):
        c, sc = quantize_rows_e4m3(host_tensor_values(s, i, stream), row_of(s))
        out.append((c.numpy(), sc.numpy(), row_of(s)))
    return out


def device_f8params(wl, device="cuda", seed=1234):
    """The workload's weights drawn on the device (as device_params) and
    quantized per row into one flat buffer of E4M3 code bytes (tensors
    256-byte aligned).  Returns (flat_codes, [code views], [scales], [rows])."""
    import torch
    offs, total = flat_layout(wl.numels, align=256)
    flat = torch.empty(total, dtype=torch.uint8, device=device)
    gen = torch.Generator(device=device)
    gen.manual_seed(seed)
    views, scales, rows = [], [], []
    for off, n, shape in zip(offs, wl.numels, wl.shapes):
        w = torch.empty(n, dtype=torch.float32, device=device)
        w.normal_(0.0, WEIGHT_STD, generator=gen)
        row = row_of(shape)
        c, s = quantize_rows_e4m3(w, row)
        del w
        v = flat[off:off + n]
        v.copy_(c)
        views.append(v)
        scales.append(s)
        rows.append(row)
    return flat, views, scales, rows
