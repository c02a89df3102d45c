// Device code of the quantized paths: the table, loads, stores and scales
// that int8 and E4M3 plans share, and the int8 rule -- ES on symmetric int8
// codes with per-row binary32 scales, theta_j = s_r(j) q_j, q_j in
// [-127, 127].  The paper lists quantized ES as future work (Appendix A.2):
// noise must respect the quantization scale, updates must stay numerically
// stable, and perturbations must remain replayable from a seed.  Here a
// perturbation or update step d_j (in units of the row's quantum s) becomes
// the integer offset
//   k_j = floor(d_j + r_j 2^-16),   E[k_j] = d_j,
// with a 16-bit draw r_j, and q_j <- clamp(q_j + k_j, -127, 127).
//   * perturb / restore: d_j = sign sigma eps_j / s, eps_j the bf16 path's
//     noise (domain 0) under the member seed, and
//     k_j = floor(d_j + (2 r_j + 1) 2^-10) with r_j the top 9 bits of word
//     j & 3 of element j's own noise call (the uniform map reads only the low
//     23 bits, so these are free); restore subtracts the very same k_j, so it
//     is exact wherever the perturbation did not clamp.
//   * update: d_j = sum_d w_d eps_j(seed_d) / s and
//     k_j = floor(d_j + r_j 2^-16) with a 16-bit r_j from domain 1 under the
//     update's rounding seed: one Philox call at counter
//     (g lo, g hi, tensor_id, 1), g = j >> 3, serves elements 8g .. 8g+7;
//     element j takes word (j & 7) >> 1, low half for even j, high for odd.
// Elements whose scale is not a normal positive finite binary32 value are
// left unchanged.
//
// Layout: a lane owns 16 consecutive codes (one 16-byte access); a tile is
// T lanes x U groups x 16 codes.  Both passes are VALU-bound (16 normals per
// 16 bytes), so they run one group per lane at a time at full occupancy.
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>

#include "es_noise.hpp"
#include "es_table.hpp"

namespace esq {

constexpr int kQGroup = 16;                     // one-byte codes per lane-group

// Quantized tensor table entry (a tensor, a contiguous shard of one or a
// strided block of one).  Tiles are numbered as in the bf16 path: full tiles
// (16-byte aligned base, in bounds) across all tensors, then tail tiles.
// Element j of the entry (its index in the entry's own storage) is element
//   n(j) = noise0 + j + (j / cols) * skip
// of its whole tensor: skip = 0 for a tensor or a contiguous shard; a block
// of rows of `cols` codes out of rows of cols + skip has skip > 0.  n(j)
// selects the noise, the rounding draws and the checksum term; j selects the
// code and its scale.  Every n(j) < 2^31 and numel < 2^31, so indices, and
// the end of the last tile, fit 32 bits.  n(0) and, for a block, cols and
// skip are multiples of 16, so a 16-code group of the entry is a 16-code
// group of the whole tensor.  The divisions j / row (scale index) and
// j / cols are mulhi(j, magic) >> shift, exact for every j < 2^31 (Granlund
// and Montgomery, 1994: magic = ceil(2^(31 + l) / d), l = ceil(log2 d),
// shift = l - 1).
struct DevQTensor {
    int8_t* data;
    const float* scales;
    uint32_t numel;
    uint32_t noise0;                            // whole-tensor index of element 0
    uint64_t first_full;
    uint64_t first_tail;
    uint32_t row;                               // codes per scale; 0: one scale
    uint32_t tensor_id;
    uint32_t magic;
    uint32_t shift;
    uint32_t n_tensors;                         // entries before the sentinel (same in all)
    uint32_t aligned16;                         // base 16-byte aligned: vector tail groups
    uint32_t skip;                              // 0, or whole-tensor codes between block rows
    uint32_t cmagic;                            // j / cols (read only when skip > 0)
    uint32_t cshift;
    uint32_t pad;
};
static_assert(sizeof(DevQTensor) == 80, "quantized tensor table entry layout");

struct QTileRef {
    int8_t* data;
    const float* scales;
    uint32_t numel;
    uint32_t noise0;
    uint32_t elem0;
    uint32_t row;
    uint32_t tensor_id;
    uint32_t magic;
    uint32_t shift;
    uint32_t aligned16;
    uint32_t skip;
    uint32_t cmagic;
    uint32_t cshift;
};

// n(e) of the entry above: the whole-tensor index of local element e.
__device__ __forceinline__ uint32_t qnoise_index(const QTileRef& r, uint32_t e) {
    uint32_t n = r.noise0 + e;
    if (r.skip != 0u) n += (__umulhi(e, r.cmagic) >> r.cshift) * r.skip;
    return n;
}

template <uint32_t kTileElems>
__device__ __forceinline__ QTileRef qlocate_full(const DevQTensor* __restrict__ tab, uint32_t& t,
                                                 uint64_t tile) {
    t = es::seek_tensor(t, tile, tab[0].n_tensors,
                        [tab](uint32_t i) { return tab[i].first_full; });
    return QTileRef{tab[t].data, tab[t].scales, tab[t].numel, tab[t].noise0,
                    static_cast<uint32_t>((tile - tab[t].first_full) * kTileElems), tab[t].row,
                    tab[t].tensor_id, tab[t].magic, tab[t].shift, tab[t].aligned16,
                    tab[t].skip, tab[t].cmagic, tab[t].cshift};
}

template <uint32_t kTileElems>
__device__ __forceinline__ QTileRef qlocate_tail(const DevQTensor* __restrict__ tab, uint32_t& t,
                                                 uint64_t tile) {
    t = es::seek_tensor(t, tile, tab[0].n_tensors,
                        [tab](uint32_t i) { return tab[i].first_tail; });
    const uint64_t n_full = tab[t + 1].first_full - tab[t].first_full;
    return QTileRef{tab[t].data, tab[t].scales, tab[t].numel, tab[t].noise0,
                    static_cast<uint32_t>((n_full + tile - tab[t].first_tail) * kTileElems),
                    tab[t].row, tab[t].tensor_id, tab[t].magic, tab[t].shift, tab[t].aligned16,
                    tab[t].skip, tab[t].cmagic, tab[t].cshift};
}

typedef uint32_t q32x4_t __attribute__((ext_vector_type(4)));
#define ESQ_GLOBAL __attribute__((address_space(1)))

// 16 codes of one group in 4 words (byte i of word k is code 4k + i).  The
// checked path (tail tiles) uses the 16-byte access too when the tensor is
// 16-byte aligned and the whole group is inside it.
template <bool kFast>
__device__ __forceinline__ void qload(const int8_t* __restrict__ p, uint32_t e, uint32_t numel,
                                      uint32_t raw[4], bool vec = false) {
    if (kFast || (vec && e + 16 <= numel)) {
        const q32x4_t v = __builtin_nontemporal_load((const ESQ_GLOBAL q32x4_t*)(p + e));
        raw[0] = v.x; raw[1] = v.y; raw[2] = v.z; raw[3] = v.w;
    } else {
        const ESQ_GLOBAL uint8_t* g = (const ESQ_GLOBAL uint8_t*)p;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            uint32_t w = 0;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const uint32_t j = e + 4 * k + i;
                if (j < numel) w |= uint32_t(g[j]) << (8 * i);
            }
            raw[k] = w;
        }
    }
}

template <bool kFast>
__device__ __forceinline__ void qstore(int8_t* __restrict__ p, uint32_t e, uint32_t numel,
                                       const uint32_t out[4], bool vec = false) {
    if (kFast || (vec && e + 16 <= numel)) {
        const q32x4_t v = {out[0], out[1], out[2], out[3]};
        __builtin_nontemporal_store(v, (ESQ_GLOBAL q32x4_t*)(p + e));
    } else {
        ESQ_GLOBAL uint8_t* g = (ESQ_GLOBAL uint8_t*)p;
#pragma unroll
        for (int k = 0; k < 4; ++k)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const uint32_t j = e + 4 * k + i;
                if (j < numel) g[j] = static_cast<uint8_t>(out[k] >> (8 * i));
            }
    }
}

// The reciprocal of the scale of the 8 codes starting at element j (j is a
// multiple of 8 and the row length a multiple of 8, so the 8 codes share
// one scale), or 0 when the scale is not a normal positive finite value.
// The hardware reciprocal (1 ulp) is well inside the offsets' tolerance.
__device__ __forceinline__ float inv_scale(const QTileRef& r, uint32_t j) {
    if (j >= r.numel) return 0.0f;
    const ESQ_GLOBAL float* s = (const ESQ_GLOBAL float*)r.scales;
    const uint32_t idx = r.row == 0u ? 0u : __umulhi(j, r.magic) >> r.shift;
    const float v = s[idx];
    const bool ok = v >= 0x1p-126f && v <= 0x1.fffffep127f;
    return ok ? __builtin_amdgcn_rcpf(v) : 0.0f;
}

// The two reciprocal scales of a 16-code group (codes 0-7 and 8-15); one
// lookup when the row length is a multiple of 16 (both halves in one row).
__device__ __forceinline__ void group_inv_scales(const QTileRef& r, uint32_t e, float& inv0,
                                                 float& inv1) {
    inv0 = inv_scale(r, e);
    inv1 = (r.row & 15u) == 0u ? inv0 : inv_scale(r, e + 8);
}

// One noise stream's scaled normals for the 16 codes of a group whose first
// code has whole-tensor index n: acc[i] += w_k * (normal of element n + i),
// w_k = weight * sqrt(2 ln 2).
__device__ __forceinline__ void qgroup_axpy(uint32_t n, uint32_t tensor_id, uint32_t k0,
                                            uint32_t k1, float w_k, float acc[16]) {
    const uint32_t q = n >> 2;                  // multiple of 4: q + 3 does not carry
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        const es::Words w = es::philox4x32_10(q + c, 0u, tensor_id, es::kDomainNoise, k0, k1);
        float t, cs, sn;
        es::scaled_pair(w.w0, w.w1, w_k, t, cs, sn);
        acc[4 * c] = __builtin_fmaf(t, cs, acc[4 * c]);
        acc[4 * c + 1] = __builtin_fmaf(t, sn, acc[4 * c + 1]);
        es::scaled_pair(w.w2, w.w3, w_k, t, cs, sn);
        acc[4 * c + 2] = __builtin_fmaf(t, cs, acc[4 * c + 2]);
        acc[4 * c + 3] = __builtin_fmaf(t, sn, acc[4 * c + 3]);
    }
}

// The low bytes of four 32-bit codes packed into one word (code i in byte
// i): two byte permutes and an OR.
__device__ __forceinline__ uint32_t pack_codes(int32_t c0, int32_t c1, int32_t c2, int32_t c3) {
    // v_perm_b32 numbers the second operand's bytes 0-3 and the first's 4-7;
    // selector byte 0x0c yields zero
    const uint32_t lo = __builtin_amdgcn_perm(uint32_t(c1), uint32_t(c0), 0x0c0c0400u);
    const uint32_t hi = __builtin_amdgcn_perm(uint32_t(c3), uint32_t(c2), 0x04000c0cu);
    return lo | hi;
}

// floor(x) as an integer in one instruction (the compiler emits a floor and
// a conversion); x is within +-2^31 here.
__device__ __forceinline__ int32_t floor_to_int(float x) {
    int32_t r;
    asm("v_cvt_flr_i32_f32 %0, %1" : "=v"(r) : "v"(x));
    return r;
}

// 1 + (2 r + 1) 2^-10 as a binary32 from the top 9 bits r of a noise word.
// `one_plus_half_step` is 0x3F802000 (1 + 2^-10) held in a vector register
// by the caller: with the mask in a scalar register the masking and the OR
// are then one v_and_or_b32 (a VOP3 instruction reads at most one scalar
// register or literal on this architecture).
__device__ __forceinline__ float spare_one_plus(uint32_t w, uint32_t one_plus_half_step) {
    return __uint_as_float(((w >> 9) & 0x007FC000u) | one_plus_half_step);
}

// 0x3F802000 in a vector register (see spare_one_plus).
__device__ __forceinline__ uint32_t one_plus_half_step_vgpr() {
    uint32_t c = 0x3F802000u;
    asm volatile("" : "+v"(c));
    return c;
}

// Perturb / restore code: clamp(q +- floor(d + (2 r + 1) 2^-10), lo, 127)
// from v = d + f, f = 1 + (2 r + 1) 2^-10 (formed by the caller as one FMA):
// floor(v) - 1.  v is capped at +-2^30 quanta, far beyond what any code can
// absorb, so the integer arithmetic cannot overflow.  lo is -127; a caller
// whose scale is invalid passes d = 0 (so the step is 0) and lo = -128, which
// returns every code unchanged without a branch.
template <bool kNegate>
__device__ __forceinline__ int32_t qstep9(int32_t q, float v, int32_t lo) {
    const int32_t k = floor_to_int(__builtin_amdgcn_fmed3f(v, -0x1p30f, 0x1p30f)) - 1;
    const int32_t x = kNegate ? q - k : q + k;
    // min(max(x, lo), 127) in one v_med3_i32 (lo <= 127 always; the compiler
    // only forms the median for constant bounds)
    int32_t r;
    asm("v_med3_i32 %0, %1, %2, %3" : "=v"(r) : "v"(x), "v"(lo), "s"(127));
    return r;
}

// Update code: clamp(q + s * floor(d + r 2^-16), -127, 127) with s = -1 when
// kNegate (a restore subtracts the offset its perturb added).  d + r 2^-16
// is one fused multiply-add (one rounding of the exact sum).  |d| is capped
// at 2^30 quanta, far beyond what any code can absorb, so the integer
// arithmetic cannot overflow.
template <bool kNegate>
__device__ __forceinline__ int32_t qstep(int32_t q, float d, uint32_t draw16) {
    const float dc = __builtin_amdgcn_fmed3f(d, -0x1p30f, 0x1p30f);
    const float v = __builtin_fmaf(static_cast<float>(draw16), 0x1p-16f, dc);
    const int32_t k = floor_to_int(v);
    const int32_t x = kNegate ? q - k : q + k;
    return min(max(x, -127), 127);
}

}  // namespace esq
