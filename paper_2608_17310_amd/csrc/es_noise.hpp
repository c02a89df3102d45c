// Device-side noise and bf16 helpers for gfx950.
//
// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11), the uniform maps and
// the Box-Muller transform, evaluated in binary32 registers.  The paper
// (arXiv 2608.17310, Section 3 and Appendix D.6) only requires that each
// direction be regenerated from an integer seed; the generator, the
// counter layout and the transform are this library's definition, stated in
// include/esopt.h:
//   key     = (seed lo, seed hi)
//   counter = (q lo, q hi, tensor_id, domain),  q = element >> 2
//   element 4q+0, 4q+1 <- Box-Muller(w0, w1) = (r cos phi, r sin phi)
//   element 4q+2, 4q+3 <- Box-Muller(w2, w3)
//   m(w) = w & (2^23 - 1),  u = (m(wa) + 1/2) 2^-23,  v = m(wb) 2^-23
//   r = sqrt(-2 ln u),  phi = 2 pi v
//
// Instruction choices (CDNA4 VALU):
//   * the 32x32->64 products are 64-bit multiplies of zero-extended words,
//     which select v_mad_u64_u32 (both halves in one instruction);
//   * the two three-way XORs of a round are single v_bitop3_b32 (truth table
//     0x96) from the third round on; the first two rounds keep plain XORs,
//     where the counter's high words, the tensor id and the key are
//     wave-uniform and the compiler moves those parts to the scalar unit, and
//     so does the third round's second XOR, whose two other operands are
//     still uniform (a bitop3 may read only one scalar register);
//   * OR-ing the low 23 bits of a word into the exponent of 1.0 (one
//     v_and_or_b32) gives f = 1 + m 2^-23 in [1, 2); u = f - (1 - 2^-24) is
//     exact, and v_sin_f32 / v_cos_f32 take turns and are periodic, so f
//     itself is the angle with no further instruction;
//   * r = sqrt(2 ln 2) sqrt(-log2 u) with the hardware v_log_f32 (log2) and
//     v_sqrt_f32; the constant sqrt(2 ln 2) is folded into the caller's
//     per-pair scale, so applying a scaled normal is one FMA per element;
//   * bf16 results use the gfx950 packed convert (round to nearest even).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace es {

constexpr uint32_t kPhiloxM0 = 0xD2511F53u;
constexpr uint32_t kPhiloxM1 = 0xCD9E8D57u;
constexpr uint32_t kWeyl0 = 0x9E3779B9u;
constexpr uint32_t kWeyl1 = 0xBB67AE85u;
constexpr uint32_t kDomainNoise = 0u;
constexpr uint32_t kDomainRounding = 1u;     // draws of the update's stochastic rounding

struct Words {
    uint32_t w0, w1, w2, w3;
};

constexpr float kSqrt2Ln2 = 1.17741002251547466f;       // sqrt(2 ln 2)

// One Philox round: two 32x32->64 products, two three-way XORs (each a
// single bitop3 when its flag is set).
template <bool kBitop0, bool kBitop2>
__device__ __forceinline__ void philox_round(uint32_t& c0, uint32_t& c1, uint32_t& c2,
                                             uint32_t& c3, uint32_t k0, uint32_t k1) {
    const uint64_t p0 = static_cast<uint64_t>(kPhiloxM0) * c0;
    const uint64_t p1 = static_cast<uint64_t>(kPhiloxM1) * c2;
    uint32_t n0, n2;
    if constexpr (kBitop0)
        n0 = __builtin_amdgcn_bitop3_b32(static_cast<uint32_t>(p1 >> 32), c1, k0, 0x96);
    else
        n0 = static_cast<uint32_t>(p1 >> 32) ^ c1 ^ k0;
    if constexpr (kBitop2)
        n2 = __builtin_amdgcn_bitop3_b32(static_cast<uint32_t>(p0 >> 32), c3, k1, 0x96);
    else
        n2 = static_cast<uint32_t>(p0 >> 32) ^ c3 ^ k1;
    c1 = static_cast<uint32_t>(p1);
    c3 = static_cast<uint32_t>(p0);
    c0 = n0;
    c2 = n2;
}

// One Philox4x32-10 call: ten rounds, the key advanced by the Weyl
// increments between rounds.
__device__ __forceinline__ Words philox4x32_10(uint32_t c0, uint32_t c1, uint32_t c2,
                                               uint32_t c3, uint32_t k0, uint32_t k1) {
    philox_round<false, false>(c0, c1, c2, c3, k0, k1);
    philox_round<false, false>(c0, c1, c2, c3, k0 + kWeyl0, k1 + kWeyl1);
    philox_round<true, false>(c0, c1, c2, c3, k0 + 2 * kWeyl0, k1 + 2 * kWeyl1);
#pragma unroll
    for (uint32_t round = 3; round < 10; ++round)
        philox_round<true, true>(c0, c1, c2, c3, k0 + round * kWeyl0, k1 + round * kWeyl1);
    return Words{c0, c1, c2, c3};
}

// f = 1 + m(w) 2^-23 in [1, 2): the low 23 bits under the exponent of 1.0.
__device__ __forceinline__ float unit_interval_plus_one(uint32_t w) {
    return __uint_as_float((w & 0x007FFFFFu) | 0x3F800000u);
}

// Box-Muller on one word pair, in two parts: the radius factor
// sqrt(-log2 u) (the radius divided by sqrt(2 ln 2)) from the first word,
// and cos / sin of the angle from the second.
__device__ __forceinline__ float pair_radius(uint32_t wa) {
    const float u = unit_interval_plus_one(wa) - 0x1.fffffep-1f;   // (m + 1/2) 2^-23, exact
    return __builtin_amdgcn_sqrtf(-__builtin_amdgcn_logf(u));
}
__device__ __forceinline__ void pair_angle(uint32_t wb, float& c, float& s) {
    const float turns = unit_interval_plus_one(wb);                // 1 + v: same sin / cos as v
    c = __builtin_amdgcn_cosf(turns);
    s = __builtin_amdgcn_sinf(turns);
}

// Box-Muller on one word pair, scaled: the pair's two normals times `scale`
// are t * c and t * s.  t = scale sqrt(2 ln 2) sqrt(-log2 u) is returned
// separately so the caller applies each normal with one FMA.
// scale_k must be scale * kSqrt2Ln2.
__device__ __forceinline__ void scaled_pair(uint32_t wa, uint32_t wb, float scale_k, float& t,
                                            float& c, float& s) {
    t = scale_k * pair_radius(wa);
    pair_angle(wb, c, s);
}

// The four normals of one Philox call, in element order 4q .. 4q+3.
__device__ __forceinline__ void quad_normals(uint32_t q_lo, uint32_t q_hi, uint32_t tensor_id,
                                             uint32_t k0, uint32_t k1, float e[4]) {
    const Words w = philox4x32_10(q_lo, q_hi, tensor_id, kDomainNoise, k0, k1);
    float t, c, s;
    scaled_pair(w.w0, w.w1, kSqrt2Ln2, t, c, s);
    e[0] = t * c;
    e[1] = t * s;
    scaled_pair(w.w2, w.w3, kSqrt2Ln2, t, c, s);
    e[2] = t * c;
    e[3] = t * s;
}

// bf16 <-> binary32.  A bf16 value is the high half of a binary32.
__device__ __forceinline__ float bf16_lo(uint32_t packed) {
    return __uint_as_float(packed << 16);
}
__device__ __forceinline__ float bf16_hi(uint32_t packed) {
    return __uint_as_float(packed & 0xFFFF0000u);
}

typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// Two binary32 values rounded to bf16 (nearest even), packed low/high.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    const f32x2_t v = {lo, hi};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}

// Two binary32 values rounded to bf16 stochastically, packed low/high, with
// the 16-bit draws r_lo = draws mod 2^16 and r_hi = draws div 2^16.  Adding
// r to the binary32 pattern carries into the bf16 part exactly when
// r >= 2^16 - (low 16 bits), i.e. with probability (low 16 bits) / 2^16:
// the fraction of a bf16 step by which |x| exceeds its truncation.  The
// carry out of the largest finite value gives infinity; infinities keep
// their pattern; NaN becomes the quiet NaN 0x7FC0.
__device__ __forceinline__ uint32_t pack_bf16x2_sr(float lo, float hi, uint32_t draws) {
    uint32_t a = __builtin_bit_cast(uint32_t, lo) + (draws & 0xFFFFu);
    uint32_t b = __builtin_bit_cast(uint32_t, hi) + (draws >> 16);
    a = (lo != lo) ? 0x7FC00000u : a;
    b = (hi != hi) ? 0x7FC00000u : b;
    return (b & 0xFFFF0000u) | (a >> 16);
}

__device__ __forceinline__ uint16_t to_bf16(float x) {
    return static_cast<uint16_t>(pack_bf16x2(x, 0.0f) & 0xFFFFu);
}

}  // namespace es
