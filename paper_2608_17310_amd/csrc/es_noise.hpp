// Device-side noise and bf16 helpers for gfx950.
//
// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11), the uniform map and
// the Box-Muller transform, evaluated in binary32 registers.  The paper
// (arXiv 2608.17310, Section 3 and Appendix D.6) only requires that each
// direction be regenerated from an integer seed; the generator, the
// counter layout and the transform are this library's definition, stated in
// include/esopt.h:
//   key     = (seed lo, seed hi)
//   counter = (q lo, q hi, tensor_id, domain),  q = element >> 2
//   element 4q+0, 4q+1 <- Box-Muller(w0, w1) = (r cos phi, r sin phi)
//   element 4q+2, 4q+3 <- Box-Muller(w2, w3)
//   u(w) = ((w >> 9) + 1/2) 2^-23,  r = sqrt(-2 ln u(wa)),  phi = 2 pi u(wb)
//
// Instruction choices (CDNA4 VALU):
//   * the 32x32->64 products are written as 64-bit multiplies of zero-
//     extended words, which select v_mad_u64_u32 (one instruction for both
//     halves); products and XORs whose operands are wave-uniform (the
//     counter's high words, tensor id, key) are left to the scalar unit;
//   * ln u is taken as ln 2 * log2 u with the hardware v_log_f32, the root
//     with v_sqrt_f32, and the angle goes to v_sin_f32 / v_cos_f32, which
//     take their argument in revolutions, so 2 pi u needs no multiply;
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

struct Words {
    uint32_t w0, w1, w2, w3;
};

// One Philox4x32-10 call: ten rounds of two 32x32->64 products and two
// three-way XORs, the key advanced by the Weyl increments between rounds.
__device__ __forceinline__ Words philox4x32_10(uint32_t c0, uint32_t c1, uint32_t c2,
                                               uint32_t c3, uint32_t k0, uint32_t k1) {
#pragma unroll
    for (int round = 0; round < 10; ++round) {
        const uint64_t p0 = static_cast<uint64_t>(kPhiloxM0) * c0;
        const uint64_t p1 = static_cast<uint64_t>(kPhiloxM1) * c2;
        const uint32_t n0 = static_cast<uint32_t>(p1 >> 32) ^ c1 ^ k0;
        const uint32_t n2 = static_cast<uint32_t>(p0 >> 32) ^ c3 ^ k1;
        c1 = static_cast<uint32_t>(p1);
        c3 = static_cast<uint32_t>(p0);
        c0 = n0;
        c2 = n2;
        k0 += kWeyl0;
        k1 += kWeyl1;
    }
    return Words{c0, c1, c2, c3};
}

// u(w) = ((w >> 9) + 1/2) * 2^-23: the conversion of a 23-bit integer and
// the fused multiply-add are both exact, so u is bit-identical to its fp64
// value.
__device__ __forceinline__ float uniform_open(uint32_t w) {
    return __builtin_fmaf(static_cast<float>(w >> 9), 0x1p-23f, 0x1p-24f);
}

// Box-Muller on one word pair: (r cos phi, r sin phi).
__device__ __forceinline__ void box_muller(uint32_t wa, uint32_t wb, float& e_cos, float& e_sin) {
    const float ua = uniform_open(wa);
    const float ub = uniform_open(wb);                    // revolutions
    // -2 ln u = (-2 ln 2) log2 u
    const float r = __builtin_amdgcn_sqrtf(-1.38629436111989061883f * __builtin_amdgcn_logf(ua));
    e_cos = r * __builtin_amdgcn_cosf(ub);
    e_sin = r * __builtin_amdgcn_sinf(ub);
}

// The four normals of one Philox call, in element order 4q .. 4q+3.
__device__ __forceinline__ void quad_normals(uint32_t q_lo, uint32_t q_hi, uint32_t tensor_id,
                                             uint32_t k0, uint32_t k1, float e[4]) {
    const Words w = philox4x32_10(q_lo, q_hi, tensor_id, kDomainNoise, k0, k1);
    box_muller(w.w0, w.w1, e[0], e[1]);
    box_muller(w.w2, w.w3, e[2], e[3]);
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

__device__ __forceinline__ uint16_t to_bf16(float x) {
    return static_cast<uint16_t>(pack_bf16x2(x, 0.0f) & 0xFFFFu);
}

}  // namespace es
