// Device code of the fp8 path: ES on E4M3 codes (the OCP 8-bit format with
// 4 exponent and 3 mantissa bits, bias 7, largest value 448; codes 0x7F and
// 0xFF are not numbers) with per-row binary32 scales, theta_j = s_r v(c_j).
// The paper lists quantized ES as future work (Appendix A.2).  A pass forms
// x = v(c) + step in scale units in binary32 and rounds it onto the E4M3
// grid:
//   lo = the largest grid point <= x, h its spacing, f = (x - lo) / h,
//   result = lo + h [f >= thr] (strictly f > thr for a restore),
//   clamped to [-448, 448],
// with thr = 1 - u for a perturbation (u = (2 r + 1) 2^-10, r the spare top 9
// bits of the element's own noise word), u itself for a restore (which then
// undoes the perturbation inside a binade), and 1 - r 2^-16 for an update
// (16-bit draw of domain 1 under the rounding seed).
//
// On gfx950 the rounding is the hardware's stochastically rounded
// conversion (v_cvt_sr_fp8_f32).  It rounds |x| away from zero exactly when
// F + R >= 2^32, with F the fraction of |x| above the grid point below it in
// units of the spacing, as 32-bit fixed point (truncated), and R its 32-bit
// random operand; checked on MI355X against that rule for every kind of input
// (normal and subnormal results, exact carry boundaries, signed zeros, values
// next to 448).  A rule on the signed f of x (f = F / 2^32 for x >= 0,
// 1 - F / 2^32 for x < 0 off the grid) maps onto it with one exclusive-or: for
// a threshold thr with 2^32 thr a multiple of 2^16,
//   f >= thr: R = 2^32 - 2^32 thr  for x >= 0,  R = 2^32 thr - 1   for x < 0,
//   f >  thr: R = 2^32 - 2^32 thr - 1,           R = 2^32 thr,
// that is R = A ^ s, s = all ones for x < 0, with A = U for a perturbation
// (thr = 1 - u, U = 2^32 u), ~U for a restore (thr = u, strict) and r 2^16
// for an update (thr = 1 - r 2^-16).  The only inputs where this differs
// from the rule on the exact f are |x| < 2^-18 (below 2^-9 of the smallest
// subnormal) whose fraction lies less than 2^-32 beyond the threshold of a
// comparison that is strict on |x| (a restore with x >= 0, a perturbation or
// update with x < 0): the hardware sees F truncated to 32 bits, and only
// such tiny values have fraction bits below 2^-32.  x is clamped to +-448 first, so no result exceeds the
// format.  Codes decode with the hardware conversion as well.
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>

namespace esf {

typedef float f32x2_t __attribute__((ext_vector_type(2)));

constexpr float kE4M3Max = 448.0f;

// The four codes of a word (code i in byte i) as binary32.
__device__ __forceinline__ void decode4(uint32_t w, float v[4]) {
    const f32x2_t lo = __builtin_amdgcn_cvt_pk_f32_fp8(static_cast<int>(w), false);
    const f32x2_t hi = __builtin_amdgcn_cvt_pk_f32_fp8(static_cast<int>(w), true);
    v[0] = lo.x; v[1] = lo.y; v[2] = hi.x; v[3] = hi.y;
}

// A = U = 2^32 u, u = (2 r + 1) 2^-10, r the word's top 9 bits (the spare
// draw of a perturbation or restore).
__device__ __forceinline__ uint32_t draw9_fixed(uint32_t w) {
    return (w & 0xFF800000u) | 0x00400000u;
}

// Four values rounded onto the grid by the rules above, a[i] the operand for
// x[i] >= 0 (its complement serves x[i] < 0), as the codes of one word.  A
// zero result is +0 (the conversion gives -0 for a negative x that rounds to
// zero; its sign is cleared).
__device__ __forceinline__ uint32_t round4(const float x[4], const uint32_t a[4]) {
    float xc[4];
    uint32_t rn[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        xc[i] = __builtin_amdgcn_fmed3f(x[i], -kE4M3Max, kE4M3Max);
        const uint32_t s = static_cast<uint32_t>(static_cast<int32_t>(__float_as_uint(xc[i])) >> 31);
        rn[i] = a[i] ^ s;
    }
    int w = __builtin_amdgcn_cvt_sr_fp8_f32(xc[0], static_cast<int>(rn[0]), 0, 0);
    w = __builtin_amdgcn_cvt_sr_fp8_f32(xc[1], static_cast<int>(rn[1]), w, 1);
    w = __builtin_amdgcn_cvt_sr_fp8_f32(xc[2], static_cast<int>(rn[2]), w, 2);
    w = __builtin_amdgcn_cvt_sr_fp8_f32(xc[3], static_cast<int>(rn[3]), w, 3);
    const uint32_t u = static_cast<uint32_t>(w);
    // bit 7 of each byte of nz: its magnitude (low 7 bits) is nonzero; the
    // low bits cannot carry out of their byte
    const uint32_t nz = (u & 0x7F7F7F7Fu) + 0x7F7F7F7Fu;
    return u & (nz | 0x7F7F7F7Fu);
}

// Codes that must keep their bytes: not-a-number codes (0x7F, 0xFF) and the
// codes of a row whose scale is invalid (inv == 0; words 0-1 use inv0, 2-3
// inv1).  The check is one add and two masks per word; lanes with nothing to
// keep skip the fix-up.
__device__ __forceinline__ void keep_special(const uint32_t raw[4], float inv0, float inv1,
                                             uint32_t out[4]) {
    uint32_t nan[4], any = 0;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        // low 7 bits all set <=> the byte is 0x7F or 0xFF; +1 cannot carry
        // out of a byte whose top bit was cleared first
        nan[k] = ((raw[k] & 0x7F7F7F7Fu) + 0x01010101u) & 0x80808080u;
        any |= nan[k];
    }
    if (any == 0u && inv0 != 0.0f && inv1 != 0.0f) return;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        uint32_t keep = (nan[k] >> 7) * 0xFFu;               // 0xFF in each flagged byte
        if ((k < 2 ? inv0 : inv1) == 0.0f) keep = 0xFFFFFFFFu;
        out[k] = (out[k] & ~keep) | (raw[k] & keep);
    }
}

}  // namespace esf
