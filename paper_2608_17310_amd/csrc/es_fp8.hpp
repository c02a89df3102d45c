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
// On gfx950 the grid is reached with the exponent unit: for x = m 2^e,
// |m| in [0.5, 1), the spacing is h = 2^max(e - 4, -9) (the subnormal band
// below 2^-6 keeps 2^-9), t = x / h = ldexp(x, -log2 h) is exact, floor(t)
// and t - floor(t) are exact, and the result k h = ldexp(k, log2 h) is a grid
// point (or +-448 after the clamp), which the hardware conversion encodes
// exactly.  Codes decode with the hardware conversion as well.
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

// Four grid values (each exactly representable) as the codes of one word.
__device__ __forceinline__ uint32_t encode4(const float v[4]) {
    int w = __builtin_amdgcn_cvt_pk_fp8_f32(v[0], v[1], 0, false);
    w = __builtin_amdgcn_cvt_pk_fp8_f32(v[2], v[3], w, true);
    return static_cast<uint32_t>(w);
}

// x rounded onto the grid: lo + h when the fraction f of the step from lo
// to the next grid point satisfies f >= thr (f > thr with kStrict), else
// lo; clamped to +-448.  A zero result is +0.
template <bool kStrict>
__device__ __forceinline__ float round_grid(float x, float thr) {
    const int e = __builtin_amdgcn_frexp_expf(x);          // 0 for x = 0
    const int ke = max(e - 4, -9);                           // h = 2^ke
    const float t = __builtin_amdgcn_ldexpf(x, -ke);
    const float fl = __builtin_floorf(t);
    const float f = t - fl;
    const bool step = kStrict ? (f > thr) : (f >= thr);
    const float k = fl + (step ? 1.0f : 0.0f);
    return __builtin_amdgcn_fmed3f(__builtin_amdgcn_ldexpf(k, ke), -kE4M3Max, kE4M3Max);
}

// 1 + r 2^-16 as a binary32 from a 16-bit draw r (exact).
__device__ __forceinline__ float one_plus_draw16(uint32_t r16) {
    return __uint_as_float((r16 << 7) | 0x3F800000u);
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
