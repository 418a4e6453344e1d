// OCP E4M3 (fn) encoding shared by the 8-bit kernels.
#pragma once

#include <stdint.h>

namespace caee {

constexpr float kE4M3Max = 448.0f;   // largest finite E4M3 magnitude

// OCP E4M3 (fn) codes of a and b (a in bits 7:0, b in bits 15:8, the rest of
// `old` kept; HI = true puts them in bits 23:16 and 31:24 instead): nearest
// representable value, ties to the even code, magnitudes above 448 saturate
// to 448.  gfx950's packed conversion rounds to nearest even (subnormal
// codes included); clamping to +-448 first gives the saturation.  Checked
// bit for bit against the branch-by-branch definition (code = round(|v| /
// 2^(e - 3)) within binade e, 2^-9 steps below 2^-6, sign bit 0x80) over
// every fp32 value of magnitude up to 448.5, both signs.
template <bool HI = false>
__device__ inline uint32_t e4m3_code2(float a, float b, uint32_t old = 0u) {
    const float ca = fminf(fmaxf(a, -kE4M3Max), kE4M3Max), cb = fminf(fmaxf(b, -kE4M3Max), kE4M3Max);
    return (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(ca, cb, (int)old, HI);
}

// Four codes packed little-endian into one word.
__device__ inline uint32_t e4m3_code4(float a, float b, float c, float d) {
    return e4m3_code2<true>(c, d, e4m3_code2(a, b));
}

}  // namespace caee
