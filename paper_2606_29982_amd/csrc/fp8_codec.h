// OCP E4M3 (fn) encoding shared by the 8-bit kernels.
#pragma once

#include <stdint.h>

namespace caee {

constexpr float kE4M3Max = 448.0f;   // largest finite E4M3 magnitude

// OCP E4M3 (fn) code of v: nearest representable value, ties to the even
// code, magnitudes above 448 saturate to 448.
__device__ inline uint32_t e4m3_code(float v) {
    const uint32_t sign = (__float_as_uint(v) >> 24) & 0x80u;
    const float a = fminf(fabsf(v), kE4M3Max);
    uint32_t code;
    if (a < 0.015625f) {                       // below 2^-6: subnormal steps of 2^-9
        code = (uint32_t)rintf(a * 512.0f);     // 8 is the smallest normal, code 8
    } else {
        int e = (int)((__float_as_uint(a) >> 23) & 0xFFu) - 127;   // a in [2^e, 2^(e+1))
        uint32_t q = (uint32_t)rintf(ldexpf(a, 3 - e));            // 8 .. 16
        if (q == 16u) {
            q = 8u;
            ++e;
        }
        code = ((uint32_t)(e + 7) << 3) | (q - 8u);
        if (code > 126u) code = 126u;
    }
    return sign | code;
}

}  // namespace caee
