// MXFP8 element and scale helpers shared by the quantisation kernels and the
// fp8 GEMM epilogue: OCP E4M3 elements, one E8M0 scale 2^s per 32-element
// block with s = floor(log2(amax)) - 8 clamped to [-127, 127] (-127 for an
// all-zero block); elements are v * 2^-s clamped to +-448 and rounded to the
// nearest E4M3 value, ties to even.
#pragma once

#include "common.h"

// floor(log2(a)) - 8 clamped to [-127, 127] for a finite a >= 0; -127 for 0.
DEV int mx_shared_exp(float amax) {
    const uint32_t b = __float_as_uint(amax);
    const int ef = (int)(b >> 23);
    int fl;
    if (ef != 0) {
        fl = ef - 127;
    } else {
        const uint32_t m = b & 0x7fffffu;
        if (m == 0) return -127;
        fl = (31 - __builtin_clz(m)) - 149;   // subnormal: value = m * 2^-149
    }
    const int s = fl - 8;
    return s < -127 ? -127 : (s > 127 ? 127 : s);
}

// Two scaled values -> two E4M3 codes in the low 16 bits.
DEV uint32_t e4m3_pair(float x, float y) {
    x = fminf(fmaxf(x, -448.0f), 448.0f);
    y = fminf(fmaxf(y, -448.0f), 448.0f);
    return (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(x, y, 0, false) & 0xffffu;
}

// 8 values scaled by 2^-s -> 8 codes (little-endian) in two words.
DEV u32x2_t e4m3_pack8(const float (&v)[8], int s) {
    float t[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) t[i] = ldexpf(v[i], -s);
    const uint32_t w0 = e4m3_pair(t[0], t[1]) | (e4m3_pair(t[2], t[3]) << 16);
    const uint32_t w1 = e4m3_pair(t[4], t[5]) | (e4m3_pair(t[6], t[7]) << 16);
    return u32x2_t{w0, w1};
}

// The same for 8 values held in a vector register.
DEV u32x2_t e4m3_pack8(const f32x8 &v, int s) {
    const uint32_t w0 = e4m3_pair(ldexpf(v[0], -s), ldexpf(v[1], -s)) |
                        (e4m3_pair(ldexpf(v[2], -s), ldexpf(v[3], -s)) << 16);
    const uint32_t w1 = e4m3_pair(ldexpf(v[4], -s), ldexpf(v[5], -s)) |
                        (e4m3_pair(ldexpf(v[6], -s), ldexpf(v[7], -s)) << 16);
    return u32x2_t{w0, w1};
}
