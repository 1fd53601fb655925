// uq_device.hpp -- device-side building blocks shared by the libuq kernels
// (gfx950 / CDNA4 only).
//
//  * wht128_x8        fixed 128-point Walsh-Hadamard rotation of a vector
//                     spread over 16 lanes, 8 channels per lane (paper,
//                     section "Ultra-TurboQuant" and Algorithm 1).
//  * ue8m0_exponent   E = round(log2(c*m)) from the fp32 bits (paper,
//                     section "Constant-Optimized Scaling").
//  * e2m1_code        nearest E2M1 level of x / 2^E, ties to the even code.
//  * e4m3_byte        OCP e4m3fn, round to nearest even, saturating.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace uq {

constexpr int kHeadDim = 128;
constexpr int kPage = 16;
constexpr int kGroup = 32;
constexpr int kTileCodes = 1024;   // bytes of codes per (page, head, K|V)
constexpr int kTileScales = 64;    // bytes of scales per (page, head, K|V)

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef __bf16 v2bf __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float bits_f32(uint32_t u) { return __builtin_bit_cast(float, u); }
__device__ __forceinline__ uint32_t f32_bits(float f) { return __builtin_bit_cast(uint32_t, f); }

// fl32(1/sqrt(128)).
__device__ __forceinline__ float inv_sqrt128() { return bits_f32(0x3DB504F3u); }

// The rotation R = H_128 / sqrt(128) of one 128-vector held by 16
// consecutive lanes (lane L of the 16 holds channels 8L..8L+7 in x[0..7]).
// The butterfly runs stage widths 1, 2, 4 inside the lane and 8, 16, 32, 64
// across lanes L^1, L^2, L^4, L^8; each stage maps the pair (i, i+h) to
// (x_i + x_{i+h}, x_i - x_{i+h}) in fp32, and one fp32 multiply by
// fl32(1/sqrt(128)) follows.  The quantised codes are decided from these
// exact fp32 values, so the stage order is part of the cache format.
__device__ __forceinline__ void wht128_x8(float (&x)[8], int L) {
#pragma clang fp contract(off)
#pragma unroll
    for (int h = 1; h < 8; h <<= 1) {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            if (i & h) continue;
            float a = x[i], b = x[i + h];
            x[i] = a + b;
            x[i + h] = a - b;
        }
    }
#pragma unroll
    for (int s = 1; s < 16; s <<= 1) {
        const bool upper = (L & s) != 0;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            float o = __shfl_xor(x[i], s, 16);
            x[i] = upper ? (o - x[i]) : (x[i] + o);
        }
    }
    const float r = inv_sqrt128();
#pragma unroll
    for (int i = 0; i < 8; ++i) x[i] = x[i] * r;
}

// E = round(log2(fl32(c * m))), nearest integer in the log domain: the
// significand of y = c*m is compared with sqrt(2) through its 23 fraction
// bits (1 + f/2^23 >= sqrt(2)  <=>  f >= 0x3504F4).  y == 0 gives -127;
// the result is clamped to [-127, 127].
__device__ __forceinline__ int ue8m0_exponent(float m, float c) {
#pragma clang fp contract(off)
    const float y = c * m;
    if (!(y > 0.0f)) return -127;
    const uint32_t u = f32_bits(y);
    int e = int((u >> 23) & 0xFFu);
    uint32_t frac = u & 0x7FFFFFu;
    int k;
    if (e == 0) {                                  // subnormal y: normalise
        const int p = 31 - __clz(frac);            // position of the leading one
        k = p - 149;
        frac = (frac << (23 - p)) & 0x7FFFFFu;
    } else {
        k = e - 127;
    }
    int E = k + (frac >= 0x3504F4u ? 1 : 0);
    E = E < -127 ? -127 : E;
    E = E > 127 ? 127 : E;
    return E;
}

// Code of x on the E2M1 grid {0,.5,1,1.5,2,3,4,6} after division by 2^E:
// the magnitude index counts the decision thresholds passed, strict at
// thresholds whose lower neighbour has the even index and inclusive where
// the upper neighbour has it (ties to even); |t| > 5 saturates to 6.  The
// sign bit of x is kept.  x * 2^-E is exact (a power-of-two scaling).
__device__ __forceinline__ uint32_t e2m1_code(float x, int E) {
    const float a = __builtin_fabsf(__builtin_ldexpf(x, -E));
    uint32_t k = (a > 0.25f) + (a >= 0.75f) + (a > 1.25f) + (a >= 1.75f) + (a > 2.5f) + (a >= 3.5f) + (a > 5.0f);
    return k | ((f32_bits(x) >> 28) & 8u);
}

// OCP e4m3fn byte of x, round to nearest even, saturating to +-448.
// Normal range: keep 3 fraction bits of the fp32 pattern with RNE (a carry
// moves into the exponent by itself) and rebias 127 -> 7.  Below 2^-6 the
// value is m * 2^-9 with m = rne(|x| * 512) in 0..8 (8 is the smallest normal).
__device__ __forceinline__ uint32_t e4m3_byte(float x) {
    const uint32_t u = f32_bits(x);
    const uint32_t sign = (u >> 24) & 0x80u;
    const uint32_t ua = u & 0x7FFFFFFFu;
    const float a = bits_f32(ua);
    uint32_t mag;
    if (a < 0.015625f) {
        mag = uint32_t(__builtin_rintf(a * 512.0f));
    } else {
        const uint32_t r = (ua + 0x7FFFFu + ((ua >> 20) & 1u)) >> 20;
        mag = r - (120u << 3);
        mag = mag > 0x7Eu ? 0x7Eu : mag;
    }
    return sign | mag;
}

// Scale float 2^(byte-127) for the hardware conversions.  Byte 0 maps to
// 0.0 instead of the subnormal 2^-127: a group with that byte has every
// element below 6 * 2^-127 in magnitude (all zero in practice), so the
// difference is under 1e-37 per element.
__device__ __forceinline__ float ue8m0_to_f32(uint32_t byte) { return bits_f32((byte & 0xFFu) << 23); }

}  // namespace uq
