// uq_device.hpp -- device-side building blocks shared by the libuq kernels
// (gfx950 / CDNA4 only).
//
//  * wht128_x8        fixed 128-point Walsh-Hadamard rotation of a vector
//                     spread over 16 lanes, 8 channels per lane (paper,
//                     section "Ultra-TurboQuant" and Algorithm 1).
//  * ue8m0_exponent   E = round(log2(c*m)) from the fp32 bits (paper,
//                     section "Constant-Optimized Scaling").
//  * e4m3_byte        OCP e4m3fn, round to nearest even, saturating.
//  * load_x8, encode_token, place_token, store_token
//                     one token's K/V from the input rows into a cache tile.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "uq_internal.hpp"

namespace uq {

constexpr int kHeadDim = 128;
constexpr int kPage = 16;
constexpr int kGroup = 32;
constexpr int kTileCodes = 1024;   // bytes of codes per (page, head, K|V)
constexpr int kTileScales = 64;    // bytes of scales per (page, head, K|V)

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef float v2f __attribute__((ext_vector_type(2)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef __bf16 v2bf __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float bits_f32(uint32_t u) { return __builtin_bit_cast(float, u); }
__device__ __forceinline__ uint32_t f32_bits(float f) { return __builtin_bit_cast(uint32_t, f); }

// fl32(1/sqrt(128)).
__device__ __forceinline__ float inv_sqrt128() { return bits_f32(0x3DB504F3u); }
// fl32(1/sqrt(d)) of the rotation's normalisation: exact for 64 and 256.
template <int D> __device__ __forceinline__ float inv_sqrt_d() {
    static_assert(D == 64 || D == 128 || D == 256, "head size");
    return D == 64 ? 0.125f : D == 256 ? 0.0625f : inv_sqrt128();
}

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

// The same rotation for a head vector of 16 N channels spread over 16 lanes,
// N per lane (lane L holds channels N L + i): stage widths 1 .. N/2 inside a
// lane, then N .. 8 N across lanes, then one multiply by fl32(1/sqrt(16 N)).
// wht_x<8> is wht128_x8.
template <int N>
__device__ __forceinline__ void wht_x(float (&x)[N], int L) {
#pragma clang fp contract(off)
#pragma unroll
    for (int h = 1; h < N; h <<= 1) {
#pragma unroll
        for (int i = 0; i < N; ++i) {
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
        for (int i = 0; i < N; ++i) {
            float o = __shfl_xor(x[i], s, 16);
            x[i] = upper ? (o - x[i]) : (x[i] + o);
        }
    }
    const float r = inv_sqrt_d<16 * N>();
#pragma unroll
    for (int i = 0; i < N; ++i) x[i] = x[i] * r;
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

// The same rule as the UE8M0 byte E + 127, by integer arithmetic on the
// bits u of y = fl32(c * m): for a normal y, adding 2^23 - 0x3504F4 carries
// into the exponent field exactly when the fraction is >= 0x3504F4, so the
// byte is the exponent field of the sum (clamped to 254: E <= 127, also for
// y = +inf); a subnormal y gives E = -126 when y >= sqrt(2) 2^-127 (fraction
// >= 0x5A827A), else E <= -127 (clamped): byte 1 or 0; y = 0 gives byte 0.
// Equal to ue8m0_exponent(m, c) + 127 for every m >= 0 (m is a running
// maximum of magnitudes, never negative or NaN).
__device__ __forceinline__ uint32_t ue8m0_byte(float m, float c) {
#pragma clang fp contract(off)
    const uint32_t u = f32_bits(c * m);
    const uint32_t b = __builtin_elementwise_min((u + 0x4AFB0Cu) >> 23, 254u);
    return u < 0x800000u ? (u >= 0x5A827Au ? 1u : 0u) : b;
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

// Eight consecutive channels starting at element `elem` as fp32 (DT: 0 f32,
// 1 bf16, 2 f16; 16-byte aligned).
template <int DT>
__device__ __forceinline__ void load_x4(const void* base, int64_t elem, float (&x)[4]) {
    if constexpr (DT == 0) {
        const float4 a = *reinterpret_cast<const float4*>(static_cast<const float*>(base) + elem);
        x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
    } else {
        const uint2 w = *reinterpret_cast<const uint2*>(static_cast<const uint16_t*>(base) + elem);
        const uint32_t d[2] = {w.x, w.y};
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            if constexpr (DT == 1) {
                x[2 * i] = bits_f32(d[i] << 16);
                x[2 * i + 1] = bits_f32(d[i] & 0xFFFF0000u);
            } else {
                x[2 * i] = float(__builtin_bit_cast(_Float16, uint16_t(d[i] & 0xFFFFu)));
                x[2 * i + 1] = float(__builtin_bit_cast(_Float16, uint16_t(d[i] >> 16)));
            }
        }
    }
}

template <int DT>
__device__ __forceinline__ void load_x8(const void* base, int64_t elem, float (&x)[8]) {
    if constexpr (DT == 0) {  // f32
        const float4* p = reinterpret_cast<const float4*>(static_cast<const float*>(base) + elem);
        float4 a = p[0], b = p[1];
        x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
        x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
    } else {  // bf16 (1) or f16 (2): 16 bytes
        const uint4 w = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(base) + elem);
        const uint32_t d[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            if constexpr (DT == 1) {
                x[2 * i] = bits_f32(d[i] << 16);
                x[2 * i + 1] = bits_f32(d[i] & 0xFFFF0000u);
            } else {
                x[2 * i] = float(__builtin_bit_cast(_Float16, uint16_t(d[i] & 0xFFFFu)));
                x[2 * i + 1] = float(__builtin_bit_cast(_Float16, uint16_t(d[i] >> 16)));
            }
        }
    }
}

// Quantise the 8 channels this lane holds; returns the packed codes and
// (in the first lane of every 4-lane group) the scale byte.
__device__ __forceinline__ uint32_t quantize_x8(float (&x)[8], int L, float c, bool rotate, uint32_t& scale_byte) {
    if (rotate) wht128_x8(x, L);
    float m = 0.0f;
#pragma unroll
    for (int i = 0; i < 8; ++i) m = __builtin_fmaxf(m, __builtin_fabsf(x[i]));
    m = __builtin_fmaxf(m, __shfl_xor(m, 1, 16));
    m = __builtin_fmaxf(m, __shfl_xor(m, 2, 16));
    const int E = ue8m0_exponent(m, c);
    scale_byte = uint32_t(E + 127);
    // E2M1 codes of x / 2^E by the hardware conversion (nearest level, ties
    // to the even code, saturating at 6, sign kept), channel order, low
    // nibble first; 2^E exactly, subnormal for E = -127
    const float sc = __builtin_ldexpf(1.0f, E);
    uint32_t w = 0u;
    w = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(w, x[0], x[1], sc, 0);
    w = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(w, x[2], x[3], sc, 1);
    w = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(w, x[4], x[5], sc, 2);
    w = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(w, x[6], x[7], sc, 3);
    return w;
}

// One token's K and V as this lane (8 channels 8*lane16..+7 of each)
// stores them, per cache format:
//   kFp4   E2M1 codes (8 per dword) of the rotated K and (rotate_v) V, and
//          the UE8M0 byte of the lane's 32-channel group;
//   kFp8   e4m3(x / scale) bytes, 8 per uint2;
//   kBf16  round-to-nearest-even BF16, 8 per uint4.
template <int F> struct TokenBits;
template <> struct TokenBits<kFp4> { uint32_t k, v, ks, vs; };
template <> struct TokenBits<kFp8> { uint2 k, v; };
template <> struct TokenBits<kBf16> { uint4 k, v; };
template <> struct TokenBits<kTq4> { uint32_t k, v; float n; uint32_t vm; };

// BF16 nearest-even of x, as the fp32 it stands for.
__device__ __forceinline__ float bf16_round(float x) {
    const v2bf h = {__bf16(x), __bf16(0.0f)};
    return bits_f32(__builtin_bit_cast(uint32_t, h) << 16);
}

// s + e = a + b exactly (Knuth's two-sum).
__device__ __forceinline__ void two_sum(double a, double b, double& s, double& e) {
#pragma clang fp contract(off)
    s = a + b;
    const double bb = s - a;
    e = (a - (s - bb)) + (b - bb);
}
// (sh, sl) = (ah, al) + (bh, bl) in double-double arithmetic (about 106
// significant bits), operands in a fixed order.
__device__ __forceinline__ void dd_add(double ah, double al, double bh, double bl, double& sh, double& sl) {
#pragma clang fp contract(off)
    double s, e;
    two_sum(ah, bh, s, e);
    e += al + bl;
    sh = s + e;
    sl = e - (sh - s);
}

// The l2 norm of a 128-vector held 8 channels per lane by 16 lanes, rounded
// once to fp32: the squares (exact in fp64) are summed in double-double
// arithmetic (exact while the magnitudes lie within about 2^25 of each
// other), the square root is taken in fp64 and refined by one Newton step
// on the double-double sum, then rounded to fp32.  Every lane gets the same
// bits: each butterfly step adds the lower lane's partial first.
__device__ __forceinline__ float exact_norm128(const float (&x)[8], int lane16) {
#pragma clang fp contract(off)
    double h = double(x[0]) * double(x[0]), l = 0.0;
#pragma unroll
    for (int i = 1; i < 8; ++i) dd_add(h, l, double(x[i]) * double(x[i]), 0.0, h, l);
#pragma unroll
    for (int s = 1; s < 16; s <<= 1) {
        const double oh = __shfl_xor(h, s, 16), ol = __shfl_xor(l, s, 16);
        if (lane16 & s) dd_add(oh, ol, h, l, h, l);
        else dd_add(h, l, oh, ol, h, l);
    }
    if (!(h > 0.0)) return 0.0f;
    // sqrt(h + l) = r + c to about 2^-100 relative (c: one Newton step)
    const double r = __builtin_sqrt(h);
    const double c = (__builtin_fma(-r, r, h) + l) / (2.0 * r);
    double rh, rl;
    two_sum(r, c, rh, rl);
    const float f = float(rh);
    // rh exactly halfway between f and its neighbour g (the rounding went to
    // the even one) while the remainder rl lies beyond it: the norm is
    // nearer to g
    const double d = rh - double(f);
    if (rl != 0.0 && d != 0.0 && (rl > 0.0) == (d > 0.0) && f > 0.0f && f < 0x1p127f) {
        const float g = bits_f32(f32_bits(f) + (d > 0.0 ? 1u : 0xFFFFFFFFu));   // f > 0: the next float up / down
        if (__builtin_fabs(d) == 0.5 * __builtin_fabs(double(g) - double(f))) return g;
    }
    return f;
}

// Ultra-TQ encoding of the 8 channels this lane holds (all 16 lanes of the
// vector take part).  K: rotated; n = the l2 norm rounded once to fp32
// (exact_norm128); index = that of the level nearest to x / n, ties to the
// lower one: the number of midpoints m_j (exact doubles) with x > m_j n,
// each decided by the sign of fma(-m_j, n, x) in fp64, which is the sign of
// the exact x - m_j n (index 0 when n = 0).  V: per 32-channel group (4
// lanes) zero = bf16(min), scale = bf16(max(max - zero, 0) / 15), code =
// clamp(rint((x - zero) / scale), 0, 15).
__device__ __forceinline__ void tq4_encode(float (&xk)[8], const float (&xv)[8], int lane16, const TqTables& tq,
                                           TokenBits<kTq4>& t) {
    wht128_x8(xk, lane16);
    const float n = exact_norm128(xk, lane16);
    const double nd = n;
    uint32_t wk = 0;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        uint32_t idx = 0;
        if (n > 0.0f) {
#pragma unroll
            for (int j = 0; j < 15; ++j) idx += __builtin_fma(-tq.mid[j], nd, double(xk[i])) > 0.0 ? 1u : 0u;
        }
        wk |= idx << (4 * i);
    }
    float mn = xv[0], mx = xv[0];
#pragma unroll
    for (int i = 1; i < 8; ++i) {
        mn = __builtin_fminf(mn, xv[i]);
        mx = __builtin_fmaxf(mx, xv[i]);
    }
    mn = __builtin_fminf(mn, __shfl_xor(mn, 1, 16));
    mn = __builtin_fminf(mn, __shfl_xor(mn, 2, 16));
    mx = __builtin_fmaxf(mx, __shfl_xor(mx, 1, 16));
    mx = __builtin_fmaxf(mx, __shfl_xor(mx, 2, 16));
    const float z = bf16_round(mn);
    float d = mx - z;
    if (!(d > 0.0f)) d = 0.0f;
    const float s = bf16_round(d / 15.0f);
    uint32_t wv = 0;
    if (s > 0.0f) {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            float r = __builtin_rintf((xv[i] - z) / s);
            r = __builtin_fminf(__builtin_fmaxf(r, 0.0f), 15.0f);
            wv |= uint32_t(r) << (4 * i);
        }
    }
    t.k = wk;
    t.v = wv;
    t.n = n;
    t.vm = (f32_bits(s) >> 16) | (f32_bits(z) & 0xFFFF0000u);
}

// Encode (all 16 lanes of the vector take part: the FP4 rotation and group
// maximum exchange values between them).
template <int F>
__device__ __forceinline__ TokenBits<F> encode_token(float (&xk)[8], float (&xv)[8], int lane16, float c,
                                                     bool rotate_v, float k_scale, float v_scale,
                                                     const TqTables& tq) {
    TokenBits<F> t;
    if constexpr (F == kTq4) {
        tq4_encode(xk, xv, lane16, tq, t);
    } else if constexpr (F == kFp4) {
        t.k = quantize_x8(xk, lane16, c, true, t.ks);
        t.v = quantize_x8(xv, lane16, c, rotate_v, t.vs);
    } else if constexpr (F == kFp8) {
        uint32_t kw[2] = {0u, 0u}, vw[2] = {0u, 0u};
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            kw[i >> 2] |= e4m3_byte(xk[i] / k_scale) << (8 * (i & 3));
            vw[i >> 2] |= e4m3_byte(xv[i] / v_scale) << (8 * (i & 3));
        }
        t.k = make_uint2(kw[0], kw[1]);
        t.v = make_uint2(vw[0], vw[1]);
    } else {
        uint32_t kw[4], vw[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const v2bf hk = {__bf16(xk[2 * i]), __bf16(xk[2 * i + 1])};
            const v2bf hv = {__bf16(xv[2 * i]), __bf16(xv[2 * i + 1])};
            kw[i] = __builtin_bit_cast(uint32_t, hk);
            vw[i] = __builtin_bit_cast(uint32_t, hv);
        }
        t.k = uint4{kw[0], kw[1], kw[2], kw[3]};
        t.v = uint4{vw[0], vw[1], vw[2], vw[3]};
    }
    return t;
}

// Bytes of one (page, head) K or V tile per format (Ultra-TQ: half of the
// page-head block, whose codes, norms and (scale, zero) words sit together).
template <int F> constexpr int tile_bytes() {
    return F == kFp4 ? kTileCodes : F == kFp8 ? 2048 : F == kBf16 ? 4096 : kTqBlock / 2;
}

typedef __attribute__((address_space(3))) uint8_t lds_u8;

// Stores of 1, 4, 8 and 16 bytes at base + off, to global memory or LDS.
__device__ __forceinline__ void st(uint8_t* base, int off, uint8_t x) { base[off] = x; }
__device__ __forceinline__ void st(uint8_t* base, int off, uint32_t x) { *reinterpret_cast<uint32_t*>(base + off) = x; }
__device__ __forceinline__ void st(uint8_t* base, int off, uint2 x) { *reinterpret_cast<uint2*>(base + off) = x; }
__device__ __forceinline__ void st(uint8_t* base, int off, uint4 x) { *reinterpret_cast<uint4*>(base + off) = x; }
__device__ __forceinline__ void st(lds_u8* base, int off, uint8_t x) { base[off] = x; }
__device__ __forceinline__ void st(lds_u8* base, int off, uint32_t x) {
    *reinterpret_cast<__attribute__((address_space(3))) uint32_t*>(base + off) = x;
}
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ void st(lds_u8* base, int off, uint2 x) {
    *reinterpret_cast<__attribute__((address_space(3))) u32x2*>(base + off) = u32x2{x.x, x.y};
}
__device__ __forceinline__ void st(lds_u8* base, int off, uint4 x) {
    *reinterpret_cast<__attribute__((address_space(3))) u32x4*>(base + off) = u32x4{x.x, x.y, x.z, x.w};
}

// Place this lane's part of token `off` into a (page, head) tile pair
// (`tiles`: the K tile, the V tile follows it; `scales`: the pair's 128
// scale bytes, K then V, FP4 only).  Layouts, t = token, c = channel:
//   kFp4   K codes [c/32][t][16 B], nibble order = channel order;
//          V codes [t/4][c/8][t%4][4 B]; scales [K|V][c/32][t].
//   kFp8   K [(c%64)/16][t][32 B]: bytes 0..15 = channels 16g..16g+15,
//          16..31 = channels 64+16g..64+16g+15 (the FP8 operand order of
//          the 16x16x128 MFMA); V [t/4][c/8][t%4][8 B].
//   kBf16  K [c/8][t][16 B]; V [t/4][c/8][t%4][16 B].
//   kTq4   K indices [(c%32)/8][t][c/32][4 B]; V codes (at +1024)
//          [t/4][c/8][t%4][4 B]; `scales` points at the block's norms
//          (fp32 per token) followed at +64 by the (scale, zero) words
//          [t/4][c/32][t%4].
// PTR is a global or an LDS byte pointer: the decode kernel also patches its
// staged copy of a page with a token it has just written.
template <int F, class PTR>
__device__ __forceinline__ void place_token(PTR tiles, PTR scales, int off, int lane16, const TokenBits<F>& t) {
    constexpr int T = tile_bytes<F>();
    if constexpr (F == kFp4) {
        const int g = lane16 >> 2;
        st(tiles, (g * kPage + off) * 16 + 4 * (lane16 & 3), t.k);
        st(tiles, T + ((off >> 2) * 16 + lane16) * 16 + (off & 3) * 4, t.v);
        if ((lane16 & 3) == 0) {
            st(scales, g * kPage + off, uint8_t(t.ks));
            st(scales, kTileScales + g * kPage + off, uint8_t(t.vs));
        }
    } else if constexpr (F == kFp8) {
        const int c0 = 8 * lane16;
        const int g = (c0 & 63) >> 4;
        const int e0 = (c0 & 15) + (c0 >= 64 ? 16 : 0);
        st(tiles, (g * kPage + off) * 32 + e0, t.k);
        st(tiles, T + ((off >> 2) * 16 + lane16) * 32 + (off & 3) * 8, t.v);
    } else if constexpr (F == kBf16) {
        st(tiles, (lane16 * kPage + off) * 16, t.k);
        st(tiles, T + ((off >> 2) * 16 + lane16) * 64 + (off & 3) * 16, t.v);
    } else {
        st(tiles, 16 * (off + 16 * (lane16 & 3)) + 4 * (lane16 >> 2), t.k);
        st(tiles, 1024 + 16 * (lane16 + 16 * (off >> 2)) + 4 * (off & 3), t.v);
        if (lane16 == 0) st(scales, 4 * off, f32_bits(t.n));
        if ((lane16 & 3) == 0) st(scales, 64 + 16 * (4 * (off >> 2) + (lane16 >> 2)) + 4 * (off & 3), t.vm);
    }
}

// Global-memory write of one token into the cache pools (tile = K tile index
// of (page, head); FP4 scales at tile * 64).
template <int F>
__device__ __forceinline__ void store_token(uint8_t* codes, uint8_t* scales, int64_t tile, int off, int lane16,
                                            const TokenBits<F>& t) {
    uint8_t* base = codes + tile * tile_bytes<F>();
    uint8_t* sc = F == kFp4 ? scales + tile * kTileScales : F == kTq4 ? base + kTqMeta : nullptr;
    place_token<F>(base, sc, off, lane16, t);
}

// Scale float 2^(byte-127) for the hardware conversions.  Byte 0 maps to
// 0.0 instead of the subnormal 2^-127: a group with that byte has every
// element below 6 * 2^-127 in magnitude (all zero in practice), so the
// difference is under 1e-37 per element.
__device__ __forceinline__ float ue8m0_to_f32(uint32_t byte) { return bits_f32((byte & 0xFFu) << 23); }

}  // namespace uq
