// uq_quantize.hip -- quantize-on-write into the FP4 cache (paper,
// Algorithm 1, "Write") and the FP8 query preparation (Algorithm 1,
// "Decode", first step).
//
// One 128-vector is handled by a quad of 4 lanes holding 32 channels each,
// so a wave64 processes 16 (token, kv head) pairs and a 256-thread block 64.
// Per vector and per K/V: 16-byte loads, the in-register WHT butterfly (5
// in-lane stages and 2 DPP quad-permute stages), the group maxima, the
// UE8M0 exponents, the hardware E2M1 conversion, 4 dword stores of codes
// and one scale byte per lane.
#include "uq_device.hpp"
#include "uq_internal.hpp"

namespace uq {

// Lane exchange inside a quad (4 consecutive lanes) with DPP quad_perm:
// partner lane L^1 or L^2.
template <int S>
__device__ __forceinline__ float quad_xor(float x) {
    constexpr int ctrl = S == 1 ? 0xB1 : 0x4E;   // quad_perm [1,0,3,2] / [2,3,0,1]
    return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, x), ctrl, 0xF, 0xF, true));
}

// One cross-lane butterfly stage for the 8 values of a lane, partner L^S:
// y <- dpp(y) * t + y, one v_fmac_f32 per value with the partner lane's
// value as a DPP (quad_perm) operand (the compiler does not fold the DPP move
// into this tied instruction itself).  s_nop 1 first: a DPP read needs two
// wait states after a VALU write of its register, and inside the block no
// register is read after it is written.  All 64 lanes are active.
#define UQ_FMAC_DPP(P, i) "v_fmac_f32_dpp %" #i ", %" #i ", %8 quad_perm:" P " row_mask:0xf bank_mask:0xf bound_ctrl:1\n\t"
#define UQ_FMAC_DPP8(P)                                                                                          \
    "s_nop 1\n\t" UQ_FMAC_DPP(P, 0) UQ_FMAC_DPP(P, 1) UQ_FMAC_DPP(P, 2) UQ_FMAC_DPP(P, 3) UQ_FMAC_DPP(P, 4)      \
        UQ_FMAC_DPP(P, 5) UQ_FMAC_DPP(P, 6) UQ_FMAC_DPP(P, 7)
template <int S>
__device__ __forceinline__ void quad_stage8(float (&y)[8], float t) {
    if constexpr (S == 1) {
        asm volatile(UQ_FMAC_DPP8("[1,0,3,2]")
                     : "+v"(y[0]), "+v"(y[1]), "+v"(y[2]), "+v"(y[3]), "+v"(y[4]), "+v"(y[5]), "+v"(y[6]), "+v"(y[7])
                     : "v"(t));
    } else {
        asm volatile(UQ_FMAC_DPP8("[2,3,0,1]")
                     : "+v"(y[0]), "+v"(y[1]), "+v"(y[2]), "+v"(y[3]), "+v"(y[4]), "+v"(y[5]), "+v"(y[6]), "+v"(y[7])
                     : "v"(t));
    }
}
#undef UQ_FMAC_DPP8
#undef UQ_FMAC_DPP

// The rotation in its plain form: each cross-lane stage moves the partner's
// value (DPP) and combines it with one fma, fma(s, x, o) = x + o or o - x.
// wht_quad below gives the same values with one instruction per value and
// stage, except for the signs of exact zeros when the input vector is all
// zero; quantize_xq falls back to this form for such vectors.
template <int NG>
__device__ __forceinline__ void wht_quad_plain(float (&x)[NG][8], int L) {
#pragma clang fp contract(off)
#pragma unroll
    for (int h = 1; h < 8; h <<= 1) {
#pragma unroll
        for (int j = 0; j < NG; ++j) {
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                if (i & h) continue;
                const float a = x[j][i], b = x[j][i + h];
                x[j][i] = a + b;
                x[j][i + h] = a - b;
            }
        }
    }
    const float s1 = (L & 1) ? -1.0f : 1.0f;
    const float s2 = (L & 2) ? -1.0f : 1.0f;
#pragma unroll
    for (int j = 0; j < NG; ++j)
#pragma unroll
        for (int i = 0; i < 8; ++i) x[j][i] = __builtin_fmaf(s1, x[j][i], quad_xor<1>(x[j][i]));
#pragma unroll
    for (int j = 0; j < NG; ++j)
#pragma unroll
        for (int i = 0; i < 8; ++i) x[j][i] = __builtin_fmaf(s2, x[j][i], quad_xor<2>(x[j][i]));
#pragma unroll
    for (int h = 1; h < NG; h <<= 1) {
#pragma unroll
        for (int j = 0; j < NG; ++j) {
            if (j & h) continue;
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const float a = x[j][i], b = x[j + h][i];
                x[j][i] = a + b;
                x[j + h][i] = a - b;
            }
        }
    }
    const float r = inv_sqrt_d<32 * NG>();
#pragma unroll
    for (int j = 0; j < NG; ++j)
#pragma unroll
        for (int i = 0; i < 8; ++i) x[j][i] = x[j][i] * r;
}

// The rotation of one head vector of D = 32 NG channels held by 4 lanes of
// a quad: lane L holds channels 32j + 8L + i in x[j][i] (j < NG, i < 8).
// The stages run in the order of the format (widths 1, 2, 4, ..., D/2): 1,
// 2, 4 inside a lane over i, 8 and 16 across lanes L^1, L^2, then 32, 64
// (and 128 for D = 256) inside a lane over j; each maps (a, b) to
// (a + b, a - b) in fp32, then one multiply by fl32(1/sqrt(D)).  The values
// equal those of the 16-lane form wht_x bit for bit.
//
// The two cross-lane stages take one instruction per value,
// v_fmac_f32 with the partner's value as a DPP operand: y <- dpp(y) * t + y
// with t = +-1 per lane.  The upper lane of a pair needs o - x but a single
// form gives it x - o, so it keeps the negated value (every fp32 rounding is
// symmetric under negation) and its sign sigma is tracked: t1 = sigma after
// the first stage, and since both lanes of a second-stage pair carry the
// same sigma, t2 makes the second stage right up to sign too; the final
// multiply by sigma * fl32(1/sqrt(D)) (exact) restores every value.
// Negation symmetry fails at exact zeros only: an exact cancellation gives
// +0 whatever the signs.  The reference form yields -0 only from a subtree
// of zeros, and every output depends on all inputs, so for an input that is
// not all zero every zero output is +0: the final step is fma(y, sigma r,
// +0), which keeps every nonzero result (and the sign of an underflow) and
// turns every exact zero into +0.  An all-zero input is left to
// wht_quad_plain.
template <int NG>
__device__ __forceinline__ void wht_quad(float (&x)[NG][8], int L) {
#pragma clang fp contract(off)
#pragma unroll
    for (int h = 1; h < 8; h <<= 1) {
#pragma unroll
        for (int j = 0; j < NG; ++j) {
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                if (i & h) continue;
                const float a = x[j][i], b = x[j][i + h];
                x[j][i] = a + b;
                x[j][i + h] = a - b;
            }
        }
    }
    const float t1 = (L & 1) ? -1.0f : 1.0f;
    const float t2 = (L & 2) ? -1.0f : 1.0f;
#pragma unroll
    for (int j = 0; j < NG; ++j) quad_stage8<1>(x[j], t1);
#pragma unroll
    for (int j = 0; j < NG; ++j) quad_stage8<2>(x[j], t2);
#pragma unroll
    for (int h = 1; h < NG; h <<= 1) {
#pragma unroll
        for (int j = 0; j < NG; ++j) {
            if (j & h) continue;
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const float a = x[j][i], b = x[j + h][i];
                x[j][i] = a + b;
                x[j + h][i] = a - b;
            }
        }
    }
    const float r = inv_sqrt_d<32 * NG>() * (t1 * t2);
#pragma unroll
    for (int j = 0; j < NG; ++j)
#pragma unroll
        for (int i = 0; i < 8; ++i) x[j][i] = __builtin_fmaf(x[j][i], r, 0.0f);
}

__device__ __forceinline__ void wht128_x32(float (&x)[4][8], int L) { wht_quad<4>(x, L); }

// Quantise one head vector held by a quad (rotated first if `rotate`): per
// 32-channel group j the UE8M0 byte b_j = E_j + 127 of the group maximum
// (ue8m0_byte), and the E2M1 codes of the lane's 8 channels of the group in
// w[j] (channel order, low nibble first) by the hardware conversion, which
// rounds x / 2^E_j to the nearest E2M1 level with ties to the even code,
// saturates at 6 and keeps the sign (checked against a threshold encoder
// over every tie, both zeros, subnormal inputs and scales 2^-127 .. 2^127).
// `src` and `row` locate the vector's input (rows of dtype DT) for the
// all-zero case.
template <int DT, int NG>
__device__ __forceinline__ void quantize_xq(float (&x)[NG][8], int L, float c, bool rotate, uint32_t (&w)[NG],
                                            uint32_t (&byte)[NG], const void* src, int64_t row) {
    if (rotate) wht_quad<NG>(x, L);
    float m[NG];
    float mall = 0.0f;
#pragma unroll
    for (int j = 0; j < NG; ++j) {
        // group maximum of |x|: three-input maxima, then the quad
        float mj = __builtin_fmaxf(__builtin_fmaxf(__builtin_fabsf(x[j][0]), __builtin_fabsf(x[j][1])),
                                   __builtin_fabsf(x[j][2]));
        mj = __builtin_fmaxf(__builtin_fmaxf(mj, __builtin_fabsf(x[j][3])), __builtin_fabsf(x[j][4]));
        mj = __builtin_fmaxf(__builtin_fmaxf(mj, __builtin_fabsf(x[j][5])), __builtin_fabsf(x[j][6]));
        mj = __builtin_fmaxf(mj, __builtin_fabsf(x[j][7]));
        mj = __builtin_fmaxf(mj, quad_xor<1>(mj));
        m[j] = __builtin_fmaxf(mj, quad_xor<2>(mj));
        mall = __builtin_fmaxf(mall, m[j]);
    }
    // every rotated value zero (quad-uniform): the signs of the zeros, which
    // the codes keep, come from the plain form of the rotation
    if (rotate && __builtin_amdgcn_ballot_w64(mall == 0.0f) != 0 && mall == 0.0f) {
#pragma unroll
        for (int j = 0; j < NG; ++j) load_x8<DT>(src, row + 32 * j, x[j]);
        wht_quad_plain<NG>(x, L);
    }
#pragma unroll
    for (int j = 0; j < NG; ++j) {
        byte[j] = ue8m0_byte(m[j], c);
        const float sc = __builtin_ldexpf(1.0f, int(byte[j]) - 127);   // 2^E exactly (subnormal for E = -127)
        uint32_t v = 0u;
        v = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(v, x[j][0], x[j][1], sc, 0);
        v = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(v, x[j][2], x[j][3], sc, 1);
        v = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(v, x[j][4], x[j][5], sc, 2);
        v = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(v, x[j][6], x[j][7], sc, 3);
        w[j] = v;
    }
}

// Element j of a small register array at a lane-dependent index, by selects
// (a dynamic index would put the array in scratch memory).
template <int NG>
__device__ __forceinline__ uint32_t pick(const uint32_t (&e)[NG], int j) {
    uint32_t r = e[0];
#pragma unroll
    for (int k = 1; k < NG; ++k) r = j == k ? e[k] : r;
    return r;
}

// Quantize-on-write, 4 lanes (one quad) per (token, kv head) vector of
// D = 32 NG channels, 16 tokens of one kv head per wave.  The waves run kv
// head fastest (a 256-thread block takes 4 kv heads of the same 16 tokens),
// so a block reads 4 heads' slices of the same rows and, when the tokens
// fill a page in order, writes 4 of that page's (page, head) tiles and 4 of
// its scale blocks, next to each other (3 % faster than 64 tokens of one
// head per block, whose page tiles went to 8 XCDs).  K's codes and scale
// bytes are stored as soon as K is encoded, so that those stores overlap
// V's encoding.  Lane L loads and keeps channels 32j + 8L + i (16-byte
// loads, a quad covers 64 contiguous bytes per j), so the two cross-lane
// stages of the rotation and the group maxima are DPP quad permutes.
// Stores: one codes dword per group for K and V, and the scale bytes of
// groups L, L + 4, ... for K and V.  Tiles are 8 D code bytes and D/2 scale
// bytes per (page, head, K|V).
template <int DT, int NG>
__global__ void __launch_bounds__(256) quantize_kv_kernel(QuantizeParams p) {
    constexpr int D = 32 * NG;
    const int L = threadIdx.x & 3;
    const unsigned wi = blockIdx.x * 4u + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave unit
    const int h = int(wi % unsigned(p.num_kv_heads));                       // wave-uniform
    const int64_t t = int64_t(wi / unsigned(p.num_kv_heads)) * 16 + ((threadIdx.x & 63) >> 2);
    if (t >= p.num_tokens) return;   // whole quads leave together

    // The rows are loaded together with the slot, before the slot is known
    // to be valid: the row loads then overlap the slot and page-table
    // lookups instead of waiting behind them (a padding token's row is read
    // for nothing).
    const int64_t slot = p.slot_mapping[t];
    const int64_t row = t * p.token_stride + int64_t(h) * D + 8 * L;
    float xk[NG][8], xv[NG][8];
#pragma unroll
    for (int j = 0; j < NG; ++j) {
        load_x8<DT>(p.k, row + 32 * j, xk[j]);
        load_x8<DT>(p.v, row + 32 * j, xv[j]);
    }
    if (slot < 0) return;
    int64_t page;
    int off;
    if (p.page_table != nullptr) {
        const int64_t per_seq = int64_t(p.max_pages_per_seq) * kPage;
        const int64_t seq = slot / per_seq;
        const int64_t pos = slot - seq * per_seq;
        if (seq >= p.num_seqs) return;
        page = p.page_table[seq * p.max_pages_per_seq + pos / kPage];
        off = int(pos % kPage);
    } else {
        page = slot >> 4;
        off = int(slot & (kPage - 1));
    }
    if (page < 0 || page >= p.num_pages) return;

    uint32_t wk[NG], wv[NG], bk[NG], bv[NG];
    const int64_t ph = page * p.num_kv_heads + h;
    uint8_t* kc = p.codes + ph * (16 * D);
    uint8_t* vc = kc + 8 * D;
    uint8_t* ks = p.scales + ph * D;
    quantize_xq<DT, NG>(xk, L, p.c, true, wk, bk, p.k, row);
#pragma unroll
    for (int j = 0; j < NG; ++j) *reinterpret_cast<uint32_t*>(kc + (j * kPage + off) * 16 + 4 * L) = wk[j];
#pragma unroll
    for (int q = 0; q < (NG + 3) / 4; ++q) {
        const int j = L + 4 * q;
        if (j < NG) ks[j * kPage + off] = uint8_t(pick<NG>(bk, j));
    }
    quantize_xq<DT, NG>(xv, L, p.c, p.rotate_v != 0, wv, bv, p.v, row);
#pragma unroll
    for (int j = 0; j < NG; ++j)
        *reinterpret_cast<uint32_t*>(vc + ((off >> 2) * (D / 8) + 4 * j + L) * 16 + (off & 3) * 4) = wv[j];
#pragma unroll
    for (int q = 0; q < (NG + 3) / 4; ++q) {
        const int j = L + 4 * q;
        if (j < NG) ks[D / 2 + j * kPage + off] = uint8_t(pick<NG>(bv, j));
    }
}

// Round-trip error of the FP4 encoder for a list of constants c, the
// one-dimensional fit of section "Constant-Optimized Scaling": per row
// (rotated like K when `rotate`), per 32-channel group with maximum m, the
// codes of x / s are decoded back to code * s and the squared error summed,
// for the deployed scale s = 2^round(log2(c m)) (UE8M0, pow2) or the
// continuous s = c m.  One quad per row as in quantize_kv_kernel, 64 rows
// per tile, tiles strided over the grid.  Each wave folds its per-tile sums
// into its own fp64 LDS slots; at the end the block adds its totals to
// `sums` with one fp64 atomic per value.
template <int DT>
__global__ void __launch_bounds__(256) quantize_error_kernel(ErrorParams p) {
    __shared__ double acc[4][kMaxErrorConstants];
    __shared__ double energy[4];
    for (int i = threadIdx.x; i < 4 * kMaxErrorConstants; i += 256) (&acc[0][0])[i] = 0.0;
    if (threadIdx.x < 4) energy[threadIdx.x] = 0.0;
    __syncthreads();
    const int L = threadIdx.x & 3;
    const int wave = threadIdx.x >> 6;
    const bool lead = (threadIdx.x & 63) == 0;
    const int64_t tiles = (p.rows + 63) / 64;
    for (int64_t tile = blockIdx.x; tile < tiles; tile += gridDim.x) {
        const int64_t row = tile * 64 + (threadIdx.x >> 2);
        float x[4][8];
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int i = 0; i < 8; ++i) x[j][i] = 0.0f;
        if (row < p.rows) {
#pragma unroll
            for (int j = 0; j < 4; ++j) load_x8<DT>(p.x, row * p.row_stride + 32 * j + 8 * L, x[j]);
        }
        if (p.rotate) wht128_x32(x, L);   // whole quads: rows past the end rotate zeros
        float m[4];
        float sq = 0.0f;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            m[j] = 0.0f;
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                m[j] = __builtin_fmaxf(m[j], __builtin_fabsf(x[j][i]));
                sq = __builtin_fmaf(x[j][i], x[j][i], sq);
            }
            m[j] = __builtin_fmaxf(m[j], quad_xor<1>(m[j]));
            m[j] = __builtin_fmaxf(m[j], quad_xor<2>(m[j]));
        }
#pragma unroll
        for (int s = 1; s < 64; s <<= 1) sq += __shfl_xor(sq, s);
        if (lead) energy[wave] += double(sq);
        for (int ci = 0; ci < p.num_c; ++ci) {
            const float c = p.c_values[ci];
            float err = 0.0f;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                if (!(m[j] > 0.0f)) continue;   // an all-zero group decodes exactly
                if (p.pow2) {
                    // The cache encoder itself: scale operand 2^E, decode by the same scale.
                    const float sc = __builtin_ldexpf(1.0f, int(ue8m0_byte(m[j], c)) - 127);
#pragma unroll
                    for (int i = 0; i < 8; i += 2) {
                        const uint32_t w = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(0u, x[j][i], x[j][i + 1], sc, 0);
                        const v2f d = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(w, sc, 0);
                        const float e0 = x[j][i] - d[0], e1 = x[j][i + 1] - d[1];
                        err = __builtin_fmaf(e0, e0, err);
                        err = __builtin_fmaf(e1, e1, err);
                    }
                } else {
                    // Continuous scale: nearest E2M1 level of fl32(x / s), times s.
                    const float sc = c * m[j];
#pragma unroll
                    for (int i = 0; i < 8; i += 2) {
                        const float t0 = x[j][i] / sc, t1 = x[j][i + 1] / sc;
                        const uint32_t w = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(0u, t0, t1, 1.0f, 0);
                        const v2f d = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(w, 1.0f, 0);
                        const float e0 = x[j][i] - d[0] * sc, e1 = x[j][i + 1] - d[1] * sc;
                        err = __builtin_fmaf(e0, e0, err);
                        err = __builtin_fmaf(e1, e1, err);
                    }
                }
            }
#pragma unroll
            for (int s = 1; s < 64; s <<= 1) err += __shfl_xor(err, s);
            if (lead) acc[wave][ci] += double(err);
        }
    }
    __syncthreads();
    if (threadIdx.x < p.num_c) {
        const int ci = threadIdx.x;
        atomicAdd(&p.sums[2 * ci], acc[0][ci] + acc[1][ci] + acc[2][ci] + acc[3][ci]);
        atomicAdd(&p.sums[2 * ci + 1], energy[0] + energy[1] + energy[2] + energy[3]);
    }
}

// Writer of the comparison caches (FP8 E4M3 with one scale per tensor,
// BF16, or the Ultra-TQ codebook cache), 16 lanes per (token, kv head)
// vector; the layouts are those of place_token.
template <int DT, int FMT>
__global__ void __launch_bounds__(256) write_kv_ref_kernel(RefWriteParams p) {
    const int lane16 = threadIdx.x & 15;
    const int64_t vec = int64_t(blockIdx.x) * 16 + (threadIdx.x >> 4);
    const int64_t nvec = p.num_tokens * p.num_kv_heads;
    if (vec >= nvec) return;
    const int64_t t = vec / p.num_kv_heads;
    const int h = int(vec - t * p.num_kv_heads);
    const int64_t slot = p.slot_mapping[t];
    if (slot < 0) return;
    int64_t page;
    int off;
    if (p.page_table != nullptr) {
        const int64_t per_seq = int64_t(p.max_pages_per_seq) * kPage;
        const int64_t seq = slot / per_seq;
        const int64_t pos = slot - seq * per_seq;
        if (seq >= p.num_seqs) return;
        page = p.page_table[seq * p.max_pages_per_seq + pos / kPage];
        off = int(pos % kPage);
    } else {
        page = slot / kPage;
        off = int(slot % kPage);
    }
    if (page < 0 || page >= p.num_pages) return;
    const int64_t elem = t * p.token_stride + int64_t(h) * kHeadDim + 8 * lane16;
    float xk[8], xv[8];
    load_x8<DT>(p.k, elem, xk);
    load_x8<DT>(p.v, elem, xv);
    const TokenBits<FMT> tb = encode_token<FMT>(xk, xv, lane16, 0.0f, false, p.k_scale, p.v_scale, p.tq);
    store_token<FMT>(p.cache, nullptr, (page * p.num_kv_heads + h) * 2, off, lane16, tb);
}

template <int DT>
__global__ void __launch_bounds__(256) prepare_query_kernel(const void* q, int64_t rows, uint8_t* q8) {
    const int lane16 = threadIdx.x & 15;
    const int64_t row = int64_t(blockIdx.x) * 16 + (threadIdx.x >> 4);
    if (row >= rows) return;
    float x[8];
    load_x8<DT>(q, row * kHeadDim + 8 * lane16, x);
    wht128_x8(x, lane16);
    uint32_t lo = 0, hi = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        lo |= e4m3_byte(x[i]) << (8 * i);
        hi |= e4m3_byte(x[i + 4]) << (8 * i);
    }
    *reinterpret_cast<uint2*>(q8 + row * kHeadDim + 8 * lane16) = make_uint2(lo, hi);
}

template <int NG>
static void launch_quantize_ng(const QuantizeParams& p, int dtype, const dim3& grid, hipStream_t stream) {
    const dim3 block{256u};
    if (dtype == 0) launch_kernel(quantize_kv_kernel<0, NG>, grid, block, stream, p);
    else if (dtype == 1) launch_kernel(quantize_kv_kernel<1, NG>, grid, block, stream, p);
    else launch_kernel(quantize_kv_kernel<2, NG>, grid, block, stream, p);
}

hipError_t launch_quantize_kv(const QuantizeParams& p, int dtype, hipStream_t stream) {
    // wave units of 16 tokens of one kv head, kv head fastest, 4 per block
    const int64_t units = (p.num_tokens + 15) / 16 * p.num_kv_heads;
    if (units == 0) return hipSuccess;
    if (units > 0x7FFFFFFF) return hipErrorInvalidValue;   // the kernel numbers them in 32 bits
    const int64_t blocks = (units + 3) / 4;
    const dim3 grid{unsigned(blocks)};
    if (p.head_dim == 64) launch_quantize_ng<2>(p, dtype, grid, stream);
    else if (p.head_dim == 256) launch_quantize_ng<8>(p, dtype, grid, stream);
    else launch_quantize_ng<4>(p, dtype, grid, stream);
    return hipGetLastError();
}

template <int DT>
static hipError_t launch_ref(const RefWriteParams& p, const dim3& grid, hipStream_t stream) {
    if (p.kv_fmt == kFp8) hipLaunchKernelGGL((write_kv_ref_kernel<DT, kFp8>), grid, dim3(256), 0, stream, p);
    else if (p.kv_fmt == kTq4) hipLaunchKernelGGL((write_kv_ref_kernel<DT, kTq4>), grid, dim3(256), 0, stream, p);
    else hipLaunchKernelGGL((write_kv_ref_kernel<DT, kBf16>), grid, dim3(256), 0, stream, p);
    return hipGetLastError();
}

hipError_t launch_write_kv_ref(const RefWriteParams& p, int dtype, hipStream_t stream) {
    const int64_t nvec = p.num_tokens * p.num_kv_heads;
    const int64_t blocks = (nvec + 15) / 16;
    if (blocks == 0) return hipSuccess;
    if (blocks > 0x7FFFFFFF) return hipErrorInvalidValue;
    const dim3 grid{unsigned(blocks)};
    if (dtype == 0) return launch_ref<0>(p, grid, stream);
    if (dtype == 1) return launch_ref<1>(p, grid, stream);
    return launch_ref<2>(p, grid, stream);
}

hipError_t launch_quantize_error(const ErrorParams& p, int dtype, hipStream_t stream) {
    const int64_t tiles = (p.rows + 63) / 64;
    if (tiles == 0 || p.num_c == 0) return hipSuccess;
    if (p.num_c > kMaxErrorConstants) return hipErrorInvalidValue;
    // 8 blocks of 4 waves per CU over 256 CUs; each block strides over the tiles.
    const dim3 grid{unsigned(tiles < 2048 ? tiles : 2048)}, block{256u};
    if (dtype == 0) hipLaunchKernelGGL(quantize_error_kernel<0>, grid, block, 0, stream, p);
    else if (dtype == 1) hipLaunchKernelGGL(quantize_error_kernel<1>, grid, block, 0, stream, p);
    else hipLaunchKernelGGL(quantize_error_kernel<2>, grid, block, 0, stream, p);
    return hipGetLastError();
}

hipError_t launch_prepare_query(const void* q, int dtype, int64_t rows, uint8_t* q8, hipStream_t stream) {
    const int64_t blocks = (rows + 15) / 16;
    if (blocks == 0) return hipSuccess;
    if (blocks > 0x7FFFFFFF) return hipErrorInvalidValue;
    const dim3 grid{unsigned(blocks)}, block{256u};
    if (dtype == 0) hipLaunchKernelGGL(prepare_query_kernel<0>, grid, block, 0, stream, q, rows, q8);
    else if (dtype == 1) hipLaunchKernelGGL(prepare_query_kernel<1>, grid, block, 0, stream, q, rows, q8);
    else hipLaunchKernelGGL(prepare_query_kernel<2>, grid, block, 0, stream, q, rows, q8);
    return hipGetLastError();
}

}  // namespace uq
