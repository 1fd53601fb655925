// uq_decode.hip -- split-context decode attention over the FP4 cache
// (paper, Algorithm 1, "Decode"; section "Kernel Implementation in vLLM").
//
// decode_split_kernel: one 256-thread block (4 waves) per (partition,
// kv head, sequence).
//   prologue  the block rotates its G query heads with the in-register WHT
//             butterfly and casts them to FP8 E4M3 once, into LDS in the
//             lane order of the MFMA B operand; every wave keeps it in 8
//             VGPRs for the whole partition (the query is hoisted out of the
//             K-tile loop).
//   loop      each wave takes pairs of pages (32 tokens) round-robin.  Per
//             page and lane: one 16-byte load of K codes, one of V codes,
//             one scale byte for K and one scale dword for V, prefetched one
//             iteration ahead into registers.
//             QK^T: one v_mfma_scale_f32_16x16x128_f8f6f4 per page, the FP4
//             K tile as operand A (rows = tokens) with its UE8M0 bytes as
//             the A scales, the FP8 query as operand B (columns = query
//             heads) with scale byte 127 (1.0).  Dequantisation is folded
//             into the instruction.
//             Online softmax in the log2 domain with a lazy rescale (the
//             running max only moves when it grows by more than 8).
//             V: v_cvt_scalef32_pk_bf16_fp4 turns code pairs into exact
//             BF16 values with the token's scale; byte permutes build the
//             A operand of v_mfma_f32_16x16x32_bf16 (rows = channels, k =
//             tokens), and P enters as operand B split into a BF16 high
//             part and a BF16 residual, so the PV product carries ~16
//             significant bits of P.
//   epilogue  the 4 waves merge (max, sum, accumulators) through LDS and
//             the block writes one partial per query head.
// decode_reduce_kernel: merges the partitions of every (sequence, query
// head), divides by the softmax sum and, when V was stored rotated, maps
// the output back with the same butterfly (R is its own inverse).
#include "uq_device.hpp"
#include "uq_internal.hpp"

namespace uq {

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr float kLazyRescale = 8.0f;   // log2 units
constexpr int kAccStride = 129;        // LDS row stride (floats) of the merge buffer

struct PageRegs {
    uint4 kc;      // K codes, this lane's 16 bytes: token lane%16, group lane/16
    uint4 vc;      // V codes, 16 bytes: tokens 4*(lane/16)+0..3, channels 8*(lane%16)+0..7
    uint32_t ks;   // K scale byte of (token lane%16, group lane/16)
    uint32_t vs;   // V scale bytes of tokens 4*(lane/16)+0..3, group (lane%16)/4
};

__device__ __forceinline__ void load_page(const uint8_t* __restrict__ codes, const uint8_t* __restrict__ scales,
                                          int64_t tile, int lane, PageRegs& r) {
    const uint8_t* kc = codes + tile * kTileCodes;
    r.kc = *reinterpret_cast<const uint4*>(kc + 16 * lane);
    r.vc = *reinterpret_cast<const uint4*>(kc + kTileCodes + 16 * lane);
    const uint8_t* sc = scales + tile * kTileScales;
    r.ks = sc[lane];
    r.vs = *reinterpret_cast<const uint32_t*>(sc + kTileScales + ((lane & 15) >> 2) * 16 + 4 * (lane >> 4));
}

// Exchange with the lane 16 (or 32) positions away: after
// v_permlane16_swap a b (a = b = x on entry) the pair (a, b) holds x of this
// lane and of lane l^16 in some order, and v_permlane32_swap does the same
// for l^32.  Written as inline assembly on two distinct registers: the
// compiler builtins fold the two results into one when both inputs are the
// same value, which loses the exchange.
__device__ __forceinline__ void swap16(float& a, float& b) {
    asm volatile("s_nop 1\n\tv_permlane16_swap_b32 %0, %1" : "+v"(a), "+v"(b));
}
__device__ __forceinline__ void swap32(float& a, float& b) {
    asm volatile("s_nop 1\n\tv_permlane32_swap_b32 %0, %1" : "+v"(a), "+v"(b));
}

__device__ __forceinline__ float max_across_groups(float x) {
    // lanes l, l^16, l^32, l^48 hold the same query head
    float a = x, b = x;
    swap16(a, b);
    x = __builtin_fmaxf(a, b);
    a = x;
    b = x;
    swap32(a, b);
    return __builtin_fmaxf(a, b);
}

__device__ __forceinline__ float sum_across_groups(float x) {
    float a = x, b = x;
    swap16(a, b);
    x = a + b;
    a = x;
    b = x;
    swap32(a, b);
    return a + b;
}

__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
    v2bf h = {__bf16(a), __bf16(b)};
    return __builtin_bit_cast(uint32_t, h);
}

__device__ __forceinline__ float bf16_lo_f32(uint32_t w) { return bits_f32(w << 16); }
__device__ __forceinline__ float bf16_hi_f32(uint32_t w) { return bits_f32(w & 0xFFFF0000u); }

template <int DT>
__device__ __forceinline__ void load_q8(const void* q, int64_t elem, float (&x)[8]) {
    if constexpr (DT == 0) {
        const float4* p = reinterpret_cast<const float4*>(static_cast<const float*>(q) + elem);
        float4 a = p[0], b = p[1];
        x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
        x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
    } else {
        const uint4 w = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(q) + elem);
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

// Page ids of one wave, 64 at a time: lane j holds the id of the wave's
// page 2*(32*chunk + j/2) + j%2 counted in its own iteration order
// (iteration k of wave w covers partition pages 2*(w + 4k) and +1).
__device__ __forceinline__ int32_t load_page_ids(const int32_t* __restrict__ pt_row, int first_page, int n_pages,
                                                 int wave, int chunk, int lane, int64_t num_pages) {
    const int k = 32 * chunk + (lane >> 1);
    const int pg = 2 * (wave + kWaves * k) + (lane & 1);
    int32_t id = 0;
    if (pg < n_pages) id = pt_row[first_page + pg];
    if (id < 0 || int64_t(id) >= num_pages) id = 0;   // out-of-range ids never leave the pools
    return id;
}

// PV for the channel pair selected by byte BS of every V dword: channels
// 8n+2BS (block 2BS, low halves) and 8n+2BS+1 (block 2BS+1, high halves).
// The converted BF16 values of tokens (t, t+1) are paired by byte permutes
// into the k-slot order of the P operand.
template <int BS>
__device__ __forceinline__ void pv_pair(const uint32_t (&v0d)[4], const uint32_t (&v1d)[4], const float (&sc0)[4],
                                        const float (&sc1)[4], const v8bf& Phi, const v8bf& Plo, v4f& acc_e,
                                        v4f& acc_o) {
    uint32_t cv0[4], cv1[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        cv0[t] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(v0d[t], sc0[t], BS));
        cv1[t] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(v1d[t], sc1[t], BS));
    }
    const uint4 ae = {__builtin_amdgcn_perm(cv0[1], cv0[0], 0x05040100u), __builtin_amdgcn_perm(cv0[3], cv0[2], 0x05040100u),
                      __builtin_amdgcn_perm(cv1[1], cv1[0], 0x05040100u), __builtin_amdgcn_perm(cv1[3], cv1[2], 0x05040100u)};
    const uint4 ao = {__builtin_amdgcn_perm(cv0[1], cv0[0], 0x07060302u), __builtin_amdgcn_perm(cv0[3], cv0[2], 0x07060302u),
                      __builtin_amdgcn_perm(cv1[1], cv1[0], 0x07060302u), __builtin_amdgcn_perm(cv1[3], cv1[2], 0x07060302u)};
    const v8bf Ve = __builtin_bit_cast(v8bf, ae);
    const v8bf Vo = __builtin_bit_cast(v8bf, ao);
    acc_e = __builtin_amdgcn_mfma_f32_16x16x32_bf16(Ve, Phi, acc_e, 0, 0, 0);
    acc_e = __builtin_amdgcn_mfma_f32_16x16x32_bf16(Ve, Plo, acc_e, 0, 0, 0);
    acc_o = __builtin_amdgcn_mfma_f32_16x16x32_bf16(Vo, Phi, acc_o, 0, 0, 0);
    acc_o = __builtin_amdgcn_mfma_f32_16x16x32_bf16(Vo, Plo, acc_o, 0, 0, 0);
}

__global__ void __launch_bounds__(kThreads) decode_split_kernel(DecodeParams p) {
    const int part = blockIdx.x;
    const int hk = blockIdx.y;
    const int b = blockIdx.z;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int G = p.group;

    int ctx = p.context_lens[b];
    ctx = ctx < p.max_context ? ctx : p.max_context;
    const int start = part * p.partition_tokens;
    if (start >= ctx) return;   // whole block: nothing of this sequence here
    const int end = (start + p.partition_tokens) < ctx ? (start + p.partition_tokens) : ctx;

    __shared__ __attribute__((aligned(16))) uint8_t q_lds[64 * 32];
    __shared__ float red_acc[kWaves][16 * kAccStride];
    __shared__ float red_m[kWaves][16];
    __shared__ float red_l[kWaves][16];

    // ---------------- query prologue: rotate, cast to FP8, B-operand order
    {
        const int r = tid >> 4;        // query head within the group
        const int L = tid & 15;        // channels 8L..8L+7
        uint32_t lo = 0, hi = 0;
        if (r < G) {
            const int hq = hk * G + r;
            const int64_t elem = (int64_t(b) * p.num_q_heads + hq) * kHeadDim + 8 * L;
            if (p.q_dtype == 3) {
                const uint2 w = *reinterpret_cast<const uint2*>(static_cast<const uint8_t*>(p.q) + elem);
                lo = w.x;
                hi = w.y;
            } else {
                float x[8];
                if (p.q_dtype == 0) load_q8<0>(p.q, elem, x);
                else if (p.q_dtype == 1) load_q8<1>(p.q, elem, x);
                else load_q8<2>(p.q, elem, x);
                wht128_x8(x, L);
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    lo |= e4m3_byte(x[i]) << (8 * i);
                    hi |= e4m3_byte(x[i + 4]) << (8 * i);
                }
            }
        }
        // FP8 operand of the 16x16x128 scaled MFMA: lane 16*g + n holds
        // column n, channels 16g..16g+15 in bytes 0..15 and 64+16g..64+16g+15
        // in bytes 16..31.
        const int ch = 8 * L;
        const int g = (ch & 63) >> 4;
        const int e0 = (ch & 15) + (ch >= 64 ? 16 : 0);
        *reinterpret_cast<uint2*>(q_lds + (g * 16 + r) * 32 + e0) = make_uint2(lo, hi);
    }
    __syncthreads();
    v8i qop;
    {
        const uint4* src = reinterpret_cast<const uint4*>(q_lds + lane * 32);
        const uint4 a = src[0], c = src[1];
        qop = v8i{int(a.x), int(a.y), int(a.z), int(a.w), int(c.x), int(c.y), int(c.z), int(c.w)};
    }

    // ---------------- main loop over page pairs
    const int first_page = start >> 4;
    const int n_pages = (end - start + 15) >> 4;
    const int n_iter = (n_pages + 1) >> 1;
    const int n_local = wave < n_iter ? (n_iter - wave + kWaves - 1) / kWaves : 0;
    const int32_t* pt_row = p.page_table + int64_t(b) * p.max_pages_per_seq;
    const int g4 = lane >> 4;           // lane group: tokens 4*g4..4*g4+3 of each page
    const float sl2 = p.scale_log2;

    float m_run = -__builtin_inff();
    float l_run = 0.0f;
    v4f acc[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[j] = v4f{0.f, 0.f, 0.f, 0.f};

    if (n_local > 0) {
        int32_t ids = load_page_ids(pt_row, first_page, n_pages, wave, 0, lane, p.num_pages);
        int32_t ids_next = 0;
        if (n_local > 32) ids_next = load_page_ids(pt_row, first_page, n_pages, wave, 1, lane, p.num_pages);
        PageRegs c0, c1;
        {
            const int64_t id0 = __builtin_amdgcn_readlane(ids, 0);
            const int64_t id1 = __builtin_amdgcn_readlane(ids, 1);
            load_page(p.codes, p.scales, id0 * p.num_kv_heads * 2 + hk * 2, lane, c0);
            load_page(p.codes, p.scales, id1 * p.num_kv_heads * 2 + hk * 2, lane, c1);
        }
        for (int k = 0; k < n_local; ++k) {
            // prefetch the next pair (the last iteration re-reads its own pair)
            const int kn = (k + 1 < n_local) ? k + 1 : k;
            if ((kn & 31) == 0 && kn != k) {
                ids = ids_next;
                if (kn + 32 < n_local)
                    ids_next = load_page_ids(pt_row, first_page, n_pages, wave, (kn >> 5) + 1, lane, p.num_pages);
            }
            PageRegs n0, n1;
            {
                const int s = 2 * (kn & 31);
                const int64_t id0 = __builtin_amdgcn_readlane(ids, s);
                const int64_t id1 = __builtin_amdgcn_readlane(ids, s + 1);
                load_page(p.codes, p.scales, id0 * p.num_kv_heads * 2 + hk * 2, lane, n0);
                load_page(p.codes, p.scales, id1 * p.num_kv_heads * 2 + hk * 2, lane, n1);
            }

            // ---- QK^T: S^T[token][head] per page, FP4 x FP8 with the UE8M0 bytes as A scales
            const v4f zero = {0.f, 0.f, 0.f, 0.f};
            const v8i ka0 = {int(c0.kc.x), int(c0.kc.y), int(c0.kc.z), int(c0.kc.w), 0, 0, 0, 0};
            const v8i ka1 = {int(c1.kc.x), int(c1.kc.y), int(c1.kc.z), int(c1.kc.w), 0, 0, 0, 0};
            const v4f s0 = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(ka0, qop, zero, 4, 0, 0, int(c0.ks), 0, 127);
            const v4f s1 = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(ka1, qop, zero, 4, 0, 0, int(c1.ks), 0, 127);

            float x[8];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                x[i] = s0[i] * sl2;
                x[4 + i] = s1[i] * sl2;
            }
            uint32_t vs0 = c0.vs, vs1 = c1.vs;
            const int it = wave + kWaves * k;
            const int tok0 = start + 32 * it + 4 * g4;   // token of x[0]; x[4] is tok0 + 16
            if (start + 32 * it + 32 > end) {
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    if (tok0 + i >= end) { x[i] = -__builtin_inff(); vs0 &= ~(0xFFu << (8 * i)); }
                    if (tok0 + 16 + i >= end) { x[4 + i] = -__builtin_inff(); vs1 &= ~(0xFFu << (8 * i)); }
                }
            }

            // ---- online softmax (log2 domain), lazy rescale
            float mloc = x[0];
#pragma unroll
            for (int i = 1; i < 8; ++i) mloc = __builtin_fmaxf(mloc, x[i]);
            mloc = max_across_groups(mloc);
            if (mloc > m_run + kLazyRescale) {
                const float alpha = __builtin_amdgcn_exp2f(m_run - mloc);
                l_run *= alpha;
#pragma unroll
                for (int j = 0; j < 8; ++j) acc[j] *= alpha;
                m_run = mloc;
            }
            float pr[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                pr[i] = __builtin_amdgcn_exp2f(x[i] - m_run);
                l_run += pr[i];
            }
            uint32_t phi[4], plo[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                phi[r] = pack_bf16x2(pr[2 * r], pr[2 * r + 1]);
                plo[r] = pack_bf16x2(pr[2 * r] - bf16_lo_f32(phi[r]), pr[2 * r + 1] - bf16_hi_f32(phi[r]));
            }
            const v8bf Phi = __builtin_bit_cast(v8bf, uint4{phi[0], phi[1], phi[2], phi[3]});
            const v8bf Plo = __builtin_bit_cast(v8bf, uint4{plo[0], plo[1], plo[2], plo[3]});

            // ---- V: FP4 -> BF16 with the token scale, then PV on bf16 MFMA
            const uint32_t v0d[4] = {c0.vc.x, c0.vc.y, c0.vc.z, c0.vc.w};
            const uint32_t v1d[4] = {c1.vc.x, c1.vc.y, c1.vc.z, c1.vc.w};
            float sc0[4], sc1[4];
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                sc0[t] = ue8m0_to_f32(vs0 >> (8 * t));
                sc1[t] = ue8m0_to_f32(vs1 >> (8 * t));
            }
            pv_pair<0>(v0d, v1d, sc0, sc1, Phi, Plo, acc[0], acc[1]);
            pv_pair<1>(v0d, v1d, sc0, sc1, Phi, Plo, acc[2], acc[3]);
            pv_pair<2>(v0d, v1d, sc0, sc1, Phi, Plo, acc[4], acc[5]);
            pv_pair<3>(v0d, v1d, sc0, sc1, Phi, Plo, acc[6], acc[7]);
            c0 = n0;
            c1 = n1;
        }
    }

    // ---------------- merge the 4 waves through LDS, write the partial
    l_run = sum_across_groups(l_run);
    const int n = lane & 15;
    if (g4 == 0) {
        red_m[wave][n] = m_run;
        red_l[wave][n] = l_run;
    }
    // acc[j][i] of lane (n, g4) is O^T[channel 8*(4*g4+i)+j][head n]
#pragma unroll
    for (int j = 0; j < 8; ++j) {
#pragma unroll
        for (int i = 0; i < 4; ++i) red_acc[wave][n * kAccStride + 32 * g4 + 8 * i + j] = acc[j][i];
    }
    __syncthreads();
    {
        const int r = tid >> 4;   // query head within the group
        const int L = tid & 15;   // channels 8L..8L+7
        if (r < G) {
            float M = red_m[0][r];
#pragma unroll
            for (int w = 1; w < kWaves; ++w) M = __builtin_fmaxf(M, red_m[w][r]);
            float f[kWaves];
            float lsum = 0.f;
#pragma unroll
            for (int w = 0; w < kWaves; ++w) {
                f[w] = __builtin_amdgcn_exp2f(red_m[w][r] - M);
                lsum += f[w] * red_l[w][r];
            }
            float o[8];
#pragma unroll
            for (int c = 0; c < 8; ++c) {
                float s = 0.f;
#pragma unroll
                for (int w = 0; w < kWaves; ++w) s += f[w] * red_acc[w][r * kAccStride + 8 * L + c];
                o[c] = s;
            }
            const int hq = hk * G + r;
            const int64_t row = (int64_t(b) * p.num_q_heads + hq) * p.num_partitions + part;
            float4* dst = reinterpret_cast<float4*>(p.part_acc + row * kHeadDim + 8 * L);
            dst[0] = make_float4(o[0], o[1], o[2], o[3]);
            dst[1] = make_float4(o[4], o[5], o[6], o[7]);
            if (L == 0) *reinterpret_cast<float2*>(p.part_ml + row * 2) = make_float2(M, lsum);
        }
    }
}

__global__ void __launch_bounds__(256) decode_reduce_kernel(DecodeParams p) {
    const int hk = blockIdx.x;
    const int b = blockIdx.y;
    const int r = threadIdx.x >> 4;
    const int L = threadIdx.x & 15;
    if (r >= p.group) return;   // whole 16-lane rows leave together
    const int hq = hk * p.group + r;
    int ctx = p.context_lens[b];
    ctx = ctx < p.max_context ? ctx : p.max_context;
    const int np = ctx > 0 ? (ctx + p.partition_tokens - 1) / p.partition_tokens : 0;
    const int64_t row0 = (int64_t(b) * p.num_q_heads + hq) * p.num_partitions;

    float o[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    if (np > 0) {
        float M = -__builtin_inff();
        for (int q = 0; q < np; ++q) M = __builtin_fmaxf(M, p.part_ml[(row0 + q) * 2]);
        float lsum = 0.f;
        for (int q = 0; q < np; ++q) {
            const float2 ml = *reinterpret_cast<const float2*>(p.part_ml + (row0 + q) * 2);
            const float f = __builtin_amdgcn_exp2f(ml.x - M);
            lsum += f * ml.y;
            const float4* src = reinterpret_cast<const float4*>(p.part_acc + (row0 + q) * kHeadDim + 8 * L);
            const float4 a = src[0], c = src[1];
            o[0] += f * a.x; o[1] += f * a.y; o[2] += f * a.z; o[3] += f * a.w;
            o[4] += f * c.x; o[5] += f * c.y; o[6] += f * c.z; o[7] += f * c.w;
        }
        const float inv = 1.0f / lsum;
#pragma unroll
        for (int i = 0; i < 8; ++i) o[i] *= inv;
        if (p.rotate_v) wht128_x8(o, L);
    }
    const int64_t ob = (int64_t(b) * p.num_q_heads + hq) * kHeadDim + 8 * L;
    if (p.out_dtype == 0) {
        float4* dst = reinterpret_cast<float4*>(static_cast<float*>(p.out) + ob);
        dst[0] = make_float4(o[0], o[1], o[2], o[3]);
        dst[1] = make_float4(o[4], o[5], o[6], o[7]);
    } else {
        *reinterpret_cast<uint4*>(static_cast<uint16_t*>(p.out) + ob) =
            uint4{pack_bf16x2(o[0], o[1]), pack_bf16x2(o[2], o[3]), pack_bf16x2(o[4], o[5]), pack_bf16x2(o[6], o[7])};
    }
}

hipError_t launch_decode_split(const DecodeParams& p, hipStream_t stream) {
    dim3 grid(unsigned(p.num_partitions), unsigned(p.num_kv_heads), unsigned(p.batch));
    hipLaunchKernelGGL(decode_split_kernel, grid, dim3(kThreads), 0, stream, p);
    return hipGetLastError();
}

hipError_t launch_decode_reduce(const DecodeParams& p, hipStream_t stream) {
    dim3 grid(unsigned(p.num_kv_heads), unsigned(p.batch));
    hipLaunchKernelGGL(decode_reduce_kernel, grid, dim3(256), 0, stream, p);
    return hipGetLastError();
}

}  // namespace uq
