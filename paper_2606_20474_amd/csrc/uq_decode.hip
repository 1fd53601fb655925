// uq_decode.hip -- split-context decode attention over the FP4 cache
// (paper, Algorithm 1, "Decode"; section "Kernel Implementation in vLLM").
//
// decode_kernel: one 256-thread block (4 waves) per (partition, kv head,
// sequence).
//   prologue  the block rotates its G query heads with the in-register WHT
//             butterfly and casts them to FP8 E4M3 once, into LDS in the
//             lane order of the MFMA B operand; every wave keeps it in 8
//             VGPRs for the whole partition (the query is hoisted out of the
//             K-tile loop).
//   loop      each wave takes pairs of pages (32 tokens) round-robin and
//             stages them through its own 2-slot LDS ring with
//             global_load_lds_dwordx4 (16 bytes per lane, 1 KiB per
//             instruction): as soon as a slot has been read into registers
//             it is refilled with the pair two iterations ahead, so two
//             pairs (8.7 KB) per wave are in flight while one is computed.
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
//   epilogue  the 4 waves merge (max, sum, accumulators) through LDS.  A
//             sequence that fits one partition is finished in place;
//             otherwise the block writes one partial per query head.
// merge_kernel: merges the partitions of every (sequence, query head),
// divides by the softmax sum and, when V was stored rotated, maps the output
// back with the same butterfly (R is its own inverse).  A separate launch:
// merging in the last-arriving block needs cross-XCD visibility of the
// other blocks' partials, and both ways to get it (an L2 writeback and
// invalidate per block, or write-through stores) measured slower than the
// second launch.
#include "uq_device.hpp"
#include "uq_internal.hpp"

namespace uq {

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr float kLazyRescale = 8.0f;   // log2 units
constexpr int kAccStride = 129;        // LDS row stride (floats) of the merge buffer

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

// Per-wave staging ring in LDS: 2 stages of one iteration (2 pages) each:
//   [K page0 1024][V page0 1024][K page1 1024][V page1 1024][scales page0 128][scales page1 128]
constexpr int kStageBytes = 4 * kTileCodes + 4 * kTileScales;   // 4352
constexpr int kRingBytes = 2 * kStageBytes;                      // per wave
constexpr int kMergeBytes = kWaves * 16 * kAccStride * 4;
static_assert(kMergeBytes <= kWaves * kRingBytes, "merge buffer aliases the staging rings");

typedef __attribute__((address_space(3))) void* lds_ptr_t;

// Asynchronous copy of one iteration (two pages of one kv head) from HBM
// into an LDS stage with global_load_lds_dwordx4: every lane moves 16 bytes
// and the hardware places lane i's bytes at stage + 16 i, so each 1 KiB tile
// lands in lane order.  Five instructions per stage; the scale blocks of both
// pages (2 x 128 bytes) are moved by lanes 0..15.
__device__ __forceinline__ void stage_issue(uint8_t* stage, const uint8_t* __restrict__ codes,
                                            const uint8_t* __restrict__ scales, int64_t tile0, int64_t tile1,
                                            int lane) {
    const uint8_t* k0 = codes + tile0 * kTileCodes + 16 * lane;
    const uint8_t* k1 = codes + tile1 * kTileCodes + 16 * lane;
    __builtin_amdgcn_global_load_lds(k0, (lds_ptr_t)(stage), 16, 0, 0);
    __builtin_amdgcn_global_load_lds(k0 + kTileCodes, (lds_ptr_t)(stage + kTileCodes), 16, 0, 0);
    __builtin_amdgcn_global_load_lds(k1, (lds_ptr_t)(stage + 2 * kTileCodes), 16, 0, 0);
    __builtin_amdgcn_global_load_lds(k1 + kTileCodes, (lds_ptr_t)(stage + 3 * kTileCodes), 16, 0, 0);
    if (lane < 16) {
        const int64_t t = lane < 8 ? tile0 : tile1;
        const uint8_t* sc = scales + t * kTileScales + 16 * (lane & 7);
        __builtin_amdgcn_global_load_lds(sc, (lds_ptr_t)(stage + 4 * kTileCodes), 16, 0, 0);
    }
}
constexpr int kDmaPerStage = 5;

// Wait until at most N of this wave's vector-memory loads are outstanding
// (loads complete in issue order, so the older stage is then in LDS).
template <int N>
__device__ __forceinline__ void wait_vmem() {
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

struct StageRegs {
    uint4 k0, v0, k1, v1;   // this lane's 16 bytes of each tile
    uint32_t ks0, ks1;      // K scale byte (token lane%16, group lane/16)
    uint32_t vs0, vs1;      // V scale bytes of tokens 4*(lane/16)+0..3, group (lane%16)/4
};

// Read this lane's operands of one stage.  The reads are inline assembly so
// that the compiler does not guard them with a wait for every outstanding
// LDS copy; the caller has already waited for this stage's copies, and the
// trailing lgkmcnt(0) makes the results safe to use.
__device__ __forceinline__ StageRegs stage_read(uint32_t stage_addr, uint32_t off_codes, uint32_t off_ks,
                                                uint32_t off_vs) {
    StageRegs r;
    const uint32_t ac = stage_addr + off_codes;
    const uint32_t ak = stage_addr + off_ks;
    const uint32_t av = stage_addr + off_vs;
    asm volatile(
        "ds_read_b128 %0, %8\n\t"
        "ds_read_b128 %1, %8 offset:1024\n\t"
        "ds_read_b128 %2, %8 offset:2048\n\t"
        "ds_read_b128 %3, %8 offset:3072\n\t"
        "ds_read_u8 %4, %9 offset:4096\n\t"
        "ds_read_u8 %5, %9 offset:4224\n\t"
        "ds_read_b32 %6, %10 offset:4096\n\t"
        "ds_read_b32 %7, %10 offset:4224\n\t"
        "s_waitcnt lgkmcnt(0)"
        : "=&v"(r.k0), "=&v"(r.v0), "=&v"(r.k1), "=&v"(r.v1), "=&v"(r.ks0), "=&v"(r.ks1), "=&v"(r.vs0), "=&v"(r.vs1)
        : "v"(ac), "v"(ak), "v"(av)
        : "memory");
    return r;
}

__device__ __forceinline__ void write_out(const DecodeParams& p, int64_t row, int L, const float (&o)[8]) {
    const int64_t ob = row * kHeadDim + 8 * L;
    if (p.out_dtype == 0) {
        float4* dst = reinterpret_cast<float4*>(static_cast<float*>(p.out) + ob);
        dst[0] = make_float4(o[0], o[1], o[2], o[3]);
        dst[1] = make_float4(o[4], o[5], o[6], o[7]);
    } else {
        *reinterpret_cast<uint4*>(static_cast<uint16_t*>(p.out) + ob) =
            uint4{pack_bf16x2(o[0], o[1]), pack_bf16x2(o[2], o[3]), pack_bf16x2(o[4], o[5]), pack_bf16x2(o[6], o[7])};
    }
}

__global__ void __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(4, 4))) decode_kernel(DecodeParams p) {
    const int part = blockIdx.x;
    const int hk = blockIdx.y;
    const int b = blockIdx.z;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform: scalar control flow
    const int G = p.group;

    int ctx = p.context_lens[b];
    ctx = ctx < p.max_context ? ctx : p.max_context;
    const int start = part * p.partition_tokens;
    if (start >= ctx) {
        // nothing of this sequence here; an empty context still gets its zero output
        if (ctx <= 0 && part == 0 && (tid >> 4) < G) {
            const float z[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
            write_out(p, int64_t(b) * p.num_q_heads + hk * G + (tid >> 4), tid & 15, z);
        }
        return;
    }
    const int end = (start + p.partition_tokens) < ctx ? (start + p.partition_tokens) : ctx;
    const int np_b = (ctx + p.partition_tokens - 1) / p.partition_tokens;

    __shared__ __attribute__((aligned(16))) uint8_t smem[kWaves * kRingBytes];
    __shared__ __attribute__((aligned(16))) uint8_t q_lds[64 * 32];
    __shared__ float red_m[kWaves][16];
    __shared__ float red_l[kWaves][16];

    // ---------------- query load first (its latency overlaps the page walk set-up)
    const int qr = tid >> 4;        // query head within the group
    const int qL = tid & 15;        // channels 8*qL..8*qL+7
    float qx[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    uint32_t qlo = 0, qhi = 0;
    if (qr < G) {
        const int64_t elem = (int64_t(b) * p.num_q_heads + hk * G + qr) * kHeadDim + 8 * qL;
        if (p.q_dtype == 3) {
            const uint2 w = *reinterpret_cast<const uint2*>(static_cast<const uint8_t*>(p.q) + elem);
            qlo = w.x;
            qhi = w.y;
        } else if (p.q_dtype == 0) {
            load_q8<0>(p.q, elem, qx);
        } else if (p.q_dtype == 1) {
            load_q8<1>(p.q, elem, qx);
        } else {
            load_q8<2>(p.q, elem, qx);
        }
    }

    // ---------------- page walk set-up and the first two stages in flight
    const int first_page = start >> 4;
    const int n_pages = (end - start + 15) >> 4;
    const int n_iter = (n_pages + 1) >> 1;
    const int n_local = wave < n_iter ? (n_iter - wave + kWaves - 1) / kWaves : 0;
    const int32_t* pt_row = p.page_table + int64_t(b) * p.max_pages_per_seq;
    const int g4 = lane >> 4;           // lane group: tokens 4*g4..4*g4+3 of each page
    const int n = lane & 15;
    uint8_t* ring = smem + wave * kRingBytes;
    const uint32_t ring_addr = uint32_t(reinterpret_cast<uintptr_t>((lds_ptr_t)ring));
    const uint32_t off_codes = 16 * lane;
    const uint32_t off_ks = lane;
    const uint32_t off_vs = kTileScales + (n >> 2) * 16 + 4 * g4;
    const int64_t head_tile = int64_t(hk) * 2;
    const int64_t tiles_per_page = int64_t(p.num_kv_heads) * 2;

    int32_t ids = 0, ids_next = 0;
    if (n_local > 0) {
        ids = load_page_ids(pt_row, first_page, n_pages, wave, 0, lane, p.num_pages);
        if (n_local > 32) ids_next = load_page_ids(pt_row, first_page, n_pages, wave, 1, lane, p.num_pages);
        for (int s = 0; s < 2 && s < n_local; ++s) {
            const int64_t id0 = __builtin_amdgcn_readlane(ids, 2 * s);
            const int64_t id1 = __builtin_amdgcn_readlane(ids, 2 * s + 1);
            stage_issue(ring + s * kStageBytes, p.codes, p.scales, id0 * tiles_per_page + head_tile,
                        id1 * tiles_per_page + head_tile, lane);
        }
    }

    // ---------------- query prologue: rotate, cast to FP8, B-operand order
    if (qr < G && p.q_dtype != 3) {
        wht128_x8(qx, qL);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            qlo |= e4m3_byte(qx[i]) << (8 * i);
            qhi |= e4m3_byte(qx[i + 4]) << (8 * i);
        }
    }
    {
        // FP8 operand of the 16x16x128 scaled MFMA: lane 16*g + n holds
        // column n, channels 16g..16g+15 in bytes 0..15 and 64+16g..64+16g+15
        // in bytes 16..31.  Rows qr >= G stay zero.
        const int ch = 8 * qL;
        const int g = (ch & 63) >> 4;
        const int e0 = (ch & 15) + (ch >= 64 ? 16 : 0);
        *reinterpret_cast<uint2*>(q_lds + (g * 16 + qr) * 32 + e0) = make_uint2(qlo, qhi);
    }
    __syncthreads();
    v8i qop;
    {
        const uint4* src = reinterpret_cast<const uint4*>(q_lds + lane * 32);
        const uint4 a = src[0], c = src[1];
        qop = v8i{int(a.x), int(a.y), int(a.z), int(a.w), int(c.x), int(c.y), int(c.z), int(c.w)};
    }

    const float sl2 = p.scale_log2;
    float m_run = -__builtin_inff();
    float l_run = 0.0f;
    v4f acc[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[j] = v4f{0.f, 0.f, 0.f, 0.f};

    // ---------------- main loop: one stage (2 pages, 32 tokens) per iteration
    for (int k = 0; k < n_local; ++k) {
        if (k + 1 < n_local) wait_vmem<kDmaPerStage>();
        else wait_vmem<0>();
        const uint32_t slot = uint32_t(k & 1);
        const StageRegs c = stage_read(ring_addr + slot * kStageBytes, off_codes, off_ks, off_vs);
        if (k + 2 < n_local) {
            // refill this slot with iteration k+2 while iteration k computes
            const int kn = k + 2;
            if ((kn & 31) == 0) {
                ids = ids_next;
                if (kn + 32 < n_local)
                    ids_next = load_page_ids(pt_row, first_page, n_pages, wave, (kn >> 5) + 1, lane, p.num_pages);
            }
            const int s = 2 * (kn & 31);
            const int64_t id0 = __builtin_amdgcn_readlane(ids, s);
            const int64_t id1 = __builtin_amdgcn_readlane(ids, s + 1);
            stage_issue(ring + slot * kStageBytes, p.codes, p.scales, id0 * tiles_per_page + head_tile,
                        id1 * tiles_per_page + head_tile, lane);
        }

        // ---- QK^T: S^T[token][head] per page, FP4 x FP8 with the UE8M0 bytes as A scales
        const v4f zero = {0.f, 0.f, 0.f, 0.f};
        const v8i ka0 = {int(c.k0.x), int(c.k0.y), int(c.k0.z), int(c.k0.w), 0, 0, 0, 0};
        const v8i ka1 = {int(c.k1.x), int(c.k1.y), int(c.k1.z), int(c.k1.w), 0, 0, 0, 0};
        const v4f s0 = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(ka0, qop, zero, 4, 0, 0, int(c.ks0), 0, 127);
        const v4f s1 = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(ka1, qop, zero, 4, 0, 0, int(c.ks1), 0, 127);

        // raw scores; the softmax scale (times log2 e, positive) is applied
        // inside the exponent's fma
        float x[8];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            x[i] = s0[i];
            x[4 + i] = s1[i];
        }
        uint32_t vs0 = c.vs0, vs1 = c.vs1;
        const int it = wave + kWaves * k;
        const int tok0 = start + 32 * it + 4 * g4;   // token of x[0]; x[4] is tok0 + 16
        if (start + 32 * it + 32 > end) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                if (tok0 + i >= end) { x[i] = -__builtin_inff(); vs0 &= ~(0xFFu << (8 * i)); }
                if (tok0 + 16 + i >= end) { x[4 + i] = -__builtin_inff(); vs1 &= ~(0xFFu << (8 * i)); }
            }
        }

        // ---- online softmax (log2 domain, m_run in scaled units), lazy rescale
        float smax = x[0];
#pragma unroll
        for (int i = 1; i < 8; ++i) smax = __builtin_fmaxf(smax, x[i]);
        const float mloc = max_across_groups(smax) * sl2;
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
            pr[i] = __builtin_amdgcn_exp2f(__builtin_fmaf(x[i], sl2, -m_run));
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
        const uint32_t v0d[4] = {c.v0.x, c.v0.y, c.v0.z, c.v0.w};
        const uint32_t v1d[4] = {c.v1.x, c.v1.y, c.v1.z, c.v1.w};
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
    }

    // ---------------- merge the 4 waves through LDS (the rings are free now)
    l_run = sum_across_groups(l_run);
    __syncthreads();
    float* red_acc = reinterpret_cast<float*>(smem);
    if (g4 == 0) {
        red_m[wave][n] = m_run;
        red_l[wave][n] = l_run;
    }
    // acc[j][i] of lane (n, g4) is O^T[channel 8*(4*g4+i)+j][head n]
#pragma unroll
    for (int j = 0; j < 8; ++j) {
#pragma unroll
        for (int i = 0; i < 4; ++i) red_acc[(wave * 16 + n) * kAccStride + 32 * g4 + 8 * i + j] = acc[j][i];
    }
    __syncthreads();

    const int r = tid >> 4;   // query head within the group
    const int L = tid & 15;   // channels 8L..8L+7
    const bool row_ok = r < G;
    const int hq = hk * G + r;
    float o[8];
    float M = 0.f, lsum = 0.f;
    if (row_ok) {
        M = red_m[0][r];
#pragma unroll
        for (int w = 1; w < kWaves; ++w) M = __builtin_fmaxf(M, red_m[w][r]);
        float f[kWaves];
#pragma unroll
        for (int w = 0; w < kWaves; ++w) {
            f[w] = __builtin_amdgcn_exp2f(red_m[w][r] - M);
            lsum += f[w] * red_l[w][r];
        }
#pragma unroll
        for (int cc = 0; cc < 8; ++cc) {
            float s = 0.f;
#pragma unroll
            for (int w = 0; w < kWaves; ++w) s += f[w] * red_acc[(w * 16 + r) * kAccStride + 8 * L + cc];
            o[cc] = s;
        }
    }

    if (np_b == 1) {
        // the whole context is in this block: finish here
        if (row_ok) {
            const float inv = 1.0f / lsum;
#pragma unroll
            for (int i = 0; i < 8; ++i) o[i] *= inv;
            if (p.rotate_v) wht128_x8(o, L);
            write_out(p, int64_t(b) * p.num_q_heads + hq, L, o);
        }
        return;
    }

    // several partitions: publish this one for the merge kernel
    if (row_ok) {
        const int64_t prow = (int64_t(b) * p.num_q_heads + hq) * p.num_partitions + part;
        float4* dst = reinterpret_cast<float4*>(p.part_acc + prow * kHeadDim + 8 * L);
        dst[0] = make_float4(o[0], o[1], o[2], o[3]);
        dst[1] = make_float4(o[4], o[5], o[6], o[7]);
        if (L == 0) *reinterpret_cast<float2*>(p.part_ml + prow * 2) = make_float2(M, lsum);
    }
}

// Merge the partitions of every (sequence, query head) with more than one:
// online over the partitions (loads independent of the running state, so
// they overlap), divide by the softmax sum, rotate back when V was stored
// rotated, write the output.  One 16-lane row per query head.
__global__ void __launch_bounds__(256) merge_kernel(DecodeParams p) {
    const int hk = blockIdx.x;
    const int b = blockIdx.y;
    const int r = threadIdx.x >> 4;
    const int L = threadIdx.x & 15;
    if (r >= p.group) return;   // whole 16-lane rows leave together
    int ctx = p.context_lens[b];
    ctx = ctx < p.max_context ? ctx : p.max_context;
    const int np = ctx > 0 ? (ctx + p.partition_tokens - 1) / p.partition_tokens : 0;
    if (np <= 1) return;        // finished by the decode kernel
    const int hq = hk * p.group + r;
    const int64_t row0 = (int64_t(b) * p.num_q_heads + hq) * p.num_partitions;
    float M = -__builtin_inff();
    float lsum = 0.f;
    float o[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll 4
    for (int q = 0; q < np; ++q) {
        const float2 ml = *reinterpret_cast<const float2*>(p.part_ml + (row0 + q) * 2);
        const float4* src = reinterpret_cast<const float4*>(p.part_acc + (row0 + q) * kHeadDim + 8 * L);
        const float4 a = src[0], c = src[1];
        const float Mn = __builtin_fmaxf(M, ml.x);
        const float fo = __builtin_amdgcn_exp2f(M - Mn);
        const float fn = __builtin_amdgcn_exp2f(ml.x - Mn);
        lsum = lsum * fo + ml.y * fn;
        o[0] = o[0] * fo + a.x * fn; o[1] = o[1] * fo + a.y * fn; o[2] = o[2] * fo + a.z * fn; o[3] = o[3] * fo + a.w * fn;
        o[4] = o[4] * fo + c.x * fn; o[5] = o[5] * fo + c.y * fn; o[6] = o[6] * fo + c.z * fn; o[7] = o[7] * fo + c.w * fn;
        M = Mn;
    }
    const float inv = 1.0f / lsum;
#pragma unroll
    for (int i = 0; i < 8; ++i) o[i] *= inv;
    if (p.rotate_v) wht128_x8(o, L);
    write_out(p, int64_t(b) * p.num_q_heads + hq, L, o);
}

hipError_t launch_decode_partials(const DecodeParams& p, hipStream_t stream) {
    const dim3 grid{unsigned(p.num_partitions), unsigned(p.num_kv_heads), unsigned(p.batch)};
    hipLaunchKernelGGL(decode_kernel, grid, dim3(kThreads), 0, stream, p);
    return hipGetLastError();
}

hipError_t launch_decode_merge(const DecodeParams& p, hipStream_t stream) {
    if (p.num_partitions <= 1) return hipSuccess;   // every sequence was finished in place
    const dim3 grid{unsigned(p.num_kv_heads), unsigned(p.batch)};
    hipLaunchKernelGGL(merge_kernel, grid, dim3(256), 0, stream, p);
    return hipGetLastError();
}

}  // namespace uq
