// uq_decode.hip -- split-context decode attention over a paged KV cache
// (paper, Algorithm 1, "Decode"; section "Kernel Implementation in vLLM").
//
// One kernel template serves the cache formats so that the comparison
// between them measures the format, not the kernel:
//   kFp4   the UltraQuant cache: FP4 E2M1 codes + UE8M0 scales per 32
//          channels, K (and V with rotate_v) Walsh-Hadamard rotated
//          (kFp4d64x2, kFp4d64, kFp4d256: the same cache at head sizes 64
//          and 256; kFp4d64x2 takes two KV heads per block);
//   kFp8   a plain FP8 E4M3 cache with one scale per tensor;
//   kBf16  a plain BF16 cache;
//   kTq4   the Ultra-TQ codebook cache (rotated K as 4-bit indices into 16
//          levels times a per-token norm; V as 4-bit uniform codes with a
//          BF16 (scale, zero) per 32 channels): K is decoded in registers
//          by byte-permute table lookups into BF16 levels, QK^T runs on
//          BF16 matrix instructions and each score is multiplied by its
//          token's norm; V is decoded with one fused multiply-add per
//          element into BF16.
//
// decode_kernel<F, S, WP, PROBE, W>: one block of W waves per (partition,
// kv head, sequence), in an XCD-aware linear order (kv head fastest); S ring
// slots per wave; WP: one wave per partition (below); PROBE: the same launch
// as the page-gather bandwidth probe (no query prologue, arithmetic or
// epilogue); W: the format's kWaves, or 8 on the wave grid of the FP4 and
// FP8 caches (see launch_waves).
//   prologue  the block loads its G query heads (G <= 16), rotates them
//             with the in-register WHT butterfly and casts them to FP8
//             E4M3 (FP4 cache), casts them to FP8 (FP8 cache) or to BF16
//             (BF16 cache), and stores them in LDS in the lane order of the
//             MFMA B operand; every wave keeps the operand in registers for
//             the whole partition (the query is hoisted out of the K-tile
//             loop).
//   loop      each wave takes pairs of pages (32 tokens) round-robin and
//             stages them through its own S-slot LDS ring (S = 2) with
//             global_load_lds_dwordx4 (16 bytes per lane, 1 KiB per
//             instruction; non-temporal for the pages of one sequence,
//             default policy for shared-prefix pages); a slot is refilled
//             with the pair S iterations ahead as soon as it has been read
//             into registers, so S pairs per wave are in flight while one
//             is computed.  The next 64
//             page ids are copied into LDS the same way, so the wave never
//             waits on a register load while pages are in flight.
//             QK^T: FP4 -- one v_mfma_scale_f32_16x16x128_f8f6f4 per page,
//             the FP4 K tile as operand A (rows = tokens) with its UE8M0
//             bytes as the A scales and the FP8 query as operand B (columns
//             = query heads): dequantisation is folded into the
//             instruction.  FP8 -- the same instruction with FP8 on both
//             sides.  BF16 -- four v_mfma_f32_16x16x32_bf16 per page.
//             Online softmax in the log2 domain with a lazy rescale (the
//             running max only moves when it grows by more than 8).
//             V: the hardware conversions v_cvt_scalef32_pk_bf16_fp4 (with
//             the token's UE8M0 scale) or v_cvt_scalef32_pk_bf16_fp8 turn
//             code pairs into exact BF16 values; byte permutes pair two
//             tokens per register for the A operand of
//             v_mfma_f32_16x16x32_bf16 (rows = channels, k = tokens).  P
//             enters as operand B split into a BF16 high part and a BF16
//             residual, so PV carries ~16 significant bits of P.
//   epilogue  the waves merge (max, sum, accumulators) through LDS.  A
//             sequence that fits one partition is finished in place;
//             otherwise the block writes one partial per query head.
// merge_kernel: merges the partitions of every (sequence, query head),
// divides by the softmax sum, applies the per-tensor V scale and, when V was
// stored rotated, maps the output back with the same butterfly (R is its
// own inverse).  A separate launch: merging in the last-arriving block needs
// cross-XCD visibility of the other blocks' partials, and both ways to get
// it (an L2 writeback and invalidate per block, or write-through stores)
// measured slower than the second launch.
#include "uq_device.hpp"
#include "uq_internal.hpp"

namespace uq {

constexpr float kLazyRescale = 8.0f;   // log2 units
constexpr int kWaitVmcnt0 = 0x0F70;    // s_waitcnt vmcnt(0) expcnt(7) lgkmcnt(15) (gfx9 encoding)

// Per-format constants.  kTile: bytes of one (page, kv head) K or V tile;
// kScaleBlock: scale bytes per (page, kv head) for K and V together.
template <int F> struct Fmt;
// kWaves: waves per block (the FP4 and FP8 caches run blocks of 8 waves on
// the wave grid, see launch_waves); kOccupancy: waves per SIMD the LDS footprint allows
// (160 KiB per CU), which sets the register budget.
template <> struct Fmt<kFp4> {
    static constexpr int kTile = 1024;
    static constexpr int kScaleBlock = 2 * kTileScales;
    static constexpr int kWaves = 4;
    static constexpr int kOccupancy = 4;
};
template <> struct Fmt<kFp8> {
    static constexpr int kTile = 2048;
    static constexpr int kScaleBlock = 0;
    static constexpr int kWaves = 4;
    static constexpr int kOccupancy = 2;
};
template <> struct Fmt<kBf16> {
    static constexpr int kTile = 4096;
    static constexpr int kScaleBlock = 0;
    static constexpr int kWaves = 2;
    static constexpr int kOccupancy = 1;
};
// The FP4 cache at head sizes 64 and 256: tiles of 8 D code bytes and D/2
// scale bytes per (page, head, K|V).
template <> struct Fmt<kFp4d64> {
    static constexpr int kTile = 512;
    static constexpr int kScaleBlock = 64;
    static constexpr int kWaves = 4;
    static constexpr int kOccupancy = 4;
};
template <> struct Fmt<kFp4d256> {
    static constexpr int kTile = 2048;
    static constexpr int kScaleBlock = 256;
    static constexpr int kWaves = 4;
    static constexpr int kOccupancy = 2;
};
// Head size 64, two KV heads A and B per block.  A stage holds them in the
// layout of one 128-channel head: K tile = A's two channel groups then B's
// (k 0..63 and 64..127 of the QK operand), V tile = per 4 tokens A's eight
// 8-channel blocks then B's (channel blocks 0..7 and 8..15 of PV), scales
// [K: A, B][V: A, B].  The query operand is block diagonal: columns 0..7
// hold A's query heads on k 0..63, columns 8..15 B's on k 64..127, so the
// scores of each column see only its own head's keys; of the PV output only
// the tiles (A's channels, A's columns) and (B's, B's) are kept.  The block
// then does the arithmetic of one head-size-128 block for two heads of 64.
template <> struct Fmt<kFp4d64x2> {
    static constexpr int kTile = 1024;
    static constexpr int kScaleBlock = 2 * kTileScales;
    static constexpr int kWaves = 4;
    static constexpr int kOccupancy = 4;
};
template <int F> constexpr bool is_fp4() { return F == kFp4 || F == kFp4d64 || F == kFp4d256 || F == kFp4d64x2; }
template <int F> constexpr int head_dim_of() {
    return (F == kFp4d64 || F == kFp4d64x2) ? 64 : F == kFp4d256 ? 256 : 128;
}
// The register and operand formats: the paired head-size-64 stage is read
// and computed as a head-size-128 FP4 stage.
template <int F> constexpr int regs_fmt() { return F == kFp4d64x2 ? kFp4 : F; }
// Ultra-TQ: per page 1 KiB of K indices, 1 KiB of V codes and 320 bytes of
// norms and (scale, zero) words ("scale block").
template <> struct Fmt<kTq4> {
    static constexpr int kTile = 1024;
    static constexpr int kScaleBlock = kTqBlock - 2048;
    static constexpr int kWaves = 4;
    static constexpr int kOccupancy = 3;
};

// One stage of the ring: [K page0][V page0][K page1][V page1][scales0][scales1].
template <int F> constexpr int stage_bytes() { return 4 * Fmt<F>::kTile + 2 * Fmt<F>::kScaleBlock; }
template <int F, int S> constexpr int ring_bytes() { return S * stage_bytes<F>(); }
// LDS of one block besides the rings and id slots: the query operand and
// the merge's (max, sum).
template <int F> constexpr int q_lds_bytes() {
    return (F == kBf16 || F == kTq4) ? 4 * 64 * 16 : (head_dim_of<F>() / 128 + (head_dim_of<F>() < 128)) * 64 * 32;
}
constexpr int kIdsSlot = 256;   // LDS bytes per wave for the next 64 page ids
template <int F, int S, int W = Fmt<F>::kWaves> constexpr int block_lds_bytes() {
    return W * (ring_bytes<F, S>() + kIdsSlot) + q_lds_bytes<F>() + 2 * W * 16 * 4;
}
// Waves per SIMD with an S-slot ring and W waves per block: what 160 KiB of
// LDS per CU holds, capped by the format's register-set budget.
template <int F, int S, int W = Fmt<F>::kWaves> constexpr int occupancy() {
    constexpr int blocks = (160 * 1024) / block_lds_bytes<F, S, W>();
    constexpr int waves = blocks * W / 4;
    return waves < 1 ? 1 : (waves < Fmt<F>::kOccupancy ? waves : Fmt<F>::kOccupancy);
}
template <int F> constexpr int dma_per_stage() { return 4 * Fmt<F>::kTile / 1024 + (Fmt<F>::kScaleBlock ? 1 : 0); }

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

__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
    v2bf h = {__bf16(a), __bf16(b)};
    return __builtin_bit_cast(uint32_t, h);
}

// Scale float 2^(b-127) of byte B of a word of UE8M0 bytes: one SDWA shift
// (b << 23; byte 0 gives 0.0, as ue8m0_to_f32).
#define UQ_BYTE_SCALE(B)                                                                                     \
    __device__ __forceinline__ float byte_scale##B(uint32_t w, uint32_t k23) {                                \
        float r;                                                                                           \
        asm("v_lshlrev_b32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_" #B \
            : "=v"(r)                                                                                      \
            : "v"(k23), "v"(w));                                                                           \
        return r;                                                                                          \
    }
UQ_BYTE_SCALE(0)
UQ_BYTE_SCALE(1)
UQ_BYTE_SCALE(2)
UQ_BYTE_SCALE(3)
#undef UQ_BYTE_SCALE

// The two BF16 terms of P = hi + lo for two values a, b: hi keeps the upper
// 16 bits of each fp32 pattern (one byte permute for both), lo is the
// remainder, exact in fp32, rounded to BF16; |P - hi - lo| <= 2^-16 |P|.
__device__ __forceinline__ void split_p(float a, float b, uint32_t& hi, uint32_t& lo) {
    const uint32_t ua = f32_bits(a), ub = f32_bits(b);
    hi = __builtin_amdgcn_perm(ub, ua, 0x07060302u);
    lo = pack_bf16x2(a - bits_f32(ua & 0xFFFF0000u), b - bits_f32(ub & 0xFFFF0000u));
}

typedef __attribute__((address_space(3))) void* lds_ptr_t;

// Page ids of one wave, 64 at a time: lane j holds the id of the wave's
// page 2*(32*chunk + j/2) + j%2 counted in its own iteration order
// (iteration k of wave w covers partition pages 2*(w + W*k) and +1).  The
// range check (clamp_ids) follows once the ids are in registers.
template <int W>
__device__ __forceinline__ int ids_page(int wave, int chunk, int lane) {
    return 2 * (wave + W * (32 * chunk + (lane >> 1))) + (lane & 1);
}
template <int W>
__device__ __forceinline__ int32_t load_page_ids(const int32_t* __restrict__ pt_row, int first_page, int n_pages,
                                                 int wave, int chunk, int lane) {
    const int pg = ids_page<W>(wave, chunk, lane);
    int32_t id = 0;
    if (pg < n_pages) id = pt_row[first_page + pg];
    return id;
}
// The same ids copied into the wave's LDS slot (lane j's id at dword j)
// with global_load_lds_dword, so that no register waits for them: loading
// them into registers would make the wave wait for this load, and with it
// for every page copy in flight, when their values are first used.  Lanes
// past the partition read its first entry (their ids are never used).
template <int W>
__device__ __forceinline__ void copy_page_ids(uint8_t* slot, const int32_t* __restrict__ pt_row, int first_page,
                                              int n_pages, int wave, int chunk, int lane) {
    const int pg = ids_page<W>(wave, chunk, lane);
    __builtin_amdgcn_global_load_lds(pt_row + first_page + (pg < n_pages ? pg : 0), (lds_ptr_t)slot, 4, 0, 0);
}
// This lane's id from the wave's LDS slot; the caller has waited for the copy.
__device__ __forceinline__ int32_t read_page_ids(uint32_t slot_addr, int lane) {
    int32_t v;
    asm volatile("ds_read_b32 %0, %1\n\ts_waitcnt lgkmcnt(0)" : "=v"(v) : "v"(slot_addr + 4 * lane) : "memory");
    return v;
}

// Out-of-range ids never leave the pools.
__device__ __forceinline__ int32_t clamp_ids(int32_t id, int64_t num_pages) {
    return (id < 0 || int64_t(id) >= num_pages) ? 0 : id;
}

// Cache policy bits of the page copies (the aux operand of
// global_load_lds): kPageStream sets nt, the non-temporal (streaming)
// policy, for pages that one block reads once; kPageShared keeps the
// default policy for the shared-prefix pages, which the column chunks of a
// prefix partition read again from L2.  On the Qwen3-like layer (570 MB of
// pages per call) the streaming policy takes the FP4 decode kernel from
// 106.5 to 93.1 us and its page-gather probe from 99 to 88 us (sc0/sc1 on
// top of nt change nothing).
constexpr int kPageStream = 2;   // nt
constexpr int kPageShared = 0;

// Asynchronous copy of one iteration (two pages of one kv head) from HBM
// into an LDS stage with global_load_lds_dwordx4: every lane moves 16 bytes
// and the hardware places lane i's bytes at dst + 16 i, so each 1 KiB chunk
// of a tile lands in lane order.  The FP4 scale blocks of both pages
// (2 x 128 bytes) are moved by lanes 0..15.  AUX: the cache policy bits.
template <int F, int AUX = kPageStream>
__device__ __forceinline__ void stage_issue(uint8_t* stage, const uint8_t* __restrict__ codes,
                                            const uint8_t* __restrict__ scales, int64_t tile0, int64_t tile1,
                                            int lane) {
    if constexpr (F == kTq4) {
        // stage: [K0][V0][K1][V1] 1 KiB each, then both pages' 320-byte
        // metadata (lanes 0..19 page 0, lanes 20..39 page 1)
        const uint8_t* b0 = codes + (tile0 >> 1) * kTqBlock;
        const uint8_t* b1 = codes + (tile1 >> 1) * kTqBlock;
        __builtin_amdgcn_global_load_lds(b0 + 16 * lane, (lds_ptr_t)stage, 16, 0, AUX);
        __builtin_amdgcn_global_load_lds(b0 + 1024 + 16 * lane, (lds_ptr_t)(stage + 1024), 16, 0, AUX);
        __builtin_amdgcn_global_load_lds(b1 + 16 * lane, (lds_ptr_t)(stage + 2048), 16, 0, AUX);
        __builtin_amdgcn_global_load_lds(b1 + 1024 + 16 * lane, (lds_ptr_t)(stage + 3072), 16, 0, AUX);
        if (lane < 40) {
            const uint8_t* m = lane < 20 ? b0 + kTqMeta + 16 * lane : b1 + kTqMeta + 16 * (lane - 20);
            __builtin_amdgcn_global_load_lds(m, (lds_ptr_t)(stage + 4096), 16, 0, AUX);
        }
        return;
    }
    if constexpr (F == kFp4d64x2) {
        // tile0/tile1: head A's K tile of each page in 512-byte tiles; the
        // pool holds [K_A][V_A][K_B][V_B] (512 B each), the scale pool
        // [K_A][V_A][K_B][V_B] (32 B each) per page and head pair
        const int u = lane & 15, r = lane >> 4;
        const int64_t ko = lane < 32 ? 16 * lane : 1024 + 16 * (lane - 32);
        const int64_t vo = (u < 8 ? 512 : 1536) + 16 * (8 * r + (u & 7));
        const uint8_t* b0 = codes + tile0 * 512;
        const uint8_t* b1 = codes + tile1 * 512;
        __builtin_amdgcn_global_load_lds(b0 + ko, (lds_ptr_t)stage, 16, 0, AUX);
        __builtin_amdgcn_global_load_lds(b0 + vo, (lds_ptr_t)(stage + 1024), 16, 0, AUX);
        __builtin_amdgcn_global_load_lds(b1 + ko, (lds_ptr_t)(stage + 2048), 16, 0, AUX);
        __builtin_amdgcn_global_load_lds(b1 + vo, (lds_ptr_t)(stage + 3072), 16, 0, AUX);
        if (lane < 16) {
            // 16-byte unit j of a page's 128-byte block: K_A K_A K_B K_B V_A V_A V_B V_B
            const int j = lane & 7;
            const int64_t so = (j < 4 ? 0 : 32) + ((j & 2) ? 64 : 0) + 16 * (j & 1);
            const uint8_t* sc = scales + ((lane < 8 ? tile0 : tile1) >> 1) * 64 + so;
            __builtin_amdgcn_global_load_lds(sc, (lds_ptr_t)(stage + 4096), 16, 0, AUX);
        }
        return;
    }
    constexpr int T = Fmt<F>::kTile;
    const uint8_t* k0 = codes + tile0 * T + 16 * lane;
    const uint8_t* k1 = codes + tile1 * T + 16 * lane;
#pragma unroll
    for (int c = 0; c < 2 * T; c += 1024) {
        __builtin_amdgcn_global_load_lds(k0 + c, (lds_ptr_t)(stage + c), 16, 0, AUX);
    }
#pragma unroll
    for (int c = 0; c < 2 * T; c += 1024) {
        __builtin_amdgcn_global_load_lds(k1 + c, (lds_ptr_t)(stage + 2 * T + c), 16, 0, AUX);
    }
    if constexpr (Fmt<F>::kScaleBlock != 0) {
        // both pages' scale blocks (K then V scales, kScaleBlock bytes per page)
        constexpr int SB = Fmt<F>::kScaleBlock;
        if (lane < SB / 8) {
            const int64_t t = lane < SB / 16 ? tile0 : tile1;
            const uint8_t* sc = scales + (t >> 1) * SB + 16 * (lane % (SB / 16));
            __builtin_amdgcn_global_load_lds(sc, (lds_ptr_t)(stage + 4 * T), 16, 0, AUX);
        }
    }
}

// Wait until at most N of this wave's vector-memory loads are outstanding
// (loads complete in issue order, so the older stage is then in LDS).
template <int N>
__device__ __forceinline__ void wait_vmem() {
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// This lane's operands of one stage.  The reads are inline assembly so that
// the compiler does not guard them with a wait for every outstanding LDS
// copy (the caller has waited for this stage's copies already); each read
// block ends with lgkmcnt(0), so the results are safe to use.
template <int F> struct StageRegs;

template <> struct StageRegs<kFp4> {
    uint4 k[2], v[2];   // 16 bytes of each tile
    uint32_t ks[2];     // K scale byte of (token lane%16, group lane/16)
    uint32_t vs[2];     // V scale bytes of tokens 4*(lane/16)+0..3, group (lane%16)/4
};
template <> struct StageRegs<kFp8> {
    uint4 k[2][2], v[2][2];   // 32 bytes of each tile
};
template <> struct StageRegs<kBf16> {
    uint4 k[2][4], v[2][4];   // K: 4 k-steps x 16 bytes; V: 64 bytes
};
// Head size 64: as kFp4, with lanes 32..63 (channels 64..127 of the QK
// operand) and V lanes with lane%16 >= 8 (channel blocks 8..15) zero.
template <> struct StageRegs<kFp4d64> {
    uint4 k[2], v[2];
    uint32_t ks[2], vs[2];
};
// Head size 256: two 128-channel chunks for QK (k[pg][m], ks[pg][m]) and two
// channel blocks per lane for V (blocks lane%16 and lane%16 + 16).
template <> struct StageRegs<kFp4d256> {
    uint4 k[2][2], v[2][2];
    uint32_t ks[2][2], vs[2][2];
};
template <> struct StageRegs<kTq4> {
    uint4 k[2];    // K indices of token lane%16, channels 32s + 8*(lane/16) + 0..7 in dword s
    uint4 v[2];    // V codes of tokens 4*(lane/16) + 0..3 (dword t), channels 8*(lane%16) + 0..7
    uint4 kn[2];   // K norms of tokens 4*(lane/16) + 0..3
    uint4 vm[2];   // V (scale, zero) of the same tokens, group (lane%16)/4
};

__device__ __forceinline__ void stage_read(StageRegs<kFp4>& r, uint32_t stage_addr, int lane) {
    const uint32_t ac = stage_addr + 16 * lane;
    const uint32_t ak = stage_addr + lane;
    const uint32_t av = stage_addr + kTileScales + ((lane & 15) >> 2) * 16 + 4 * (lane >> 4);
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
        : "=&v"(r.k[0]), "=&v"(r.v[0]), "=&v"(r.k[1]), "=&v"(r.v[1]), "=&v"(r.ks[0]), "=&v"(r.ks[1]), "=&v"(r.vs[0]),
          "=&v"(r.vs[1])
        : "v"(ac), "v"(ak), "v"(av)
        : "memory");
}

__device__ __forceinline__ void stage_read(StageRegs<kFp8>& r, uint32_t stage_addr, int lane) {
    const uint32_t a = stage_addr + 32 * lane;
    asm volatile(
        "ds_read_b128 %0, %8\n\t"
        "ds_read_b128 %1, %8 offset:16\n\t"
        "ds_read_b128 %2, %8 offset:2048\n\t"
        "ds_read_b128 %3, %8 offset:2064\n\t"
        "ds_read_b128 %4, %8 offset:4096\n\t"
        "ds_read_b128 %5, %8 offset:4112\n\t"
        "ds_read_b128 %6, %8 offset:6144\n\t"
        "ds_read_b128 %7, %8 offset:6160\n\t"
        "s_waitcnt lgkmcnt(0)"
        : "=&v"(r.k[0][0]), "=&v"(r.k[0][1]), "=&v"(r.v[0][0]), "=&v"(r.v[0][1]), "=&v"(r.k[1][0]),
          "=&v"(r.k[1][1]), "=&v"(r.v[1][0]), "=&v"(r.v[1][1])
        : "v"(a)
        : "memory");
}

__device__ __forceinline__ void stage_read(StageRegs<kBf16>& r, uint32_t stage_addr, int lane) {
    // K: k-step s at s*1024 + 16*lane; V: 64 bytes at 4096 + 64*lane (page 1: +8192)
    const uint32_t ak = stage_addr + 16 * lane;
    const uint32_t av = stage_addr + 64 * lane;
    asm volatile(
        "ds_read_b128 %0, %16\n\t"
        "ds_read_b128 %1, %16 offset:1024\n\t"
        "ds_read_b128 %2, %16 offset:2048\n\t"
        "ds_read_b128 %3, %16 offset:3072\n\t"
        "ds_read_b128 %4, %17 offset:4096\n\t"
        "ds_read_b128 %5, %17 offset:4112\n\t"
        "ds_read_b128 %6, %17 offset:4128\n\t"
        "ds_read_b128 %7, %17 offset:4144\n\t"
        "ds_read_b128 %8, %16 offset:8192\n\t"
        "ds_read_b128 %9, %16 offset:9216\n\t"
        "ds_read_b128 %10, %16 offset:10240\n\t"
        "ds_read_b128 %11, %16 offset:11264\n\t"
        "ds_read_b128 %12, %17 offset:12288\n\t"
        "ds_read_b128 %13, %17 offset:12304\n\t"
        "ds_read_b128 %14, %17 offset:12320\n\t"
        "ds_read_b128 %15, %17 offset:12336\n\t"
        "s_waitcnt lgkmcnt(0)"
        : "=&v"(r.k[0][0]), "=&v"(r.k[0][1]), "=&v"(r.k[0][2]), "=&v"(r.k[0][3]), "=&v"(r.v[0][0]),
          "=&v"(r.v[0][1]), "=&v"(r.v[0][2]), "=&v"(r.v[0][3]), "=&v"(r.k[1][0]), "=&v"(r.k[1][1]),
          "=&v"(r.k[1][2]), "=&v"(r.k[1][3]), "=&v"(r.v[1][0]), "=&v"(r.v[1][1]), "=&v"(r.v[1][2]),
          "=&v"(r.v[1][3])
        : "v"(ak), "v"(av)
        : "memory");
}

// Head size 64, stage [K0 512][V0 512][K1 512][V1 512][scales0 64][scales1 64].
__device__ __forceinline__ void stage_read(StageRegs<kFp4d64>& r, uint32_t stage_addr, int lane) {
    const int n = lane & 15, g4 = lane >> 4;
    const uint32_t ak = stage_addr + 16 * lane;
    const uint32_t av = stage_addr + 512 + 16 * (8 * g4 + (n & 7));
    const uint32_t as = stage_addr + 2048 + (lane & 31);
    const uint32_t avs = stage_addr + 2048 + 32 + ((n & 7) >> 2) * 16 + 4 * g4;
    asm volatile(
        "ds_read_b128 %0, %8\n\t"
        "ds_read_b128 %1, %9\n\t"
        "ds_read_b128 %2, %8 offset:1024\n\t"
        "ds_read_b128 %3, %9 offset:1024\n\t"
        "ds_read_u8 %4, %10\n\t"
        "ds_read_u8 %5, %10 offset:64\n\t"
        "ds_read_b32 %6, %11\n\t"
        "ds_read_b32 %7, %11 offset:64\n\t"
        "s_waitcnt lgkmcnt(0)"
        : "=&v"(r.k[0]), "=&v"(r.v[0]), "=&v"(r.k[1]), "=&v"(r.v[1]), "=&v"(r.ks[0]), "=&v"(r.ks[1]), "=&v"(r.vs[0]),
          "=&v"(r.vs[1])
        : "v"(ak), "v"(av), "v"(as), "v"(avs)
        : "memory");
    if (lane >= 32) {   // k-blocks 2, 3 of the QK operand: channels 64..127 do not exist
        r.k[0] = uint4{0u, 0u, 0u, 0u};
        r.k[1] = uint4{0u, 0u, 0u, 0u};
        r.ks[0] = 127u;
        r.ks[1] = 127u;
    }
    if (n >= 8) {       // channel blocks 8..15 do not exist
        r.v[0] = uint4{0u, 0u, 0u, 0u};
        r.v[1] = uint4{0u, 0u, 0u, 0u};
        r.vs[0] = 0u;
        r.vs[1] = 0u;
    }
}

// Head size 256, stage [K0 2048][V0 2048][K1 2048][V1 2048][scales0 256][scales1 256].
__device__ __forceinline__ void stage_read(StageRegs<kFp4d256>& r, uint32_t stage_addr, int lane) {
    const int n = lane & 15, g4 = lane >> 4;
    const uint32_t ak = stage_addr + 16 * lane;
    const uint32_t av = stage_addr + 2048 + 16 * (32 * g4 + n);
    const uint32_t as = stage_addr + 8192 + lane;
    const uint32_t avs = stage_addr + 8192 + 128 + (n >> 2) * 16 + 4 * g4;
    asm volatile(
        "ds_read_b128 %0, %16\n\t"
        "ds_read_b128 %1, %16 offset:1024\n\t"
        "ds_read_b128 %2, %17\n\t"
        "ds_read_b128 %3, %17 offset:256\n\t"
        "ds_read_b128 %4, %16 offset:4096\n\t"
        "ds_read_b128 %5, %16 offset:5120\n\t"
        "ds_read_b128 %6, %17 offset:4096\n\t"
        "ds_read_b128 %7, %17 offset:4352\n\t"
        "ds_read_u8 %8, %18\n\t"
        "ds_read_u8 %9, %18 offset:64\n\t"
        "ds_read_u8 %10, %18 offset:256\n\t"
        "ds_read_u8 %11, %18 offset:320\n\t"
        "ds_read_b32 %12, %19\n\t"
        "ds_read_b32 %13, %19 offset:64\n\t"
        "ds_read_b32 %14, %19 offset:256\n\t"
        "ds_read_b32 %15, %19 offset:320\n\t"
        "s_waitcnt lgkmcnt(0)"
        : "=&v"(r.k[0][0]), "=&v"(r.k[0][1]), "=&v"(r.v[0][0]), "=&v"(r.v[0][1]), "=&v"(r.k[1][0]),
          "=&v"(r.k[1][1]), "=&v"(r.v[1][0]), "=&v"(r.v[1][1]), "=&v"(r.ks[0][0]), "=&v"(r.ks[0][1]),
          "=&v"(r.ks[1][0]), "=&v"(r.ks[1][1]), "=&v"(r.vs[0][0]), "=&v"(r.vs[0][1]), "=&v"(r.vs[1][0]),
          "=&v"(r.vs[1][1])
        : "v"(ak), "v"(av), "v"(as), "v"(avs)
        : "memory");
}

__device__ __forceinline__ void stage_read(StageRegs<kTq4>& r, uint32_t stage_addr, int lane) {
    const uint32_t ak = stage_addr + 16 * lane;
    const uint32_t an = stage_addr + 4096 + 16 * (lane >> 4);
    const uint32_t am = stage_addr + 4096 + 64 + 16 * (4 * (lane >> 4) + ((lane & 15) >> 2));
    asm volatile(
        "ds_read_b128 %0, %8\n\t"
        "ds_read_b128 %1, %8 offset:1024\n\t"
        "ds_read_b128 %2, %8 offset:2048\n\t"
        "ds_read_b128 %3, %8 offset:3072\n\t"
        "ds_read_b128 %4, %9\n\t"
        "ds_read_b128 %5, %9 offset:320\n\t"
        "ds_read_b128 %6, %10\n\t"
        "ds_read_b128 %7, %10 offset:320\n\t"
        "s_waitcnt lgkmcnt(0)"
        : "=&v"(r.k[0]), "=&v"(r.v[0]), "=&v"(r.k[1]), "=&v"(r.v[1]), "=&v"(r.kn[0]), "=&v"(r.kn[1]),
          "=&v"(r.vm[0]), "=&v"(r.vm[1])
        : "v"(ak), "v"(an), "v"(am)
        : "memory");
}

// Query operand in registers.
template <int F> struct QOperand { v8i q; };               // FP8 bytes, 32 per lane
template <> struct QOperand<kBf16> { v8bf q[4]; };          // 4 k-steps x 8 BF16 per lane
template <> struct QOperand<kFp4d256> { v8i q[2]; };        // FP8 bytes of the two 128-channel chunks
// Ultra-TQ: the BF16 query with each k-step's 8 channels in the order
// 0, 2, 4, 6, 1, 3, 5, 7 (the order the index decoder produces), and the
// codebook's byte tables.
template <> struct QOperand<kTq4> {
    v8bf q[4];
    uint32_t lut[8];
};

// BF16 levels of 8 K indices (nibble i of w = channel i): the byte tables
// are looked up with v_perm (8 entries per instruction, the 4th index bit
// picks the half), high and low bytes separately, then interleaved into
// BF16 pairs (channels 0,2), (4,6), (1,3), (5,7).
__device__ __forceinline__ uint4 tq_decode8(uint32_t w, const uint32_t (&lut)[8]) {
    const uint32_t e = w & 0x0F0F0F0Fu;            // byte j: index of channel 2j
    const uint32_t o = (w >> 4) & 0x0F0F0F0Fu;     // byte j: index of channel 2j+1
    const uint32_t se = e & 0x07070707u, so = o & 0x07070707u;
    const uint32_t te = ((e >> 1) & 0x04040404u) | 0x03020100u;
    const uint32_t to = ((o >> 1) & 0x04040404u) | 0x03020100u;
    const uint32_t he = __builtin_amdgcn_perm(__builtin_amdgcn_perm(lut[3], lut[2], se),
                                              __builtin_amdgcn_perm(lut[1], lut[0], se), te);
    const uint32_t le = __builtin_amdgcn_perm(__builtin_amdgcn_perm(lut[7], lut[6], se),
                                              __builtin_amdgcn_perm(lut[5], lut[4], se), te);
    const uint32_t ho = __builtin_amdgcn_perm(__builtin_amdgcn_perm(lut[3], lut[2], so),
                                              __builtin_amdgcn_perm(lut[1], lut[0], so), to);
    const uint32_t lo = __builtin_amdgcn_perm(__builtin_amdgcn_perm(lut[7], lut[6], so),
                                              __builtin_amdgcn_perm(lut[5], lut[4], so), to);
    return uint4{__builtin_amdgcn_perm(he, le, 0x05010400u), __builtin_amdgcn_perm(he, le, 0x07030602u),
                 __builtin_amdgcn_perm(ho, lo, 0x05010400u), __builtin_amdgcn_perm(ho, lo, 0x07030602u)};
}

// S^T[token][query head] of one page: rows = the page's 16 tokens (lane's
// VGPR i holds token 4*(lane/16)+i), columns = query heads (lane%16).
__device__ __forceinline__ v4f qk_page(const StageRegs<kFp4>& r, int pg, const QOperand<kFp4>& q) {
    const v8i a = {int(r.k[pg].x), int(r.k[pg].y), int(r.k[pg].z), int(r.k[pg].w), 0, 0, 0, 0};
    const v4f zero = {0.f, 0.f, 0.f, 0.f};
    return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, q.q, zero, 4, 0, 0, int(r.ks[pg]), 0, 127);
}
__device__ __forceinline__ v4f qk_page(const StageRegs<kFp4d64>& r, int pg, const QOperand<kFp4d64>& q) {
    const v8i a = {int(r.k[pg].x), int(r.k[pg].y), int(r.k[pg].z), int(r.k[pg].w), 0, 0, 0, 0};
    const v4f zero = {0.f, 0.f, 0.f, 0.f};
    return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, q.q, zero, 4, 0, 0, int(r.ks[pg]), 0, 127);
}
__device__ __forceinline__ v4f qk_page(const StageRegs<kFp4d256>& r, int pg, const QOperand<kFp4d256>& q) {
    const v8i a0 = {int(r.k[pg][0].x), int(r.k[pg][0].y), int(r.k[pg][0].z), int(r.k[pg][0].w), 0, 0, 0, 0};
    const v8i a1 = {int(r.k[pg][1].x), int(r.k[pg][1].y), int(r.k[pg][1].z), int(r.k[pg][1].w), 0, 0, 0, 0};
    const v4f zero = {0.f, 0.f, 0.f, 0.f};
    const v4f s = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a0, q.q[0], zero, 4, 0, 0, int(r.ks[pg][0]), 0, 127);
    return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a1, q.q[1], s, 4, 0, 0, int(r.ks[pg][1]), 0, 127);
}
__device__ __forceinline__ v4f qk_page(const StageRegs<kFp8>& r, int pg, const QOperand<kFp8>& q) {
    const uint4 lo = r.k[pg][0], hi = r.k[pg][1];
    const v8i a = {int(lo.x), int(lo.y), int(lo.z), int(lo.w), int(hi.x), int(hi.y), int(hi.z), int(hi.w)};
    const v4f zero = {0.f, 0.f, 0.f, 0.f};
    return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, q.q, zero, 0, 0, 0, 127, 0, 127);
}
__device__ __forceinline__ v4f qk_page(const StageRegs<kBf16>& r, int pg, const QOperand<kBf16>& q) {
    v4f s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int st = 0; st < 4; ++st)
        s = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(v8bf, r.k[pg][st]), q.q[st], s, 0, 0, 0);
    return s;
}

__device__ __forceinline__ uint32_t dword(const uint4& v, int i) { return i == 0 ? v.x : i == 1 ? v.y : i == 2 ? v.z : v.w; }

// Ultra-TQ: <q, c[idx]> on the BF16 levels, then times the token's norm.
__device__ __forceinline__ v4f qk_page(const StageRegs<kTq4>& r, int pg, const QOperand<kTq4>& q) {
    v4f s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int st = 0; st < 4; ++st)
        s = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(v8bf, tq_decode8(dword(r.k[pg], st), q.lut)),
                                                    q.q[st], s, 0, 0, 0);
#pragma unroll
    for (int i = 0; i < 4; ++i) s[i] *= bits_f32(dword(r.kn[pg], i));
    return s;
}

// BF16 pair of this lane's V channels 8n+2C, 8n+2C+1 of token 4*(lane/16)+t
// of page pg, as one dword (even channel in the low half).
template <int C>
__device__ __forceinline__ uint32_t v_pair(const StageRegs<kFp4>& r, int pg, int t, const float (&sc)[2][4]) {
    return __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(dword(r.v[pg], t), sc[pg][t], C));
}
template <int C>
__device__ __forceinline__ uint32_t v_pair(const StageRegs<kFp8>& r, int pg, int t, const float (&)[2][4]) {
    // 8 bytes per token: dword 2t holds channels 8n..8n+3, dword 2t+1 8n+4..8n+7
    const uint32_t w = dword(r.v[pg][t >> 1], 2 * (t & 1) + (C >> 1));
    return __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w, 1.0f, (C & 1) != 0));
}
template <int C>
__device__ __forceinline__ uint32_t v_pair(const StageRegs<kBf16>& r, int pg, int t, const float (&)[2][4]) {
    // 16 bytes per token: dword C holds channels 8n+2C, 8n+2C+1
    return dword(r.v[pg][t], C);
}

// PV for channel pair C of every lane: channels 8n+2C (block 2C, low halves)
// and 8n+2C+1 (block 2C+1, high halves).  The BF16 values of tokens
// (t, t+1) are paired by byte permutes into the k-slot order of P.
template <int C, class R>
__device__ __forceinline__ void pv_pair(const R& r, const float (&sc)[2][4], const v8bf& Phi, const v8bf& Plo,
                                        v4f& acc_e, v4f& acc_o) {
    uint32_t c0[4], c1[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        c0[t] = v_pair<C>(r, 0, t, sc);
        c1[t] = v_pair<C>(r, 1, t, sc);
    }
    const uint4 ae = {__builtin_amdgcn_perm(c0[1], c0[0], 0x05040100u), __builtin_amdgcn_perm(c0[3], c0[2], 0x05040100u),
                      __builtin_amdgcn_perm(c1[1], c1[0], 0x05040100u), __builtin_amdgcn_perm(c1[3], c1[2], 0x05040100u)};
    const uint4 ao = {__builtin_amdgcn_perm(c0[1], c0[0], 0x07060302u), __builtin_amdgcn_perm(c0[3], c0[2], 0x07060302u),
                      __builtin_amdgcn_perm(c1[1], c1[0], 0x07060302u), __builtin_amdgcn_perm(c1[3], c1[2], 0x07060302u)};
    const v8bf Ve = __builtin_bit_cast(v8bf, ae);
    const v8bf Vo = __builtin_bit_cast(v8bf, ao);
    acc_e = __builtin_amdgcn_mfma_f32_16x16x32_bf16(Ve, Phi, acc_e, 0, 0, 0);
    acc_e = __builtin_amdgcn_mfma_f32_16x16x32_bf16(Ve, Plo, acc_e, 0, 0, 0);
    acc_o = __builtin_amdgcn_mfma_f32_16x16x32_bf16(Vo, Phi, acc_o, 0, 0, 0);
    acc_o = __builtin_amdgcn_mfma_f32_16x16x32_bf16(Vo, Plo, acc_o, 0, 0, 0);
}

// FP4 PV for channel pair C of one channel block per lane (v0, v1: the
// block's codes of the lane's 4 tokens of page 0 and page 1; sc: their
// scale floats), as pv_pair does for kFp4.
template <int C>
__device__ __forceinline__ void pv_pair_fp4(const uint4& v0, const uint4& v1, const float (&sc)[2][4], const v8bf& Phi,
                                            const v8bf& Plo, v4f& acc_e, v4f& acc_o) {
    uint32_t c0[4], c1[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        c0[t] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(dword(v0, t), sc[0][t], C));
        c1[t] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(dword(v1, t), sc[1][t], C));
    }
    const uint4 ae = {__builtin_amdgcn_perm(c0[1], c0[0], 0x05040100u), __builtin_amdgcn_perm(c0[3], c0[2], 0x05040100u),
                      __builtin_amdgcn_perm(c1[1], c1[0], 0x05040100u), __builtin_amdgcn_perm(c1[3], c1[2], 0x05040100u)};
    const uint4 ao = {__builtin_amdgcn_perm(c0[1], c0[0], 0x07060302u), __builtin_amdgcn_perm(c0[3], c0[2], 0x07060302u),
                      __builtin_amdgcn_perm(c1[1], c1[0], 0x07060302u), __builtin_amdgcn_perm(c1[3], c1[2], 0x07060302u)};
    const v8bf Ve = __builtin_bit_cast(v8bf, ae);
    const v8bf Vo = __builtin_bit_cast(v8bf, ao);
    acc_e = __builtin_amdgcn_mfma_f32_16x16x32_bf16(Ve, Phi, acc_e, 0, 0, 0);
    acc_e = __builtin_amdgcn_mfma_f32_16x16x32_bf16(Ve, Plo, acc_e, 0, 0, 0);
    acc_o = __builtin_amdgcn_mfma_f32_16x16x32_bf16(Vo, Phi, acc_o, 0, 0, 0);
    acc_o = __builtin_amdgcn_mfma_f32_16x16x32_bf16(Vo, Plo, acc_o, 0, 0, 0);
}

// Ultra-TQ PV for channel pair C: each V value is bf16(fma(scale, code,
// zero)) of its token's group, packed two tokens per register in the k-slot
// order of P.
template <int C>
__device__ __forceinline__ void pv_pair(const StageRegs<kTq4>& r, const float (&)[2][4], const v8bf& Phi,
                                        const v8bf& Plo, v4f& acc_e, v4f& acc_o) {
    float ve[2][4], vo[2][4];
#pragma unroll
    for (int pg = 0; pg < 2; ++pg) {
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            const uint32_t w = dword(r.v[pg], t);
            const uint32_t e = w & 0x0F0F0F0Fu, o = (w >> 4) & 0x0F0F0F0Fu;
            const uint32_t m = dword(r.vm[pg], t);
            const float s = bits_f32(m << 16), z = bits_f32(m & 0xFFFF0000u);
            ve[pg][t] = __builtin_fmaf(s, float((e >> (8 * C)) & 0xFFu), z);
            vo[pg][t] = __builtin_fmaf(s, float((o >> (8 * C)) & 0xFFu), z);
        }
    }
    const uint4 ae = {pack_bf16x2(ve[0][0], ve[0][1]), pack_bf16x2(ve[0][2], ve[0][3]), pack_bf16x2(ve[1][0], ve[1][1]),
                      pack_bf16x2(ve[1][2], ve[1][3])};
    const uint4 ao = {pack_bf16x2(vo[0][0], vo[0][1]), pack_bf16x2(vo[0][2], vo[0][3]), pack_bf16x2(vo[1][0], vo[1][1]),
                      pack_bf16x2(vo[1][2], vo[1][3])};
    const v8bf Ve = __builtin_bit_cast(v8bf, ae);
    const v8bf Vo = __builtin_bit_cast(v8bf, ao);
    acc_e = __builtin_amdgcn_mfma_f32_16x16x32_bf16(Ve, Phi, acc_e, 0, 0, 0);
    acc_e = __builtin_amdgcn_mfma_f32_16x16x32_bf16(Ve, Plo, acc_e, 0, 0, 0);
    acc_o = __builtin_amdgcn_mfma_f32_16x16x32_bf16(Vo, Phi, acc_o, 0, 0, 0);
    acc_o = __builtin_amdgcn_mfma_f32_16x16x32_bf16(Vo, Plo, acc_o, 0, 0, 0);
}

// Lane L of a 16-lane row writes channels N L .. N L + N - 1 of the row
// (head size 16 N).
template <int N>
__device__ __forceinline__ void write_out(const DecodeParams& p, int64_t row, int L, const float (&o)[N]) {
    const int64_t ob = row * (16 * N) + N * L;
    if (p.out_dtype == 0) {
        float4* dst = reinterpret_cast<float4*>(static_cast<float*>(p.out) + ob);
#pragma unroll
        for (int i = 0; i < N / 4; ++i) dst[i] = make_float4(o[4 * i], o[4 * i + 1], o[4 * i + 2], o[4 * i + 3]);
    } else if constexpr (N == 4) {
        *reinterpret_cast<uint2*>(static_cast<uint16_t*>(p.out) + ob) =
            uint2{pack_bf16x2(o[0], o[1]), pack_bf16x2(o[2], o[3])};
    } else {
        uint4* dst = reinterpret_cast<uint4*>(static_cast<uint16_t*>(p.out) + ob);
#pragma unroll
        for (int i = 0; i < N / 8; ++i)
            dst[i] = uint4{pack_bf16x2(o[8 * i], o[8 * i + 1]), pack_bf16x2(o[8 * i + 2], o[8 * i + 3]),
                           pack_bf16x2(o[8 * i + 4], o[8 * i + 5]), pack_bf16x2(o[8 * i + 6], o[8 * i + 7])};
    }
}

// Final scaling of one row: divide by the softmax sum, apply the V tensor
// scale, rotate back when V was stored rotated.
template <int N>
__device__ __forceinline__ void finish_row(const DecodeParams& p, float (&o)[N], float lsum, int L) {
    const float inv = p.out_scale / lsum;
#pragma unroll
    for (int i = 0; i < N; ++i) o[i] *= inv;
    if (p.rotate_v) wht_x<N>(o, L);
}

// Zero the V bytes of a masked token of a plain cache (garbage bytes past
// the context may decode to NaN or Inf, and 0 * NaN is NaN).
__device__ __forceinline__ void zero_token(StageRegs<kFp8>& c, int pg, int t) {
    uint4& v = c.v[pg][t >> 1];
    if (t & 1) v = uint4{v.x, v.y, 0u, 0u};
    else v = uint4{0u, 0u, v.z, v.w};
}
__device__ __forceinline__ void zero_token(StageRegs<kBf16>& c, int pg, int t) { c.v[pg][t] = uint4{0u, 0u, 0u, 0u}; }
__device__ __forceinline__ void zero_token(StageRegs<kFp4>&, int, int) {}   // handled through the scale byte
// Head sizes 64 and 256: scale byte 0 (scale 0.0) for the token's V groups.
__device__ __forceinline__ void zero_token(StageRegs<kFp4d64>& c, int pg, int t) { c.vs[pg] &= ~(0xFFu << (8 * t)); }
__device__ __forceinline__ void zero_token(StageRegs<kFp4d256>& c, int pg, int t) {
    c.vs[pg][0] &= ~(0xFFu << (8 * t));
    c.vs[pg][1] &= ~(0xFFu << (8 * t));
}
__device__ __forceinline__ void zero_token(StageRegs<kTq4>& c, int pg, int t) {
    // scale and zero 0: the value decodes to 0 whatever the bytes
    uint4& m = c.vm[pg];
    if (t == 0) m.x = 0u;
    else if (t == 1) m.y = 0u;
    else if (t == 2) m.z = 0u;
    else m.w = 0u;
}

// XOR of every 32-bit word of a stage's registers (the page-gather probe's
// checksum).
template <class R>
__device__ __forceinline__ uint32_t fold_words(const R& r) {
    static_assert(sizeof(R) % 4 == 0, "register words");
    struct Words { uint32_t w[sizeof(R) / 4]; };
    const Words x = __builtin_bit_cast(Words, r);
    uint32_t a = 0u;
#pragma unroll
    for (int i = 0; i < int(sizeof(R) / 4); ++i) a ^= x.w[i];
    return a;
}

template <int F, int S, bool WP, bool PROBE = false, int W = Fmt<F>::kWaves>
__global__ void __launch_bounds__(64 * W)
__attribute__((amdgpu_waves_per_eu(occupancy<F, S, W>(), occupancy<F, S, W>()))) decode_kernel(DecodeParams p) {
    static_assert(S == 2 || S == 4, "ring slots");
    static_assert(W == 2 || W == 4 || W == 8, "waves per block");
    static_assert(!PROBE || is_fp4<F>(), "the page-gather probe follows the FP4 kernels");
    static_assert(!WP || (head_dim_of<F>() == 128 && F != kFp4d64x2), "one wave per partition: head size 128");
    constexpr int kThreads = 64 * W;
    constexpr int kStage = stage_bytes<F>();
    constexpr int kQRounds = (256 + kThreads - 1) / kThreads;   // 16 threads per query row, 16 rows
    constexpr int D = head_dim_of<F>();         // head size
    constexpr int N = D / 16;                   // channels per lane of a 16-lane row
    constexpr bool kPair = F == kFp4d64x2;      // two kv heads of 64 per block
    constexpr int DA = kPair ? 128 : D;         // channels of the accumulators
    constexpr int kAccTiles = DA == 256 ? 16 : 8;   // PV output tiles of 16 channel blocks x 16 heads
    // Linear block order: kv head fastest, then sequence, then partition.
    // Workgroups go to the 8 XCDs round-robin by linear id, so this spreads
    // the work of every sequence evenly over the XCDs whatever the context
    // lengths (with the partition fastest, XCD k would get partition k of
    // every sequence and the XCDs holding the late partitions of short
    // sequences would idle), and it keeps one kv head on the same XCDs, whose
    // L2 then serves pages that several sequences share.
    //
    // Cascade decode takes its rows from a list that cascade_rows_kernel
    // writes: the context rows (partition, sequence) sorted by tokens,
    // longest first, then the prefix rows, then the rows without work.  With
    // the partition-major order the full partitions of the longest contexts
    // were dispatched last and ran alone at the end (the MiniMax-like
    // layer's last 60 µs), and the blocks without work went out before the
    // prefix blocks.  A prefix row is one (chunk of 16 query columns, prefix
    // partition), kv head fastest as for the context rows.  A
    // prefix block's columns are (sequence, query head) pairs f = 16 * chunk
    // + column of the flattened batch (b = f / G, head hk * G + f % G), and it
    // reads the shared prefix pages once for all of them.  Prefix blocks are
    // uniform and work mostly from L2 (the chunks of one prefix partition are
    // neighbours in the grid and meet in one XCD's L2), so placed last they
    // fill the CUs that the ragged context blocks leave idle at the end
    // (first, or spread through the grid, measured 8-16 % slower on the
    // MiniMax-like workload).
    //
    // WP (one wave per partition): block `rest / batch` of a (kv head,
    // sequence) takes partitions W * (rest / batch) + wave, one per wave.
    // Each wave streams its whole partition through its own ring; the block
    // then merges its W partials through LDS and writes one, so a block's
    // query prologue and partial write serve W partitions (on 4096-token
    // partitions of 128k contexts: 6.13 ms against 6.73 ms for one block
    // per partition).
    const int lin = blockIdx.x;
    // PROBE: the page-gather probe -- this grid, page walk, page-id copies,
    // ring copies and LDS reads, with the query prologue, the arithmetic and
    // the epilogue left out; each wave writes one XOR checksum of what it
    // staged to probe_sink[block * W + wave] (0 for a wave without pages).
    if constexpr (PROBE) {
        if ((threadIdx.x & 63) == 0) p.probe_sink[int64_t(lin) * W + (threadIdx.x >> 6)] = 0u;
    }
    const bool cascade = !WP && p.prefix_pages != nullptr;
    const int units = kPair ? p.num_kv_heads / 2 : p.num_kv_heads;   // kv heads, or pairs of them
    const int hk = lin % units;
    const int row = lin / units;
    bool pre = false;
    int rest = row;
    int row_ctx = 0, row_pl = 0;   // a cascade context row's length and prefix tokens
    if (cascade) {
        // the row list: context rows with the most tokens first, then the
        // prefix rows, then rows without work
        const int4 rec = p.cascade_rows[row];
        if (rec.x < 0) return;                                // no work left for this block
        const int context_rows = p.suffix_partitions * p.batch;
        pre = rec.x >= context_rows;                          // block-uniform
        rest = pre ? rec.x - context_rows : rec.x;
        row_ctx = rec.y;
        row_pl = rec.z;
    }
    const int nb = pre ? p.prefix_chunks : p.batch;
    const int b = pre ? 0 : rest % nb;                                 // sequence (context blocks)
    const int chunk = pre ? rest % nb : 0;                             // column chunk (prefix blocks)
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform: scalar control flow
    const int first_part = WP ? (rest / nb) * W : rest / nb;           // the block's (first) partition
    const int part = WP ? first_part + wave : first_part;
    const int G = p.group;
    const int BG = p.batch * G;

    int start, end, ctx = 0;
    if (pre) {
        start = part * p.prefix_partition;
        end = (start + p.prefix_partition) < p.prefix_tokens ? (start + p.prefix_partition) : p.prefix_tokens;
    } else {
        if (cascade) {
            ctx = row_ctx;
        } else {
            ctx = p.context_lens[b];
            ctx = ctx < p.max_context ? ctx : p.max_context;
        }
        start = part * p.partition_tokens;
        if (cascade) {
            // the context blocks start after the tokens the prefix blocks serve
            const int pl = row_pl;
            if (start + p.partition_tokens <= pl) return;              // wholly inside the prefix
            start = start > pl ? start : pl;
        }
        if ((WP ? first_part * p.partition_tokens : start) >= ctx) {
            // nothing of this sequence here; an empty context still gets its zero output
            if (!PROBE && ctx <= 0 && first_part == 0) {
                // the block's query heads: G of kv head hk, or 2 G of the pair
                for (int r = tid >> 4; r < (kPair ? 2 : 1) * G; r += kThreads / 16) {
                    float z[N];
#pragma unroll
                    for (int i = 0; i < N; ++i) z[i] = 0.f;
                    write_out<N>(p, int64_t(b) * p.num_q_heads + (kPair ? 2 : 1) * hk * G + r, tid & 15, z);
                }
            }
            return;
        }
        end = (part * p.partition_tokens + p.partition_tokens) < ctx ? (part * p.partition_tokens + p.partition_tokens) : ctx;
        if (WP && start >= ctx) {
            // a later wave of the block past a short context: no pages, but
            // it still takes part in the query prologue and the block merge
            start = end = ctx;
        }
    }
    // a context held by this block alone is finished in place: one partition,
    // or the W partitions of the first block of the wave grid
    const bool in_place = !cascade && ctx <= (WP ? W : 1) * p.partition_tokens;
    // query row r (0..15) of this block: valid, its sequence and query head
    auto row_of = [&](int r, int& rb, int& rhq) -> bool {
        if constexpr (kPair) {
            // rows 0..7: query heads of kv head 2 hk, rows 8..15: of 2 hk + 1
            rb = b;
            rhq = (2 * hk + (r >> 3)) * G + (r & 7);
            return (r & 7) < G;
        }
        if (pre) {
            const int f = 16 * chunk + r;
            rb = f / G;
            rhq = hk * G + (f - rb * G);
            return f < BG;
        }
        rb = b;
        rhq = hk * G + r;
        return r < G;
    };
    // Decode step: the block whose partition holds the last position writes
    // the sequence's new token there.  The wave that will read that page
    // encodes the token in its prologue, stores it to the pools without
    // waiting, and patches its staged copy of the page in LDS once the copy
    // has landed, so no wave waits for the store.  Only this block reads the
    // page for this kv head (partitions are whole pages).
    const int pos_new = ctx - 1;
    const int it_new = (pos_new - start) >> 5;                       // iteration holding the token
    // (the step is a head-size-128 call)
    const bool append = !PROBE && D == 128 && !pre && p.k_new != nullptr && pos_new >= start && pos_new < end &&
                        (WP || wave == it_new % W);
    const int k_new_local = WP ? it_new : it_new / W;                // that wave's local iteration

    __shared__ __attribute__((aligned(16))) uint8_t smem[W * ring_bytes<F, S>()];
    __shared__ __attribute__((aligned(16))) uint8_t q_lds[q_lds_bytes<F>()];
    __shared__ __attribute__((aligned(16))) uint8_t ids_lds[W * kIdsSlot];
    __shared__ float red_m[W][16];
    __shared__ float red_l[W][16];

    // ---------------- query load first (its latency overlaps the page walk set-up)
    float qx[kQRounds][N];
    uint32_t qw[kQRounds][2];
#pragma unroll
    for (int h = 0; h < kQRounds; ++h) {
#pragma unroll
        for (int i = 0; i < N; ++i) qx[h][i] = 0.f;
        qw[h][0] = 0u;
        qw[h][1] = 0u;
        const int qr = (tid >> 4) + h * (kThreads / 16);
        const int qL = tid & 15;
        int rb, rhq;
        if constexpr (D != 128) {
            // head sizes 64 and 256: an F32, BF16 or F16 query, N channels per thread
            if (!PROBE && qr < 16 && row_of(qr, rb, rhq)) {
                const int64_t elem = (int64_t(rb) * p.num_q_heads + rhq) * D + N * qL;
                float (&x)[N] = qx[h];
                if constexpr (N == 4) {
                    if (p.q_dtype == 0) load_x4<0>(p.q, elem, x);
                    else if (p.q_dtype == 1) load_x4<1>(p.q, elem, x);
                    else load_x4<2>(p.q, elem, x);
                } else {
                    float (&x0)[8] = *reinterpret_cast<float(*)[8]>(&x[0]);
                    float (&x1)[8] = *reinterpret_cast<float(*)[8]>(&x[8]);
                    if (p.q_dtype == 0) {
                        load_x8<0>(p.q, elem, x0);
                        load_x8<0>(p.q, elem + 8, x1);
                    } else if (p.q_dtype == 1) {
                        load_x8<1>(p.q, elem, x0);
                        load_x8<1>(p.q, elem + 8, x1);
                    } else {
                        load_x8<2>(p.q, elem, x0);
                        load_x8<2>(p.q, elem + 8, x1);
                    }
                }
            }
        } else {
          if (!PROBE && qr < 16 && row_of(qr, rb, rhq)) {
            const int64_t elem = (int64_t(rb) * p.num_q_heads + rhq) * kHeadDim + 8 * qL;
            if (p.q_dtype == 3) {
                const uint2 w = *reinterpret_cast<const uint2*>(static_cast<const uint8_t*>(p.q) + elem);
                qw[h][0] = w.x;
                qw[h][1] = w.y;
            } else if (p.q_dtype == 0) {
                load_x8<0>(p.q, elem, qx[h]);
            } else if (p.q_dtype == 1) {
                load_x8<1>(p.q, elem, qx[h]);
            } else {
                load_x8<2>(p.q, elem, qx[h]);
            }
          }
        }
    }

    float xk[8], xv[8];   // the new token's K and V (decode step, lanes 0..15 of the owning wave)
    int32_t page_new = -1;
    if (append && lane < 16) {
        page_new = p.page_table[int64_t(b) * p.max_pages_per_seq + (pos_new >> 4)];
        const int64_t elem = (int64_t(b) * p.num_kv_heads + hk) * kHeadDim + 8 * lane;
        if (p.new_dtype == 0) {
            load_x8<0>(p.k_new, elem, xk);
            load_x8<0>(p.v_new, elem, xv);
        } else if (p.new_dtype == 1) {
            load_x8<1>(p.k_new, elem, xk);
            load_x8<1>(p.v_new, elem, xv);
        } else {
            load_x8<2>(p.k_new, elem, xk);
            load_x8<2>(p.v_new, elem, xv);
        }
    }

    // ---------------- page walk set-up and the first two stages in flight
    const int first_page = start >> 4;
    const int n_pages = (end - start + 15) >> 4;
    const int n_iter = (n_pages + 1) >> 1;
    const int n_local = WP ? n_iter : wave < n_iter ? (n_iter - wave + W - 1) / W : 0;
    // page-walk order: iteration k of the wave covers partition pages
    // 2 * (woff + ws * k) and + 1
    constexpr int ws = WP ? 1 : W;
    const int woff = WP ? 0 : wave;
    const int32_t* pt_row = pre ? p.prefix_pages : p.page_table + int64_t(b) * p.max_pages_per_seq;
    // prefix blocks: this lane's column attends to the first `lim` prefix tokens
    int lim = end;
    if (pre) {
        int rb, rhq;
        lim = 0;
        if (row_of(lane & 15, rb, rhq)) {
            int c2 = p.context_lens[rb];
            c2 = c2 < p.max_context ? c2 : p.max_context;
            int pl = p.prefix_lens[rb];
            pl = pl < p.prefix_tokens ? pl : p.prefix_tokens;
            pl = pl < c2 - 1 ? pl : c2 - 1;
            lim = pl > 0 ? (pl & ~15) : 0;
            lim = lim < end ? lim : end;
        }
    }
    const int g4 = lane >> 4;           // lane group: tokens 4*g4..4*g4+3 of each page
    const int n = lane & 15;
    uint8_t* ring = smem + wave * ring_bytes<F, S>();
    const uint32_t ring_addr = uint32_t(reinterpret_cast<uintptr_t>((lds_ptr_t)ring));
    const int64_t head_tile = int64_t(kPair ? 2 * hk : hk) * 2;   // K tile of the (first) kv head
    const int64_t tiles_per_page = int64_t(p.num_kv_heads) * 2;

    uint8_t* ids_slot = ids_lds + wave * kIdsSlot;
    const uint32_t ids_addr = uint32_t(reinterpret_cast<uintptr_t>((lds_ptr_t)ids_slot));
    int32_t ids = 0;
    if (n_local > 0) {
        ids = load_page_ids<ws>(pt_row, first_page, n_pages, woff, 0, lane);
        if (n_local > 32) copy_page_ids<ws>(ids_slot, pt_row, first_page, n_pages, woff, 1, lane);
    }
    // The query, the new token and the page ids are in registers before the
    // first page copies are issued (one wait for all of them, so that the
    // query transform below overlaps the copies instead of waiting for them).
    __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
    ids = clamp_ids(ids, p.num_pages);
    if (n_local > 0) {
        for (int s = 0; s < S && s < n_local; ++s) {
            const int64_t id0 = __builtin_amdgcn_readlane(ids, 2 * s);
            const int64_t id1 = __builtin_amdgcn_readlane(ids, 2 * s + 1);
            if (pre)
                stage_issue<F, kPageShared>(ring + s * kStage, p.codes, p.scales, id0 * tiles_per_page + head_tile,
                                            id1 * tiles_per_page + head_tile, lane);
            else
                stage_issue<F, kPageStream>(ring + s * kStage, p.codes, p.scales, id0 * tiles_per_page + head_tile,
                                            id1 * tiles_per_page + head_tile, lane);
        }
    }

    // ---------------- query prologue: transform and store in B-operand order
#pragma unroll
    for (int h = 0; h < (PROBE ? 0 : kQRounds); ++h) {
        const int qr = (tid >> 4) + h * (kThreads / 16);
        // blocks of more than 4 waves: the threads past the 16 query rows
        // store nothing (their rows would land on other rows' operand bytes
        // and past the operand area); whole waves, so a scalar branch
        if (qr >= 16) continue;
        const int qL = tid & 15;
        int rb, rhq;
        const bool qvalid = row_of(qr, rb, rhq);
        if constexpr (F == kBf16 || F == kTq4) {
            // channels 8*qL..+7 are k-step qL/4, lane (qL%4)*16 + qr, 16 bytes
            uint4 w = {0u, 0u, 0u, 0u};
            if (qvalid) {
                if constexpr (F == kTq4) {
                    // rotated like the keys, channels in the decoder's order
                    wht128_x8(qx[h], qL);
                    w = uint4{pack_bf16x2(qx[h][0], qx[h][2]), pack_bf16x2(qx[h][4], qx[h][6]),
                              pack_bf16x2(qx[h][1], qx[h][3]), pack_bf16x2(qx[h][5], qx[h][7])};
                } else {
                    w = uint4{pack_bf16x2(qx[h][0], qx[h][1]), pack_bf16x2(qx[h][2], qx[h][3]),
                              pack_bf16x2(qx[h][4], qx[h][5]), pack_bf16x2(qx[h][6], qx[h][7])};
                }
            }
            *reinterpret_cast<uint4*>(q_lds + ((qL >> 2) * 64 + (qL & 3) * 16 + qr) * 16) = w;
        } else if constexpr (kPair) {
            // rotated (64-point) and cast to FP8: rows 0..7 (head A) on k
            // 0..63, rows 8..15 (head B) on k 64..127 of the B operand (layout
            // below); the other half of each row stays zero
            uint32_t wq = 0u;
            if (qvalid) {
                wht_x<N>(qx[h], qL);
#pragma unroll
                for (int j = 0; j < 4; ++j) wq |= e4m3_byte(qx[h][j]) << (8 * j);
            }
            const int ch = N * qL + (qr >= 8 ? 64 : 0);
            const int g = (ch & 63) >> 4;
            const int e0 = (ch & 15) + (ch >= 64 ? 16 : 0);
            *reinterpret_cast<uint32_t*>(q_lds + (g * 16 + qr) * 32 + e0) = wq;
            if (qL < 4) *reinterpret_cast<uint4*>(q_lds + (qL * 16 + qr) * 32 + (qr >= 8 ? 0 : 16)) = uint4{0u, 0u, 0u, 0u};
        } else if constexpr (F == kFp4d64 || F == kFp4d256) {
            // rotated (D-point) and cast to FP8; the lane's N channels go to the
            // B operand of the 128-channel chunk they belong to (layout below)
            uint32_t wq[N / 4];
#pragma unroll
            for (int i = 0; i < N / 4; ++i) wq[i] = 0u;
            if (qvalid) {
                wht_x<N>(qx[h], qL);
#pragma unroll
                for (int i = 0; i < N / 4; ++i)
#pragma unroll
                    for (int j = 0; j < 4; ++j) wq[i] |= e4m3_byte(qx[h][4 * i + j]) << (8 * j);
            }
            const int ch = N * qL;
            const int c2 = ch & 127;
            const int g = (c2 & 63) >> 4;
            const int e0 = (c2 & 15) + (c2 >= 64 ? 16 : 0);
            uint8_t* dst = q_lds + (ch >> 7) * 2048 + (g * 16 + qr) * 32 + e0;
            if constexpr (N == 4) {
                *reinterpret_cast<uint32_t*>(dst) = wq[0];
                // channels 64..127 of the chunk do not exist: zero operand
                if (qL < 4) *reinterpret_cast<uint4*>(q_lds + (qL * 16 + qr) * 32 + 16) = uint4{0u, 0u, 0u, 0u};
            } else {
                *reinterpret_cast<uint4*>(dst) = uint4{wq[0], wq[1], wq[2], wq[3]};
            }
        } else {
            uint32_t lo = qw[h][0], hi = qw[h][1];
            if (qvalid && p.q_dtype != 3) {
                if constexpr (F == kFp4) wht128_x8(qx[h], qL);
                lo = 0;
                hi = 0;
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    lo |= e4m3_byte(qx[h][i]) << (8 * i);
                    hi |= e4m3_byte(qx[h][i + 4]) << (8 * i);
                }
            }
            // FP8 operand of the 16x16x128 scaled MFMA: lane 16*g + n holds
            // column n, channels 16g..16g+15 in bytes 0..15 and
            // 64+16g..64+16g+15 in bytes 16..31.  Rows without a query stay zero.
            const int ch = 8 * qL;
            const int g = (ch & 63) >> 4;
            const int e0 = (ch & 15) + (ch >= 64 ? 16 : 0);
            *reinterpret_cast<uint2*>(q_lds + (g * 16 + qr) * 32 + e0) = make_uint2(lo, hi);
        }
    }
    if constexpr (!PROBE) __syncthreads();
    QOperand<regs_fmt<F>()> qop;
    if constexpr (F == kBf16 || F == kTq4) {
#pragma unroll
        for (int st = 0; st < 4; ++st)
            qop.q[st] = __builtin_bit_cast(v8bf, *reinterpret_cast<const uint4*>(q_lds + (st * 64 + lane) * 16));
        if constexpr (F == kTq4) {
#pragma unroll
            for (int j = 0; j < 8; ++j) qop.lut[j] = p.tq.lut[j];
        }
    } else if constexpr (F == kFp4d256) {
#pragma unroll
        for (int m = 0; m < 2; ++m) {
            const uint4* src = reinterpret_cast<const uint4*>(q_lds + m * 2048 + lane * 32);
            const uint4 a = src[0], c = src[1];
            qop.q[m] = v8i{int(a.x), int(a.y), int(a.z), int(a.w), int(c.x), int(c.y), int(c.z), int(c.w)};
        }
    } else {
        const uint4* src = reinterpret_cast<const uint4*>(q_lds + lane * 32);
        const uint4 a = src[0], c = src[1];
        qop.q = v8i{int(a.x), int(a.y), int(a.z), int(a.w), int(c.x), int(c.y), int(c.z), int(c.w)};
    }

    // Decode step, owning wave: encode and store the new token while its
    // first two stages are in flight (the store is not waited for).
    TokenBits<D == 128 ? F : kFp4> tok{};
    if constexpr (D == 128) {
        if (append && lane < 16) {
            tok = encode_token<F>(xk, xv, lane, p.c, p.rotate_v != 0, p.k_scale, p.v_scale, p.tq);
            if (page_new >= 0 && int64_t(page_new) < p.num_pages)
                store_token<F>(p.codes, p.scales, (int64_t(page_new) * p.num_kv_heads + hk) * 2, pos_new & 15, lane,
                               tok);
        }
    }

    const float sl2 = p.scale_log2;
    const uint32_t k23 = 23u;
    // finite start: a column with every score masked keeps exp2(-inf - m) = 0
    constexpr float kNoMax = -1e30f;
    float m_run = kNoMax;
    // wave-uniform: some column's running max has magnitude 2^20 or more
    // (then the exponents round the scaled score first; see below)
    bool big_max = false;
    // running softmax sum per column, on the matrix unit: every row of
    // (all ones) x P is the column sum of P
    const v8bf ones = __builtin_bit_cast(v8bf, uint4{0x3F803F80u, 0x3F803F80u, 0x3F803F80u, 0x3F803F80u});
    v4f acc_l = {0.f, 0.f, 0.f, 0.f};
    v4f acc[kAccTiles];
#pragma unroll
    for (int j = 0; j < kAccTiles; ++j) acc[j] = v4f{0.f, 0.f, 0.f, 0.f};

    uint32_t chk = 0u;   // PROBE: XOR of every staged word
    // ---------------- main loop: one stage (2 pages, 32 tokens) per iteration
    for (int k = 0; k < n_local; ++k) {
        // stage k has landed once at most the later stages' copies are outstanding
        const int ahead = (n_local - 1 - k) < (S - 1) ? (n_local - 1 - k) : (S - 1);
        if (S == 4 && ahead >= 3) wait_vmem<3 * dma_per_stage<F>()>();
        else if (S == 4 && ahead == 2) wait_vmem<2 * dma_per_stage<F>()>();
        else if (ahead >= 1) wait_vmem<dma_per_stage<F>()>();
        else wait_vmem<0>();
        const uint32_t slot = uint32_t(k & (S - 1));
        if constexpr (D == 128) {
            if (append && k == k_new_local && lane < 16) {
                // the staged page holds what the pools held before this step
                lds_u8* st0 = (lds_u8*)(ring + slot * kStage);
                const int pg = ((pos_new - start) >> 4) & 1;
                place_token<F>(st0 + pg * 2 * Fmt<F>::kTile, st0 + 4 * Fmt<F>::kTile + pg * Fmt<F>::kScaleBlock,
                               pos_new & 15, lane, tok);
            }
        }
        StageRegs<regs_fmt<F>()> c;
        stage_read(c, ring_addr + slot * kStage, lane);
        if (k + S < n_local) {
            // refill this slot with iteration k+S while iteration k computes
            const int kn = k + S;
            if ((kn & 31) == 0) {
                // the next chunk's copy is older than every stage in flight,
                // so the wait at the top of this iteration covered it
                ids = clamp_ids(read_page_ids(ids_addr, lane), p.num_pages);
                if (kn + 32 < n_local) copy_page_ids<ws>(ids_slot, pt_row, first_page, n_pages, woff, (kn >> 5) + 1, lane);
            }
            const int s = 2 * (kn & 31);
            const int64_t id0 = __builtin_amdgcn_readlane(ids, s);
            const int64_t id1 = __builtin_amdgcn_readlane(ids, s + 1);
            if (pre)
                stage_issue<F, kPageShared>(ring + slot * kStage, p.codes, p.scales, id0 * tiles_per_page + head_tile,
                                            id1 * tiles_per_page + head_tile, lane);
            else
                stage_issue<F, kPageStream>(ring + slot * kStage, p.codes, p.scales,
                                            id0 * tiles_per_page + head_tile, id1 * tiles_per_page + head_tile, lane);
        }

        if constexpr (PROBE) {
            chk ^= fold_words(c);
            continue;
        }

        // ---- QK^T: raw scores (the softmax scale is applied in the exponent)
        const v4f s0 = qk_page(c, 0, qop);
        const v4f s1 = qk_page(c, 1, qop);
        float x[8];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            x[i] = s0[i];
            x[4 + i] = s1[i];
        }
        uint32_t vs0 = 0, vs1 = 0;   // V scale bytes of the lane's 4 tokens per page (FP4)
        if constexpr (regs_fmt<F>() == kFp4) {
            vs0 = c.vs[0];
            vs1 = c.vs[1];
        }
        const int it = woff + ws * k;
        const int tok0 = start + 32 * it + 4 * g4;   // token of x[0]; x[4] is tok0 + 16
        if (__builtin_amdgcn_ballot_w64(start + 32 * it + 32 > lim) != 0) {
            // scores past the column's last token (the partition end, or a
            // prefix column's own length)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                if (tok0 + i >= lim) x[i] = -__builtin_inff();
                if (tok0 + 16 + i >= lim) x[4 + i] = -__builtin_inff();
            }
            if (start + 32 * it + 32 > end) {
                // tokens past the end: no column reads their V
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    if (tok0 + i >= end) {
                        vs0 &= ~(0xFFu << (8 * i));
                        zero_token(c, 0, i);
                    }
                    if (tok0 + 16 + i >= end) {
                        vs1 &= ~(0xFFu << (8 * i));
                        zero_token(c, 1, i);
                    }
                }
            }
        }

        // ---- online softmax (log2 domain, m_run in scaled units), lazy rescale:
        // the running max of a column moves only when a score exceeds it by
        // more than kLazyRescale; a wave-wide vote skips the cross-lane maximum
        // when no lane holds such a score (then no column would move).  m_run
        // is a rounded scaled score, so every rounded scaled score is at most
        // m_run + kLazyRescale (+ the rounding of that sum: 16 in all).
        float smax = x[0];
#pragma unroll
        for (int i = 1; i < 8; ++i) smax = __builtin_fmaxf(smax, x[i]);
        if (__builtin_amdgcn_ballot_w64(smax * sl2 > m_run + kLazyRescale) != 0) {
            const float mloc = max_across_groups(smax) * sl2;
            if (mloc > m_run + kLazyRescale) {
                const float alpha = __builtin_amdgcn_exp2f(m_run - mloc);
                acc_l *= alpha;
#pragma unroll
                for (int j = 0; j < kAccTiles; ++j) acc[j] *= alpha;
                m_run = mloc;
            }
            big_max = __builtin_amdgcn_ballot_w64(__builtin_fabsf(m_run) >= 0x1p20f && m_run != kNoMax) != 0;
        }
        float pr[8];
        if (!big_max) {
            // the fused form sees the exact product x * sl2, within 2^-4 of
            // the rounded one below 2^20 (a column still at kNoMax has only
            // masked scores)
#pragma unroll
            for (int i = 0; i < 8; ++i) pr[i] = __builtin_amdgcn_exp2f(__builtin_fmaf(x[i], sl2, -m_run));
        } else {
            // scores of 2^20 and more: the exact product can sit half an ulp
            // (over 128 from 2^32 on) away from every float, so round the
            // product first, as m_run was, and subtract (not fused)
#pragma clang fp contract(off)
#pragma unroll
            for (int i = 0; i < 8; ++i) pr[i] = __builtin_amdgcn_exp2f(x[i] * sl2 - m_run);
        }
        uint32_t phi[4], plo[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) split_p(pr[2 * r], pr[2 * r + 1], phi[r], plo[r]);
        const v8bf Phi = __builtin_bit_cast(v8bf, uint4{phi[0], phi[1], phi[2], phi[3]});
        const v8bf Plo = __builtin_bit_cast(v8bf, uint4{plo[0], plo[1], plo[2], plo[3]});
        acc_l = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones, Phi, acc_l, 0, 0, 0);
        acc_l = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones, Plo, acc_l, 0, 0, 0);

        // ---- V to BF16 pairs, then PV on bf16 MFMA
        if constexpr (F == kFp4d64 || F == kFp4d256) {
            // one channel block per lane (two for head size 256), its V scale
            // bytes already masked past the end
#pragma unroll
            for (int bl = 0; bl < (F == kFp4d256 ? 2 : 1); ++bl) {
                uint32_t w0, w1;
                uint4 v0, v1;
                if constexpr (F == kFp4d256) {
                    w0 = c.vs[0][bl];
                    w1 = c.vs[1][bl];
                    v0 = c.v[0][bl];
                    v1 = c.v[1][bl];
                } else {
                    w0 = c.vs[0];
                    w1 = c.vs[1];
                    v0 = c.v[0];
                    v1 = c.v[1];
                }
                float sc[2][4];
                sc[0][0] = byte_scale0(w0, k23);
                sc[0][1] = byte_scale1(w0, k23);
                sc[0][2] = byte_scale2(w0, k23);
                sc[0][3] = byte_scale3(w0, k23);
                sc[1][0] = byte_scale0(w1, k23);
                sc[1][1] = byte_scale1(w1, k23);
                sc[1][2] = byte_scale2(w1, k23);
                sc[1][3] = byte_scale3(w1, k23);
                pv_pair_fp4<0>(v0, v1, sc, Phi, Plo, acc[8 * bl + 0], acc[8 * bl + 1]);
                pv_pair_fp4<1>(v0, v1, sc, Phi, Plo, acc[8 * bl + 2], acc[8 * bl + 3]);
                pv_pair_fp4<2>(v0, v1, sc, Phi, Plo, acc[8 * bl + 4], acc[8 * bl + 5]);
                pv_pair_fp4<3>(v0, v1, sc, Phi, Plo, acc[8 * bl + 6], acc[8 * bl + 7]);
            }
        } else {
            float sc[2][4];
            sc[0][0] = byte_scale0(vs0, k23);
            sc[0][1] = byte_scale1(vs0, k23);
            sc[0][2] = byte_scale2(vs0, k23);
            sc[0][3] = byte_scale3(vs0, k23);
            sc[1][0] = byte_scale0(vs1, k23);
            sc[1][1] = byte_scale1(vs1, k23);
            sc[1][2] = byte_scale2(vs1, k23);
            sc[1][3] = byte_scale3(vs1, k23);
            pv_pair<0>(c, sc, Phi, Plo, acc[0], acc[1]);
            pv_pair<1>(c, sc, Phi, Plo, acc[2], acc[3]);
            pv_pair<2>(c, sc, Phi, Plo, acc[4], acc[5]);
            pv_pair<3>(c, sc, Phi, Plo, acc[6], acc[7]);
        }
    }

    if constexpr (PROBE) {
#pragma unroll
        for (int s = 1; s < 64; s <<= 1) chk ^= uint32_t(__shfl_xor(int(chk), s));
        if (lane == 0) p.probe_sink[int64_t(lin) * W + wave] = chk;
        return;
    }
    const float l_run = acc_l[0];   // the column sum, in every lane of the column
    // ---------------- merge the waves through LDS (the rings are free now).
    // WP: the block's W partitions (an idle wave holds m = kNoMax, l = 0 and
    // zero accumulators, so its weight is 0) into one partial per block.
    __syncthreads();
    float* red_acc = reinterpret_cast<float*>(smem);
    constexpr int kAS = DA + 1;   // LDS row stride (floats) of the merge buffer
    static_assert(W * 16 * kAS * 4 <= W * ring_bytes<F, S>(), "merge buffer aliases the staging rings");
    if (g4 == 0) {
        red_m[wave][n] = m_run;
        red_l[wave][n] = l_run;
    }
    // acc[8 bl + j][i] of lane (n, g4) is O^T[channel 128 bl + 8*(4*g4+i) + j][head n]
#pragma unroll
    for (int bl = 0; bl < kAccTiles / 8; ++bl) {
#pragma unroll
        for (int j = 0; j < 8; ++j) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                // head size 64: rows of channel blocks 8..15 (g4 >= 2) do not exist
                if (DA != 64 || g4 < 2) red_acc[(wave * 16 + n) * kAS + 128 * bl + 32 * g4 + 8 * i + j] = acc[8 * bl + j][i];
            }
        }
    }
    __syncthreads();

#pragma unroll
    for (int h = 0; h < kQRounds; ++h) {
        const int r = (tid >> 4) + h * (kThreads / 16);   // query row of the block
        const int L = tid & 15;                           // channels N L .. N L + N - 1
        int rb, hq;
        if (r >= 16 || !row_of(r, rb, hq)) continue;     // whole 16-lane rows skip together
        float M = red_m[0][r];
#pragma unroll
        for (int w = 1; w < W; ++w) M = __builtin_fmaxf(M, red_m[w][r]);
        float f[W];
        float lsum = 0.f;
#pragma unroll
        for (int w = 0; w < W; ++w) {
            f[w] = __builtin_amdgcn_exp2f(red_m[w][r] - M);
            lsum += f[w] * red_l[w][r];
        }
        const int c0 = (kPair && r >= 8) ? 64 : 0;   // head B's channels are 64..127 of the accumulators
        float o[N];
#pragma unroll
        for (int cc = 0; cc < N; ++cc) {
            float s = 0.f;
#pragma unroll
            for (int w = 0; w < W; ++w) s += f[w] * red_acc[(w * 16 + r) * kAS + c0 + N * L + cc];
            o[cc] = s;
        }
        if (in_place) {
            // the whole context is in this block: finish here
            finish_row<N>(p, o, lsum, L);
            write_out<N>(p, int64_t(rb) * p.num_q_heads + hq, L, o);
        } else {
            // several partitions: publish this one for the merge kernel
            // the wave grid: one slot per block of W partitions
            const int slot = pre ? p.suffix_partitions + part : WP ? first_part / W : part;
            const int64_t prow = (int64_t(rb) * p.num_q_heads + hq) * p.num_partitions + slot;
            float4* dst = reinterpret_cast<float4*>(p.part_acc + prow * D + N * L);
#pragma unroll
            for (int i = 0; i < N / 4; ++i) dst[i] = make_float4(o[4 * i], o[4 * i + 1], o[4 * i + 2], o[4 * i + 3]);
            if (L == 0) *reinterpret_cast<float2*>(p.part_ml + prow * 2) = make_float2(M, lsum);
        }
    }
}

// ---------------------------------------------------------------------------
// Prototype: PV on the block-scaled matrix instruction (FP4 cache, head size
// 128, plain decode).  QK^T and the online softmax are those of
// decode_kernel<kFp4>; PV runs on v_mfma_scale_f32_16x16x128_f8f6f4 with the
// raw E2M1 V codes as operand A (rows = 16 channels of a tile, k = tokens,
// scale byte 127) and P as operand B in FP8.  V's UE8M0 scale varies per
// (token, 32-channel group) along the contraction, which the instruction's
// per-(row, 32-k block) scales cannot carry, so it goes into P: per channel
// group g, P'_g = P * 2^(E_V(token, g) - 127), split into four FP8 terms
// t_k = fp8(r_k), r_{k+1} = (r_k - t_k) * 16, whose B scale bytes 127 - 4k undo
// the shifts (about 16 significant bits of P', as the BF16 hi + lo split of
// the BF16 path).  The running maximum moves eagerly, so that P <= 1 and
// P' <= 2^(E_V - 127) stays within FP8's 448.  K = 128 is filled with the 128 tokens of 4 consecutive
// iterations of the wave: the B lane (column n, group g4) puts its own 8 P
// values of iteration u into bytes 8u .. 8u + 7 (no exchange between lanes),
// and the matching A rows come from ds_read_b64_tr_b4: each iteration the
// V codes are written to a per-wave area as 8-byte rows (16 channels of one
// token), and a transposed read gives lane r of a 16-lane group channel r of
// the 16 tokens its group addressed.
template <int U> struct MxPvSlots {};

// Stage registers of the prototype: K as decode_kernel<kFp4>, V codes, and
// the V scale bytes of the lane's 4 tokens of each page for all 4 groups.
struct MxPvStage {
    uint4 k[2], v[2];
    uint32_t ks[2];
    uint32_t vs[2][4];   // [page][group]: bytes = tokens 4 g4 .. 4 g4 + 3
};

__device__ __forceinline__ void mxpv_stage_read(MxPvStage& r, uint32_t stage_addr, int lane) {
    const uint32_t ac = stage_addr + 16 * lane;
    const uint32_t ak = stage_addr + lane;
    const uint32_t av = stage_addr + 4096 + kTileScales + 4 * (lane >> 4);
    asm volatile(
        "ds_read_b128 %0, %14\n\t"
        "ds_read_b128 %1, %14 offset:1024\n\t"
        "ds_read_b128 %2, %14 offset:2048\n\t"
        "ds_read_b128 %3, %14 offset:3072\n\t"
        "ds_read_u8 %4, %15 offset:4096\n\t"
        "ds_read_u8 %5, %15 offset:4224\n\t"
        "ds_read_b32 %6, %16\n\t"
        "ds_read_b32 %7, %16 offset:16\n\t"
        "ds_read_b32 %8, %16 offset:32\n\t"
        "ds_read_b32 %9, %16 offset:48\n\t"
        "ds_read_b32 %10, %16 offset:128\n\t"
        "ds_read_b32 %11, %16 offset:144\n\t"
        "ds_read_b32 %12, %16 offset:160\n\t"
        "ds_read_b32 %13, %16 offset:176\n\t"
        "s_waitcnt lgkmcnt(0)"
        : "=&v"(r.k[0]), "=&v"(r.v[0]), "=&v"(r.k[1]), "=&v"(r.v[1]), "=&v"(r.ks[0]), "=&v"(r.ks[1]),
          "=&v"(r.vs[0][0]), "=&v"(r.vs[0][1]), "=&v"(r.vs[0][2]), "=&v"(r.vs[0][3]), "=&v"(r.vs[1][0]),
          "=&v"(r.vs[1][1]), "=&v"(r.vs[1][2]), "=&v"(r.vs[1][3])
        : "v"(ac), "v"(ak), "v"(av)
        : "memory");
}

typedef int v2i_t __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) v2i_t* lds_v2i_ptr;
typedef short v2s_t __attribute__((ext_vector_type(2)));

// Four FP8 E4M3 bytes of r0..r3 (round to nearest even).
__device__ __forceinline__ uint32_t fp8x4(float r0, float r1, float r2, float r3) {
    v2s_t w = {0, 0};
    w = __builtin_amdgcn_cvt_scalef32_pk_fp8_f32(w, r0, r1, 1.0f, false);
    w = __builtin_amdgcn_cvt_scalef32_pk_fp8_f32(w, r2, r3, 1.0f, true);
    return __builtin_bit_cast(uint32_t, w);
}

__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2))) decode_kernel_mxpv(DecodeParams p) {
    constexpr int W = 4, S = 2;
    constexpr int kStage = stage_bytes<kFp4>();
    constexpr int kRows = 2 * 8 * 16 * 8;   // per wave: [page][tile][token][8 B]
    const int lin = blockIdx.x;
    const int hk = lin % p.num_kv_heads;
    const int row = lin / p.num_kv_heads;
    const int b = row % p.batch;
    const int part = row / p.batch;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int G = p.group;
    int ctx = p.context_lens[b];
    ctx = ctx < p.max_context ? ctx : p.max_context;
    const int start = part * p.partition_tokens;
    if (start >= ctx) {
        if (ctx <= 0 && part == 0) {
            for (int r = tid >> 4; r < G; r += 16) {
                float z[8];
#pragma unroll
                for (int i = 0; i < 8; ++i) z[i] = 0.f;
                write_out<8>(p, int64_t(b) * p.num_q_heads + hk * G + r, tid & 15, z);
            }
        }
        return;
    }
    const int end = (start + p.partition_tokens) < ctx ? (start + p.partition_tokens) : ctx;
    const bool in_place = ctx <= p.partition_tokens;

    __shared__ __attribute__((aligned(16))) uint8_t smem[W * ring_bytes<kFp4, S>()];
    __shared__ __attribute__((aligned(16))) uint8_t q_lds[q_lds_bytes<kFp4>()];
    __shared__ __attribute__((aligned(16))) uint8_t ids_lds[W * kIdsSlot];
    __shared__ __attribute__((aligned(16))) uint8_t rows_lds[W * kRows];
    __shared__ float red_m[W][16];
    __shared__ float red_l[W][16];

    // ---- query: as decode_kernel<kFp4> (rotate, FP8 cast, B-operand order)
    {
        const int qr = tid >> 4, qL = tid & 15;
        float qx[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) qx[i] = 0.f;
        uint32_t lo = 0u, hi = 0u;
        if (qr < G) {
            const int64_t elem = (int64_t(b) * p.num_q_heads + hk * G + qr) * kHeadDim + 8 * qL;
            if (p.q_dtype == 3) {
                const uint2 w = *reinterpret_cast<const uint2*>(static_cast<const uint8_t*>(p.q) + elem);
                lo = w.x;
                hi = w.y;
            } else {
                if (p.q_dtype == 0) load_x8<0>(p.q, elem, qx);
                else if (p.q_dtype == 1) load_x8<1>(p.q, elem, qx);
                else load_x8<2>(p.q, elem, qx);
                wht128_x8(qx, qL);
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    lo |= e4m3_byte(qx[i]) << (8 * i);
                    hi |= e4m3_byte(qx[i + 4]) << (8 * i);
                }
            }
        }
        const int ch = 8 * qL;
        const int g = (ch & 63) >> 4;
        const int e0 = (ch & 15) + (ch >= 64 ? 16 : 0);
        *reinterpret_cast<uint2*>(q_lds + (g * 16 + qr) * 32 + e0) = make_uint2(lo, hi);
    }

    const int first_page = start >> 4;
    const int n_pages = (end - start + 15) >> 4;
    const int n_iter = (n_pages + 1) >> 1;
    const int n_local = wave < n_iter ? (n_iter - wave + W - 1) / W : 0;
    const int32_t* pt_row = p.page_table + int64_t(b) * p.max_pages_per_seq;
    const int g4 = lane >> 4;
    const int n = lane & 15;
    uint8_t* ring = smem + wave * ring_bytes<kFp4, S>();
    const uint32_t ring_addr = uint32_t(reinterpret_cast<uintptr_t>((lds_ptr_t)ring));
    const int64_t head_tile = int64_t(hk) * 2;
    const int64_t tiles_per_page = int64_t(p.num_kv_heads) * 2;
    uint8_t* ids_slot = ids_lds + wave * kIdsSlot;
    const uint32_t ids_addr = uint32_t(reinterpret_cast<uintptr_t>((lds_ptr_t)ids_slot));
    int32_t ids = 0;
    if (n_local > 0) {
        ids = load_page_ids<W>(pt_row, first_page, n_pages, wave, 0, lane);
        if (n_local > 32) copy_page_ids<W>(ids_slot, pt_row, first_page, n_pages, wave, 1, lane);
    }
    __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
    ids = clamp_ids(ids, p.num_pages);
    for (int s2 = 0; s2 < S && s2 < n_local; ++s2) {
        const int64_t id0 = __builtin_amdgcn_readlane(ids, 2 * s2);
        const int64_t id1 = __builtin_amdgcn_readlane(ids, 2 * s2 + 1);
        stage_issue<kFp4>(ring + s2 * kStage, p.codes, p.scales, id0 * tiles_per_page + head_tile,
                          id1 * tiles_per_page + head_tile, lane);
    }
    __syncthreads();
    QOperand<kFp4> qop;
    {
        const uint4* src = reinterpret_cast<const uint4*>(q_lds + lane * 32);
        const uint4 a = src[0], c = src[1];
        qop.q = v8i{int(a.x), int(a.y), int(a.z), int(a.w), int(c.x), int(c.y), int(c.z), int(c.w)};
    }

    // rows area of this wave: row (page, tile, token) at ((page * 8 + tile) * 16 + token) * 8
    uint8_t* rows = rows_lds + wave * kRows;
    const uint32_t rows_addr = uint32_t(reinterpret_cast<uintptr_t>((lds_ptr_t)rows));
    // this lane's writes: token 4 g4 + t of page pg, channels 8n..8n+7 -> tile n/2, byte (n%2)*4
    const uint32_t wr_addr = rows_addr + ((n >> 1) * 16 + 4 * g4) * 8 + (n & 1) * 4;
    // this lane's transposed-read row (row index n of its 16-lane group): nibble n of the result is
    // k-slot q = n (n < 8) or 16 + n - 8 of its 32-slot k-block half; page (n / 4) % 2, token offset
    // 8 (g4 % 2) + 4 (n / 8) + n % 4
    const uint32_t rd_addr =
        rows_addr + (((n >> 2) & 1) * 8 * 16 + (8 * (g4 & 1) + 4 * (n >> 3) + (n & 3))) * 8;

    const float sl2 = p.scale_log2;
    constexpr float kNoMax = -1e30f;
    float m_run = kNoMax;
    bool big_max = false;
    float l_lane = 0.f;     // this lane's share of its column's softmax sum
    v4f acc[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[j] = v4f{0.f, 0.f, 0.f, 0.f};
    uint32_t av[8][4];      // FP4 A operands of the 8 channel tiles (32 tokens x 16 channels per lane group)
#pragma unroll
    for (int j = 0; j < 8; ++j) av[j][0] = av[j][1] = av[j][2] = av[j][3] = 0u;
    float pv[32];           // P of the super-iteration, index 8 u + 4 page + i
    uint32_t ev[4][8];      // V scale bytes, [group][2 u + page], byte i = token 4 g4 + i
    const uint32_t k23 = 23u;

    for (int ks = 0; ks < n_local; ks += 4) {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int k = ks + u;
            if (k >= n_local) {
#pragma unroll
                for (int i = 0; i < 8; ++i) pv[8 * u + i] = 0.f;
#pragma unroll
                for (int g = 0; g < 4; ++g) ev[g][2 * u] = ev[g][2 * u + 1] = 0u;
                continue;
            }
            const int ahead = (n_local - 1 - k) < (S - 1) ? (n_local - 1 - k) : (S - 1);
            if (ahead >= 1) wait_vmem<dma_per_stage<kFp4>()>();
            else wait_vmem<0>();
            const uint32_t slot = uint32_t(k & (S - 1));
            MxPvStage c;
            mxpv_stage_read(c, ring_addr + slot * kStage, lane);
            if (k + S < n_local) {
                const int kn = k + S;
                if ((kn & 31) == 0) {
                    ids = clamp_ids(read_page_ids(ids_addr, lane), p.num_pages);
                    if (kn + 32 < n_local)
                        copy_page_ids<W>(ids_slot, pt_row, first_page, n_pages, wave, (kn >> 5) + 1, lane);
                }
                const int s2 = 2 * (kn & 31);
                const int64_t id0 = __builtin_amdgcn_readlane(ids, s2);
                const int64_t id1 = __builtin_amdgcn_readlane(ids, s2 + 1);
                stage_issue<kFp4>(ring + slot * kStage, p.codes, p.scales, id0 * tiles_per_page + head_tile,
                                  id1 * tiles_per_page + head_tile, lane);
            }
            // V codes -> rows area (8-byte rows: 16 channels of one token), then the transposed reads
#pragma unroll
            for (int pg = 0; pg < 2; ++pg)
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    const uint32_t a = wr_addr + pg * 8 * 16 * 8 + t * 8;
                    const uint32_t w = dword(c.v[pg], t);
                    asm volatile("ds_write_b32 %0, %1" ::"v"(a), "v"(w) : "memory");
                }
            asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
            // lanes of k-block j take this iteration's tokens when j / 2 == u / 2, into dwords u % 2
            // and 2 + u % 2 of their A operands
            const bool take = (g4 >> 1) == (u >> 1);
#pragma unroll
            for (int tile = 0; tile < 8; ++tile) {
                const v2i_t r = __builtin_amdgcn_ds_read_tr4_b64_v2i32((lds_v2i_ptr)(uintptr_t)(rd_addr + tile * 128));
                if (take) {
                    av[tile][u & 1] = uint32_t(r.x);
                    av[tile][2 + (u & 1)] = uint32_t(r.y);
                }
            }

            // ---- QK^T and the online softmax as decode_kernel<kFp4>
            const v8i a0 = {int(c.k[0].x), int(c.k[0].y), int(c.k[0].z), int(c.k[0].w), 0, 0, 0, 0};
            const v8i a1 = {int(c.k[1].x), int(c.k[1].y), int(c.k[1].z), int(c.k[1].w), 0, 0, 0, 0};
            const v4f zero = {0.f, 0.f, 0.f, 0.f};
            const v4f s0 = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a0, qop.q, zero, 4, 0, 0, int(c.ks[0]), 0, 127);
            const v4f s1 = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a1, qop.q, zero, 4, 0, 0, int(c.ks[1]), 0, 127);
            float x[8];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                x[i] = s0[i];
                x[4 + i] = s1[i];
            }
            const int it = wave + W * k;
            const int tok0 = start + 32 * it + 4 * g4;
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                ev[g][2 * u] = c.vs[0][g];
                ev[g][2 * u + 1] = c.vs[1][g];
            }
            if (__builtin_amdgcn_ballot_w64(start + 32 * it + 32 > end) != 0) {
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    if (tok0 + i >= end) {
                        x[i] = -__builtin_inff();
#pragma unroll
                        for (int g = 0; g < 4; ++g) ev[g][2 * u] &= ~(0xFFu << (8 * i));
                    }
                    if (tok0 + 16 + i >= end) {
                        x[4 + i] = -__builtin_inff();
#pragma unroll
                        for (int g = 0; g < 4; ++g) ev[g][2 * u + 1] &= ~(0xFFu << (8 * i));
                    }
                }
            }
            float smax = x[0];
#pragma unroll
            for (int i = 1; i < 8; ++i) smax = __builtin_fmaxf(smax, x[i]);
            // eager rescale (no lazy threshold): P <= 1, so P * 2^(E_V - 127) stays in the FP8 range
            if (__builtin_amdgcn_ballot_w64(smax * sl2 > m_run) != 0) {
                const float mloc = max_across_groups(smax) * sl2;
                if (mloc > m_run) {
                    const float alpha = __builtin_amdgcn_exp2f(m_run - mloc);
                    l_lane *= alpha;
#pragma unroll
                    for (int j = 0; j < 8; ++j) acc[j] *= alpha;
#pragma unroll
                    for (int e = 0; e < 8 * u; ++e) pv[e] *= alpha;   // pending P of this super-iteration
                    m_run = mloc;
                }
                big_max = __builtin_amdgcn_ballot_w64(__builtin_fabsf(m_run) >= 0x1p20f && m_run != kNoMax) != 0;
            }
            if (!big_max) {
#pragma unroll
                for (int i = 0; i < 8; ++i) pv[8 * u + i] = __builtin_amdgcn_exp2f(__builtin_fmaf(x[i], sl2, -m_run));
            } else {
#pragma clang fp contract(off)
#pragma unroll
                for (int i = 0; i < 8; ++i) pv[8 * u + i] = __builtin_amdgcn_exp2f(x[i] * sl2 - m_run);
            }
#pragma unroll
            for (int i = 0; i < 8; ++i) l_lane += pv[8 * u + i];
        }

        // ---- PV over the super-iteration's 128 tokens, channel group by channel group
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            float r[32];
#pragma unroll
            for (int w = 0; w < 8; ++w) {
                r[4 * w + 0] = pv[4 * w + 0] * byte_scale0(ev[g][w], k23);
                r[4 * w + 1] = pv[4 * w + 1] * byte_scale1(ev[g][w], k23);
                r[4 * w + 2] = pv[4 * w + 2] * byte_scale2(ev[g][w], k23);
                r[4 * w + 3] = pv[4 * w + 3] * byte_scale3(ev[g][w], k23);
            }
#pragma unroll
            for (int term = 0; term < 4; ++term) {
                uint32_t bw[8];
#pragma unroll
                for (int w = 0; w < 8; ++w) bw[w] = fp8x4(r[4 * w], r[4 * w + 1], r[4 * w + 2], r[4 * w + 3]);
                if (term < 3) {
#pragma unroll
                    for (int w = 0; w < 8; ++w) {
                        const v2s_t lo = __builtin_bit_cast(v2s_t, bw[w]);
                        const v2f b0 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp8(bw[w], 16.0f, false);
                        const v2f b1 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp8(bw[w], 16.0f, true);
                        (void)lo;
                        r[4 * w + 0] = __builtin_fmaf(r[4 * w + 0], 16.0f, -b0[0]);
                        r[4 * w + 1] = __builtin_fmaf(r[4 * w + 1], 16.0f, -b0[1]);
                        r[4 * w + 2] = __builtin_fmaf(r[4 * w + 2], 16.0f, -b1[0]);
                        r[4 * w + 3] = __builtin_fmaf(r[4 * w + 3], 16.0f, -b1[1]);
                    }
                }
                const v8i bop = {int(bw[0]), int(bw[1]), int(bw[2]), int(bw[3]), int(bw[4]), int(bw[5]), int(bw[6]),
                                 int(bw[7])};
#pragma unroll
                for (int tt = 0; tt < 2; ++tt) {
                    const int tile = 2 * g + tt;
                    const v8i aop = {int(av[tile][0]), int(av[tile][1]), int(av[tile][2]), int(av[tile][3]), 0, 0, 0, 0};
                    acc[tile] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(aop, bop, acc[tile], 4, 0, 0, 127, 0,
                                                                                 127 - 4 * term);
                }
            }
        }
    }

    // ---- merge the waves through LDS (the rings are free now)
    float l_run;
    {
        float a = l_lane, bb = l_lane;
        swap16(a, bb);
        const float s1 = a + bb;
        float c2 = s1, d2 = s1;
        swap32(c2, d2);
        l_run = c2 + d2;
    }
    __syncthreads();
    float* red_acc = reinterpret_cast<float*>(smem);
    constexpr int kAS = 129;
    if (g4 == 0) {
        red_m[wave][n] = m_run;
        red_l[wave][n] = l_run;
    }
    // acc[tile][i] of lane (n, g4) is O^T[channel 16 tile + 4 g4 + i][head n]
#pragma unroll
    for (int tile = 0; tile < 8; ++tile)
#pragma unroll
        for (int i = 0; i < 4; ++i) red_acc[(wave * 16 + n) * kAS + 16 * tile + 4 * g4 + i] = acc[tile][i];
    __syncthreads();
    {
        const int r = tid >> 4;
        const int L = tid & 15;
        if (r < G) {
            float M = red_m[0][r];
#pragma unroll
            for (int w = 1; w < W; ++w) M = __builtin_fmaxf(M, red_m[w][r]);
            float f[W];
            float lsum = 0.f;
#pragma unroll
            for (int w = 0; w < W; ++w) {
                f[w] = __builtin_amdgcn_exp2f(red_m[w][r] - M);
                lsum += f[w] * red_l[w][r];
            }
            float o[8];
#pragma unroll
            for (int cc = 0; cc < 8; ++cc) {
                float sacc = 0.f;
#pragma unroll
                for (int w = 0; w < W; ++w) sacc += f[w] * red_acc[(w * 16 + r) * kAS + 8 * L + cc];
                o[cc] = sacc;
            }
            const int hq = hk * G + r;
            if (in_place) {
                finish_row<8>(p, o, lsum, L);
                write_out<8>(p, int64_t(b) * p.num_q_heads + hq, L, o);
            } else {
                const int64_t prow = (int64_t(b) * p.num_q_heads + hq) * p.num_partitions + part;
                float4* dst = reinterpret_cast<float4*>(p.part_acc + prow * 128 + 8 * L);
                dst[0] = make_float4(o[0], o[1], o[2], o[3]);
                dst[1] = make_float4(o[4], o[5], o[6], o[7]);
                if (L == 0) *reinterpret_cast<float2*>(p.part_ml + prow * 2) = make_float2(M, lsum);
            }
        }
    }
}

hipError_t launch_decode_partials_mxpv(const DecodeParams& p, hipStream_t stream) {
    const dim3 grid{unsigned(int64_t(p.suffix_partitions) * p.num_kv_heads * p.batch)};
    launch_kernel(decode_kernel_mxpv, grid, dim3(256), stream, p);
    return hipGetLastError();
}

// Merge the partitions of every (sequence, query head) with more than one:
// online over the partitions (loads independent of the running state, so
// they overlap), then finish the row.  One 16-lane row per query head.
// Cascade decode: the context partitions after the tokens the prefix serves,
// then that sequence's prefix partitions; always merged (every block of a
// cascade call writes a partial).
template <int D>
__global__ void __launch_bounds__(256) merge_kernel(DecodeParams p) {
    constexpr int N = D / 16;   // channels per lane
    const int hk = blockIdx.x;
    const int b = blockIdx.y;
    const int r = threadIdx.x >> 4;
    const int L = threadIdx.x & 15;
    if (r >= p.group) return;   // whole 16-lane rows leave together
    int ctx = p.context_lens[b];
    ctx = ctx < p.max_context ? ctx : p.max_context;
    int np = ctx > 0 ? (ctx + p.partition_tokens - 1) / p.partition_tokens : 0;
    int first = 0, nq = 0;
    if (p.prefix_pages != nullptr) {
        int pl = p.prefix_lens[b];
        pl = pl < p.prefix_tokens ? pl : p.prefix_tokens;
        pl = pl < ctx - 1 ? pl : ctx - 1;
        pl = pl > 0 ? (pl & ~15) : 0;
        first = pl / p.partition_tokens;
        nq = (pl + p.prefix_partition - 1) / p.prefix_partition;
        if (np - first + nq <= 0) return;   // empty context: written by the decode kernel
    } else {
        // the wave grid reduces W partitions per block into one slot
        if (p.wave_parts > 1) np = (np + p.wave_parts - 1) / p.wave_parts;
        if (np <= 1) return;                // finished by the decode kernel
    }
    const int hq = hk * p.group + r;
    const int64_t row0 = (int64_t(b) * p.num_q_heads + hq) * p.num_partitions;
    float M = -__builtin_inff();
    float lsum = 0.f;
    float o[N];
#pragma unroll
    for (int i = 0; i < N; ++i) o[i] = 0.f;
    auto merge_slot = [&](int slot) {
        const float2 ml = *reinterpret_cast<const float2*>(p.part_ml + (row0 + slot) * 2);
        const float4* src = reinterpret_cast<const float4*>(p.part_acc + (row0 + slot) * D + N * L);
        float4 a[N / 4];
#pragma unroll
        for (int i = 0; i < N / 4; ++i) a[i] = src[i];
        const float Mn = __builtin_fmaxf(M, ml.x);
        const float fo = __builtin_amdgcn_exp2f(M - Mn);
        const float fn = __builtin_amdgcn_exp2f(ml.x - Mn);
        lsum = lsum * fo + ml.y * fn;
#pragma unroll
        for (int i = 0; i < N / 4; ++i) {
            o[4 * i] = o[4 * i] * fo + a[i].x * fn;
            o[4 * i + 1] = o[4 * i + 1] * fo + a[i].y * fn;
            o[4 * i + 2] = o[4 * i + 2] * fo + a[i].z * fn;
            o[4 * i + 3] = o[4 * i + 3] * fo + a[i].w * fn;
        }
        M = Mn;
    };
#pragma unroll 4
    for (int q = first; q < np; ++q) merge_slot(q);
    for (int q = 0; q < nq; ++q) merge_slot(p.suffix_partitions + q);
    finish_row<N>(p, o, lsum, L);
    write_out<N>(p, int64_t(b) * p.num_q_heads + hq, L, o);
}

// The rows of a cascade launch in dispatch order (one block).  The tokens
// of context row (part, b) are those of its partition after the prefix's
// tokens and before the context end, as the decode kernel computes them.
// A counting sort over 1024 classes of tokens / partition_tokens puts the
// context rows with the most tokens first (rows of one class in any order:
// each row is computed and stored the same way whichever block takes it); a
// row without tokens stays in the list only as the zero output of an empty
// context (partition 0).  The prefix rows follow (records R + j), then -1
// for the rest.
__global__ void __launch_bounds__(1024) cascade_rows_kernel(DecodeParams p) {
    constexpr int kClasses = 1024;
    __shared__ int hist[kClasses];
    __shared__ int total;
    const int R = p.suffix_partitions * p.batch;
    const int P = p.partition_tokens;
    const int tid = threadIdx.x;
    hist[tid] = 0;
    __syncthreads();
    // tokens of row r, or -1 when the row has nothing to do
    auto row_tokens = [&](int r, int& ctx, int& pl) -> int {
        const int b = r % p.batch, part = r / p.batch;
        ctx = p.context_lens[b];
        ctx = ctx < p.max_context ? ctx : p.max_context;
        pl = p.prefix_lens[b];
        pl = pl < p.prefix_tokens ? pl : p.prefix_tokens;
        pl = pl < ctx - 1 ? pl : ctx - 1;
        pl = pl > 0 ? (pl & ~15) : 0;
        const int s0 = part * P;
        if (s0 + P <= pl) return -1;
        const int start = s0 > pl ? s0 : pl;
        if (start >= ctx) return (ctx <= 0 && part == 0) ? 0 : -1;
        const int end = s0 + P < ctx ? s0 + P : ctx;
        return end - start;
    };
    // class 0: a whole partition; kClasses - 1: the fewest tokens
    auto class_of = [&](int t) {
        const int c = int(int64_t(P - t) * (kClasses - 1) / P);
        return c < 0 ? 0 : (c > kClasses - 1 ? kClasses - 1 : c);
    };
    for (int r = tid; r < R; r += kClasses) {
        int ctx, pl;
        const int t = row_tokens(r, ctx, pl);
        if (t >= 0) atomicAdd(&hist[class_of(t)], 1);
    }
    __syncthreads();
    // prefix sum of the class counts (Hillis-Steele over the 1024 threads)
    const int count = hist[tid];
    int v = count;
    for (int d = 1; d < kClasses; d <<= 1) {
        __syncthreads();
        hist[tid] = v;
        __syncthreads();
        if (tid >= d) v += hist[tid - d];
    }
    __syncthreads();
    if (tid == kClasses - 1) total = v;
    hist[tid] = v - count;   // the first list position of the class
    __syncthreads();
    for (int r = tid; r < R; r += kClasses) {
        int ctx, pl;
        const int t = row_tokens(r, ctx, pl);
        if (t >= 0) {
            const int pos = atomicAdd(&hist[class_of(t)], 1);
            p.cascade_rows[pos] = make_int4(r, ctx, pl, 0);
        }
    }
    const int PR = p.prefix_blocks / p.num_kv_heads;
    for (int j = tid; j < PR; j += kClasses) p.cascade_rows[total + j] = make_int4(R + j, 0, 0, 0);
    for (int i = total + PR + tid; i < R + PR; i += kClasses) p.cascade_rows[i] = make_int4(-1, 0, 0, 0);
}

// Waves per block of a partition launch (the grid choice below, the merge
// launch and the probe's sink words follow it).  The FP4 and FP8 caches at
// head size 128: 8 on the wave grid when it has enough blocks of 8
// partitions and at least 16 partitions, so that a longest context spans
// two blocks or more (fewer block prologues and partial writes per
// partition: 3 % faster on 128k contexts in 4096-token partitions; blocks
// of 8 holding whole contexts were 5 % slower on a ragged batch, whose
// short contexts leave most of such a block's waves idle), else the
// format's kWaves (4), which measured equal on 32k contexts and 2 % faster
// on the MiniMax-like cascade than blocks of 8.  Others: the format's
// kWaves.
static bool wave_grid_with(const DecodeParams& p, int W) {
    if (!p.allow_wave_parts || p.prefix_pages != nullptr || p.head_dim != kHeadDim) return false;
    if (p.kv_fmt != kFp4 && p.kv_fmt != kFp8 && p.kv_fmt != kBf16 && p.kv_fmt != kTq4) return false;
    if (p.num_partitions < W) return false;
    const int64_t blocks = int64_t(p.batch) * p.num_kv_heads * ((p.num_partitions + W - 1) / W);
    return blocks >= 8 * kNumCus;
}
static bool eight_waves(const DecodeParams& p) { return p.num_partitions >= 16 && wave_grid_with(p, 8); }
static int launch_waves(const DecodeParams& p) {
    switch (p.kv_fmt) {
        case kFp8: return eight_waves(p) ? 8 : Fmt<kFp8>::kWaves;
        case kBf16: return Fmt<kBf16>::kWaves;
        case kTq4: return Fmt<kTq4>::kWaves;
        case kFp4d64: return Fmt<kFp4d64>::kWaves;
        case kFp4d64x2: return Fmt<kFp4d64x2>::kWaves;
        case kFp4d256: return Fmt<kFp4d256>::kWaves;
        default: return eight_waves(p) ? 8 : Fmt<kFp4>::kWaves;
    }
}
// The grid of a partition launch: one wave per partition when there are
// enough partitions for W per block and enough such blocks to give every CU
// several (at least 8 per CU), head size 128, no cascade; else one block per
// partition.  The merge launch makes the same choice from the same
// parameters.
static bool choose_wave_parts(const DecodeParams& p) { return wave_grid_with(p, launch_waves(p)); }

// Two ring slots per wave: a 4-slot ring (twice the copies in flight, half
// the blocks per CU) measured no faster on 32k contexts and slower on 16k,
// also with the streaming page copies. PROBE: the same grid with the
// page-gather probe of the kernel (FP4 formats).
constexpr int kRingSlots = 2;
// The wave grid with W waves (partitions) per block.
template <int F, bool PROBE, int W>
static hipError_t launch_wave_grid(const DecodeParams& p, hipStream_t stream) {
    static_assert(occupancy<F, kRingSlots, W>() == Fmt<F>::kOccupancy, "the LDS footprint lowers the occupancy");
    DecodeParams pw = p;
    pw.wave_parts = W;
    const dim3 grid{unsigned(int64_t((p.num_partitions + W - 1) / W) * p.num_kv_heads * p.batch)};
    launch_kernel(decode_kernel<F, kRingSlots, true, PROBE, W>, grid, dim3(64 * W), stream, pw);
    return hipGetLastError();
}
template <int F, bool PROBE = false>
static hipError_t launch_partials(const DecodeParams& p, hipStream_t stream) {
    constexpr int W = Fmt<F>::kWaves;
    static_assert(occupancy<F, kRingSlots, W>() == Fmt<F>::kOccupancy, "the LDS footprint lowers the occupancy");
    if constexpr (head_dim_of<F>() == 128 && F != kFp4d64x2) {
        if (choose_wave_parts(p)) {
            if constexpr (F == kFp4 || F == kFp8) {
                if (launch_waves(p) == 8) return launch_wave_grid<F, PROBE, 8>(p, stream);
            }
            return launch_wave_grid<F, PROBE, W>(p, stream);
        }
    }
    if (p.prefix_pages != nullptr) {
        // the cascade's row list first (a plain launch: the timing hook is the partition kernel's)
        hipLaunchKernelGGL(cascade_rows_kernel, dim3(1), dim3(1024), 0, stream, p);
    }
    const int64_t units = F == kFp4d64x2 ? p.num_kv_heads / 2 : p.num_kv_heads;
    const dim3 grid{unsigned(int64_t(p.prefix_blocks) + int64_t(p.suffix_partitions) * units * p.batch)};
    launch_kernel(decode_kernel<F, kRingSlots, false, PROBE, W>, grid, dim3(64 * W), stream, p);
    return hipGetLastError();
}

int64_t partition_blocks(const DecodeParams& p) {
    const int64_t units = p.kv_fmt == kFp4d64x2 ? p.num_kv_heads / 2 : p.num_kv_heads;
    const int W = launch_waves(p);
    if (choose_wave_parts(p)) return int64_t((p.num_partitions + W - 1) / W) * units * p.batch;
    return int64_t(p.prefix_blocks) + int64_t(p.suffix_partitions) * units * p.batch;
}

int64_t probe_words(const DecodeParams& p) { return int64_t(launch_waves(p)) * partition_blocks(p); }

hipError_t launch_gather_probe(const DecodeParams& p, uint32_t* sink, hipStream_t stream) {
    DecodeParams pp = p;
    pp.probe_sink = sink;
    if (p.kv_fmt == kFp4d64) return launch_partials<kFp4d64, true>(pp, stream);
    if (p.kv_fmt == kFp4d64x2) return launch_partials<kFp4d64x2, true>(pp, stream);
    if (p.kv_fmt == kFp4d256) return launch_partials<kFp4d256, true>(pp, stream);
    if (p.kv_fmt == kFp4) return launch_partials<kFp4, true>(pp, stream);
    return hipErrorInvalidValue;
}

hipError_t launch_decode_partials(const DecodeParams& p, hipStream_t stream) {
    if (p.kv_fmt == kFp8) return launch_partials<kFp8>(p, stream);
    if (p.kv_fmt == kBf16) return launch_partials<kBf16>(p, stream);
    if (p.kv_fmt == kTq4) return launch_partials<kTq4>(p, stream);
    if (p.kv_fmt == kFp4d64) return launch_partials<kFp4d64>(p, stream);
    if (p.kv_fmt == kFp4d64x2) return launch_partials<kFp4d64x2>(p, stream);
    if (p.kv_fmt == kFp4d256) return launch_partials<kFp4d256>(p, stream);
    return launch_partials<kFp4>(p, stream);
}

hipError_t launch_decode_merge(const DecodeParams& p, hipStream_t stream) {
    if (p.num_partitions <= 1 && p.prefix_pages == nullptr) return hipSuccess;   // every sequence was finished in place
    DecodeParams pm = p;
    pm.wave_parts = choose_wave_parts(p) ? launch_waves(p) : 0;
    const dim3 grid{unsigned(p.num_kv_heads), unsigned(p.batch)};
    if (p.head_dim == 64) hipLaunchKernelGGL(merge_kernel<64>, grid, dim3(256), 0, stream, pm);
    else if (p.head_dim == 256) hipLaunchKernelGGL(merge_kernel<256>, grid, dim3(256), 0, stream, pm);
    else hipLaunchKernelGGL(merge_kernel<128>, grid, dim3(256), 0, stream, pm);
    return hipGetLastError();
}

}  // namespace uq
