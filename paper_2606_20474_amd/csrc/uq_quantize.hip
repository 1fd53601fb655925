// uq_quantize.hip -- quantize-on-write into the FP4 cache (paper,
// Algorithm 1, "Write") and the FP8 query preparation (Algorithm 1,
// "Decode", first step).
//
// One 128-vector is handled by 16 lanes holding 8 channels each, so a
// wave64 processes 4 (token, kv head) pairs and a 256-thread block 16.
// Per vector and per K/V: coalesced 16/32-byte loads, the in-register WHT
// butterfly (3 in-lane + 4 cross-lane stages), the group absmax over the 4
// lanes of a 32-channel group, the UE8M0 exponent, E2M1 encoding of 8
// values into one dword, one dword store of codes and one byte store of the
// scale per group.  The path is bound by HBM traffic.
#include "uq_device.hpp"
#include "uq_internal.hpp"

namespace uq {

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
    uint32_t w = 0;
#pragma unroll
    for (int i = 0; i < 8; ++i) w |= e2m1_code(x[i], E) << (4 * i);
    return w;
}

template <int DT>
__global__ void __launch_bounds__(256) quantize_kv_kernel(QuantizeParams p) {
    const int lane16 = threadIdx.x & 15;
    const int64_t vec = int64_t(blockIdx.x) * 16 + (threadIdx.x >> 4);
    const int64_t nvec = p.num_tokens * p.num_kv_heads;
    if (vec >= nvec) return;
    const int64_t t = vec / p.num_kv_heads;
    const int h = int(vec - t * p.num_kv_heads);

    int64_t slot = p.slot_mapping[t];
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

    uint32_t sk, sv;
    const uint32_t wk = quantize_x8(xk, lane16, p.c, true, sk);
    const uint32_t wv = quantize_x8(xv, lane16, p.c, p.rotate_v != 0, sv);

    const int64_t tile = (page * p.num_kv_heads + h) * 2;
    uint8_t* kc = p.codes + tile * kTileCodes;
    uint8_t* vc = kc + kTileCodes;
    uint8_t* ks = p.scales + tile * kTileScales;
    uint8_t* vs = ks + kTileScales;
    const int g = lane16 >> 2;
    // K tile: [group][token][16 B]; this lane's 8 channels are bytes 4*(lane16%4).. of the row.
    *reinterpret_cast<uint32_t*>(kc + (g * kPage + off) * 16 + 4 * (lane16 & 3)) = wk;
    // V tile: [token/4][channel/8][token%4][4 B]; channels 8*lane16..+7 of token `off`.
    *reinterpret_cast<uint32_t*>(vc + ((off >> 2) * 16 + lane16) * 16 + (off & 3) * 4) = wv;
    if ((lane16 & 3) == 0) {
        ks[g * kPage + off] = uint8_t(sk);
        vs[g * kPage + off] = uint8_t(sv);
    }
}

// Writer of the plain comparison caches (FP8 E4M3 with one scale per
// tensor, or BF16), no rotation, in the lane order the decode kernel reads:
//   FP8  K tile [group g][token][32 B]: bytes 0..15 = channels 16g..16g+15,
//        bytes 16..31 = channels 64+16g..64+16g+15 (the FP8 operand order of
//        the 16x16x128 MFMA); V tile [token/4][channel/8][token%4][8 B].
//   BF16 K tile [k-step s][group g][token][16 B] = channels 32s+8g..+7;
//        V tile [token/4][channel/8][token%4][16 B].
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
    constexpr int kTileBytes = FMT == kFp8 ? 2048 : 4096;
    uint8_t* kt = p.cache + ((page * p.num_kv_heads + h) * 2) * kTileBytes;
    uint8_t* vt = kt + kTileBytes;
    if constexpr (FMT == kFp8) {
        uint32_t kw[2] = {0u, 0u}, vw[2] = {0u, 0u};
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            kw[i >> 2] |= e4m3_byte(xk[i] / p.k_scale) << (8 * (i & 3));
            vw[i >> 2] |= e4m3_byte(xv[i] / p.v_scale) << (8 * (i & 3));
        }
        const int c0 = 8 * lane16;
        const int g = (c0 & 63) >> 4;
        const int e0 = (c0 & 15) + (c0 >= 64 ? 16 : 0);
        *reinterpret_cast<uint2*>(kt + (g * kPage + off) * 32 + e0) = make_uint2(kw[0], kw[1]);
        *reinterpret_cast<uint2*>(vt + ((off >> 2) * 16 + lane16) * 32 + (off & 3) * 8) = make_uint2(vw[0], vw[1]);
    } else {
        uint32_t kw[4], vw[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const v2bf hk = {__bf16(xk[2 * i]), __bf16(xk[2 * i + 1])};
            const v2bf hv = {__bf16(xv[2 * i]), __bf16(xv[2 * i + 1])};
            kw[i] = __builtin_bit_cast(uint32_t, hk);
            vw[i] = __builtin_bit_cast(uint32_t, hv);
        }
        const int st = lane16 >> 2;
        const int g = lane16 & 3;
        *reinterpret_cast<uint4*>(kt + ((st * 4 + g) * kPage + off) * 16) = uint4{kw[0], kw[1], kw[2], kw[3]};
        *reinterpret_cast<uint4*>(vt + ((off >> 2) * 16 + lane16) * 64 + (off & 3) * 16) = uint4{vw[0], vw[1], vw[2], vw[3]};
    }
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

hipError_t launch_quantize_kv(const QuantizeParams& p, int dtype, hipStream_t stream) {
    const int64_t nvec = p.num_tokens * p.num_kv_heads;
    const int64_t blocks = (nvec + 15) / 16;
    if (blocks == 0) return hipSuccess;
    if (blocks > 0x7FFFFFFF) return hipErrorInvalidValue;
    const dim3 grid{unsigned(blocks)}, block{256u};
    if (dtype == 0) hipLaunchKernelGGL(quantize_kv_kernel<0>, grid, block, 0, stream, p);
    else if (dtype == 1) hipLaunchKernelGGL(quantize_kv_kernel<1>, grid, block, 0, stream, p);
    else hipLaunchKernelGGL(quantize_kv_kernel<2>, grid, block, 0, stream, p);
    return hipGetLastError();
}

template <int DT>
static hipError_t launch_ref(const RefWriteParams& p, const dim3& grid, hipStream_t stream) {
    if (p.kv_fmt == kFp8) hipLaunchKernelGGL((write_kv_ref_kernel<DT, kFp8>), grid, dim3(256), 0, stream, p);
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
