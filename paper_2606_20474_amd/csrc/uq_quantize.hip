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

    const TokenBits<kFp4> tb = encode_token<kFp4>(xk, xv, lane16, p.c, p.rotate_v != 0, 1.0f, 1.0f);
    store_token<kFp4>(p.codes, p.scales, (page * p.num_kv_heads + h) * 2, off, lane16, tb);
}

// Writer of the plain comparison caches (FP8 E4M3 with one scale per
// tensor, or BF16); the layouts are those of place_token.
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
    const TokenBits<FMT> tb = encode_token<FMT>(xk, xv, lane16, 0.0f, false, p.k_scale, p.v_scale);
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
