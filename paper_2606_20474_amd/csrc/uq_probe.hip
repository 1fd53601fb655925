// uq_probe.hip -- measurement probes (not part of the method): the read
// bandwidth this GPU reaches on a plain stream, and the arithmetic of single
// matrix instructions on given operands.  The page-gather probe, which
// shares the decode kernel's staging code, is in uq_decode.hip.
#include "uq_device.hpp"
#include "uq_internal.hpp"

namespace uq {

// Stream read: block b of the grid reads its own contiguous share of the
// n16 16-byte words (ceil(n16 / grid) of them), 8 independent loads per
// thread in flight (every wave reads 1 KiB contiguous per load), with the
// non-temporal cache policy, XOR-folded into one checksum word per block so
// that no load is dead.  Of the stream shapes measured on 4 GiB this is
// among the fastest (7.0 TB/s against 5.6 TB/s for a grid-stride pass with
// the default policy); a share per block, rather than a grid-stride walk,
// and the streaming policy each gained about 10 %.
typedef unsigned v4u __attribute__((ext_vector_type(4)));
__global__ void __launch_bounds__(256) stream_read_kernel(const uint4* __restrict__ buf, int64_t n16,
                                                          uint32_t* __restrict__ sink) {
    constexpr int kUnroll = 8;
    const int64_t per = (n16 + gridDim.x - 1) / gridDim.x;
    const int64_t b0 = int64_t(blockIdx.x) * per;
    const int64_t b1 = b0 + per < n16 ? b0 + per : n16;
    const v4u* src = reinterpret_cast<const v4u*>(buf);
    uint32_t acc = 0u;
    int64_t i = b0 + threadIdx.x;
    for (; i + (kUnroll - 1) * 256 < b1; i += kUnroll * 256) {
        v4u w[kUnroll];
#pragma unroll
        for (int j = 0; j < kUnroll; ++j) w[j] = __builtin_nontemporal_load(src + i + j * 256);
#pragma unroll
        for (int j = 0; j < kUnroll; ++j) acc ^= w[j].x ^ w[j].y ^ w[j].z ^ w[j].w;
    }
    for (; i < b1; i += 256) {
        const v4u w = __builtin_nontemporal_load(src + i);
        acc ^= w.x ^ w.y ^ w.z ^ w.w;
    }
#pragma unroll
    for (int s = 1; s < 64; s <<= 1) acc ^= uint32_t(__shfl_xor(int(acc), s));
    __shared__ uint32_t part[4];
    if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = acc;
    __syncthreads();
    if (threadIdx.x == 0) sink[blockIdx.x] = part[0] ^ part[1] ^ part[2] ^ part[3];
}

hipError_t launch_stream_read_probe(const void* buf, int64_t n16, uint32_t* sink, int blocks, hipStream_t stream) {
    launch_kernel(stream_read_kernel, dim3(unsigned(blocks)), dim3(256), stream, static_cast<const uint4*>(buf), n16,
                  sink);
    return hipGetLastError();
}

// One wave per case: D = A x B (+ 0) by one matrix instruction, operands as
// bytes in the instruction's lane layout (32 bytes per lane; the FP4 operand
// uses the first 16), scale bytes one per lane (lane 16 j + i: row or
// column i, k-block j), D as 4 floats per lane.
//   kind 0: v_mfma_scale_f32_16x16x128_f8f6f4, A FP4 E2M1, B FP8 E4M3
//   kind 1: the same instruction, A and B FP8 E4M3
//   kind 2: v_mfma_f32_16x16x32_bf16 (8 BF16 per lane in the first 16 bytes)
//   kind 3: v_mfma_scale_f32_16x16x128_f8f6f4, A FP8 E4M3, B FP4 E2M1
template <int KIND>
__global__ void __launch_bounds__(64) mfma_probe_kernel(const uint4* __restrict__ a, const uint4* __restrict__ b,
                                                        const uint8_t* __restrict__ sa, const uint8_t* __restrict__ sb,
                                                        float4* __restrict__ d) {
    const int lane = threadIdx.x;
    const int64_t l = int64_t(blockIdx.x) * 64 + lane;
    const uint4 a0 = a[2 * l], a1 = a[2 * l + 1];
    const uint4 b0 = b[2 * l], b1 = b[2 * l + 1];
    const v4f zero = {0.f, 0.f, 0.f, 0.f};
    v4f r;
    if constexpr (KIND == 2) {
        r = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(v8bf, a0), __builtin_bit_cast(v8bf, b0), zero,
                                                    0, 0, 0);
    } else {
        const v8i av = {int(a0.x), int(a0.y), int(a0.z), int(a0.w), int(a1.x), int(a1.y), int(a1.z), int(a1.w)};
        const v8i bv = {int(b0.x), int(b0.y), int(b0.z), int(b0.w), int(b1.x), int(b1.y), int(b1.z), int(b1.w)};
        const int s_a = sa[l], s_b = sb[l];
        if constexpr (KIND == 0) r = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(av, bv, zero, 4, 0, 0, s_a, 0, s_b);
        else if constexpr (KIND == 1) r = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(av, bv, zero, 0, 0, 0, s_a, 0, s_b);
        else r = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(av, bv, zero, 0, 4, 0, s_a, 0, s_b);
    }
    d[l] = make_float4(r[0], r[1], r[2], r[3]);
}

hipError_t launch_mfma_probe(int kind, const void* a, const void* b, const uint8_t* scale_a, const uint8_t* scale_b,
                             int n, float* d, hipStream_t stream) {
    const dim3 grid{unsigned(n)}, block{64u};
    const uint4* A = static_cast<const uint4*>(a);
    const uint4* B = static_cast<const uint4*>(b);
    float4* D = reinterpret_cast<float4*>(d);
    if (kind == 0) hipLaunchKernelGGL(mfma_probe_kernel<0>, grid, block, 0, stream, A, B, scale_a, scale_b, D);
    else if (kind == 1) hipLaunchKernelGGL(mfma_probe_kernel<1>, grid, block, 0, stream, A, B, scale_a, scale_b, D);
    else if (kind == 2) hipLaunchKernelGGL(mfma_probe_kernel<2>, grid, block, 0, stream, A, B, scale_a, scale_b, D);
    else hipLaunchKernelGGL(mfma_probe_kernel<3>, grid, block, 0, stream, A, B, scale_a, scale_b, D);
    return hipGetLastError();
}

}  // namespace uq
