// uq_internal.hpp -- kernel parameter blocks and launchers shared between
// the libuq translation units (not part of the public ABI).
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace uq {

// Cache formats of the decode kernel template: the FP4 cache of this library
// and the two plain comparison caches.
// kFp4d64 / kFp4d256: the FP4 cache at head sizes 64 and 256 (kFp4 is 128).
// kFp4d64x2: head size 64 with two KV heads per block, staged and computed as
// one 128-channel head (group size at most 8, an even number of KV heads).
enum KvFmt : int32_t { kFp4 = 0, kFp8 = 1, kBf16 = 2, kTq4 = 3, kFp4d64 = 4, kFp4d256 = 5, kFp4d64x2 = 6 };

// Tables of the Ultra-TQ key codebook, built on the host from the 16 levels
// rounded to BF16: the encoder's midpoints (c_j + c_{j+1}) / 2, exact in
// fp64, and the decoder's byte lookup (lut[0..3]: high bytes of the BF16
// levels, four per dword in level order; lut[4..7]: low bytes).
struct TqTables {
    double mid[15];
    uint32_t lut[8];
};
constexpr int kNumCus = 256;     // compute units of an MI355X (8 XCDs x 32)
constexpr int kTqBlock = 2368;   // bytes per (page, kv head) of the Ultra-TQ cache
constexpr int kTqMeta = 2048;    // offset of the norms and (scale, zero) words in a block

struct QuantizeParams {
    const void* k;
    const void* v;
    int64_t num_tokens;
    int64_t token_stride;      // elements between consecutive tokens
    const int64_t* slot_mapping;
    const int32_t* page_table; // nullptr: slot_mapping holds physical slots
    int32_t max_pages_per_seq;
    int64_t num_seqs;          // rows of page_table (bound for the logical slot)
    int32_t num_kv_heads;
    int64_t num_pages;
    float c;
    int32_t rotate_v;
    uint8_t* codes;
    uint8_t* scales;
    int32_t head_dim;          // 64, 128 or 256
};

struct RefWriteParams {
    const void* k;
    const void* v;
    int64_t num_tokens;
    int64_t token_stride;
    const int64_t* slot_mapping;
    const int32_t* page_table;
    int32_t max_pages_per_seq;
    int64_t num_seqs;
    int32_t num_kv_heads;
    int64_t num_pages;
    float k_scale;             // FP8: stored = e4m3(x / k_scale)
    float v_scale;
    int32_t kv_fmt;            // kFp8, kBf16 or kTq4
    uint8_t* cache;            // [pages][Hkv][block bytes]
    TqTables tq;               // kTq4 only
};

struct DecodeParams {
    int32_t kv_fmt;            // KvFmt
    float out_scale;           // V tensor scale (FP8 cache), else 1
    const void* q;             // [B][Hq][128], dtype q_dtype
    int32_t q_dtype;           // 0 f32, 1 bf16, 2 f16, 3 fp8 (prepared)
    uint8_t* codes;            // written only by a decode step (k_new != nullptr)
    uint8_t* scales;
    // decode step: each sequence's new token, written at its last position
    const void* k_new;         // [B][Hkv][128] or nullptr
    const void* v_new;
    int32_t new_dtype;         // 0 f32, 1 bf16, 2 f16
    float c;                   // FP4 scale constant
    float k_scale;             // FP8 cache: per-tensor scales of the writer
    float v_scale;
    const int32_t* page_table;
    int32_t max_pages_per_seq;
    const int32_t* context_lens;
    int32_t max_context;
    int32_t batch;
    int32_t num_q_heads;
    int32_t num_kv_heads;
    int32_t group;             // query heads per kv head (<= 16)
    int64_t num_pages;
    float scale_log2;          // softmax_scale * log2(e)
    int32_t partition_tokens;
    int32_t num_partitions;
    float* part_acc;           // [B][Hq][NP][128]
    float* part_ml;            // [B][Hq][NP][2]  (running max in log2 units, running sum)
    void* out;                 // [B][Hq][128]
    int32_t out_dtype;         // 0 f32, 1 bf16
    int32_t rotate_v;
    int32_t head_dim;          // 64, 128 or 256 (FP4 cache; the others are 128)
    TqTables tq;               // Ultra-TQ cache only
    // cascade decode over a shared prefix (prefix_pages == nullptr: off).
    // Partial slots per (sequence, query head): the suffix_partitions of the
    // context grid, then the prefix partitions.
    const int32_t* prefix_pages;   // [prefix_tokens / 16]
    const int32_t* prefix_lens;    // [B] tokens of each sequence served by the prefix
    int32_t prefix_tokens;
    int32_t prefix_partition;      // prefix tokens per prefix block
    int32_t prefix_chunks;         // ceil(B * G / 16) column chunks per kv head
    int32_t prefix_blocks;         // Hkv * prefix_chunks * prefix partitions, after the context blocks in the grid
    int32_t suffix_partitions;
    // the rows of a cascade launch in dispatch order, written by
    // cascade_rows_kernel before the partition launch: context rows {part *
    // B + b, context length, tokens the prefix serves, 0}, longest first,
    // then prefix rows {suffix_partitions * B + j, 0, 0, 0}, then -1
    int4* cascade_rows;            // [suffix_partitions * B + prefix_blocks / Hkv]
    // grid shape of the partition launch: 0 one block per partition (its
    // waves share the partition's pages and merge through LDS); W > 1 one
    // wave per partition, a block taking W consecutive partitions of one
    // sequence and kv head and reducing them through LDS into one partial
    // slot (slot = first partition / W).  Chosen by the launchers when
    // allow_wave_parts.
    int32_t allow_wave_parts;
    int32_t wave_parts;
    // the page-gather probe's checksums, one per wave of the partition
    // launch, sink[block * W + wave] (set only by launch_gather_probe)
    uint32_t* probe_sink;
};

constexpr int kMaxErrorConstants = 256;   // constants per uq_quantize_error call

struct ErrorParams {
    const void* x;             // rows of 128 channels
    int64_t rows;
    int64_t row_stride;        // elements
    int32_t rotate;
    int32_t pow2;              // 1: UE8M0 scale 2^round(log2(c m)); 0: scale c m
    int32_t num_c;
    const float* c_values;     // [num_c]
    double* sums;              // [num_c][2]: sum of squared errors, sum of squares (accumulated)
};

hipError_t launch_quantize_kv(const QuantizeParams& p, int dtype, hipStream_t stream);
hipError_t launch_quantize_error(const ErrorParams& p, int dtype, hipStream_t stream);
hipError_t launch_write_kv_ref(const RefWriteParams& p, int dtype, hipStream_t stream);
hipError_t launch_prepare_query(const void* q, int dtype, int64_t rows, uint8_t* q8, hipStream_t stream);
hipError_t launch_decode_partials(const DecodeParams& p, hipStream_t stream);
hipError_t launch_decode_merge(const DecodeParams& p, hipStream_t stream);
hipError_t launch_decode_partials_mxpv(const DecodeParams& p, hipStream_t stream);
// measurement probes
// The FP4 partition launch for these parameters as a page-gather probe
// (its grid, page walk and copies, no arithmetic); partition_blocks: the
// blocks of that launch; probe_words: its checksum words (one per wave).
hipError_t launch_gather_probe(const DecodeParams& p, uint32_t* sink, hipStream_t stream);
int64_t partition_blocks(const DecodeParams& p);
int64_t probe_words(const DecodeParams& p);
hipError_t launch_stream_read_probe(const void* buf, int64_t n16, uint32_t* sink, int blocks, hipStream_t stream);
hipError_t launch_mfma_probe(int kind, const void* a, const void* b, const uint8_t* scale_a, const uint8_t* scale_b,
                             int n, float* d, hipStream_t stream);

// Kernel timing: the next decode partition or quantize-on-write launch of
// this host thread sets `start` and `stop` to its kernel's own start and
// end (hipExtLaunchKernel), then the pair is forgotten.
struct LaunchEvents {
    hipEvent_t start = nullptr, stop = nullptr;
};
inline thread_local LaunchEvents g_launch_events;
inline void time_next_launch(hipEvent_t start, hipEvent_t stop) { g_launch_events = LaunchEvents{start, stop}; }
template <class Kernel, class... Args>
inline void launch_kernel(Kernel kernel, const dim3& grid, const dim3& block, hipStream_t stream, Args... args) {
    const LaunchEvents ev = g_launch_events;
    if (ev.start != nullptr) {
        g_launch_events = LaunchEvents{};
        hipExtLaunchKernelGGL(kernel, grid, block, 0, stream, ev.start, ev.stop, 0, args...);
    } else {
        hipLaunchKernelGGL(kernel, grid, block, 0, stream, args...);
    }
}

}  // namespace uq
