// uq_api.hip -- the C ABI of libuq (declared in include/uq.h): argument
// validation on the host, launch configuration, workspace sizing.
#include <atomic>
#include <cstring>
#include <math.h>
#include <mutex>
#include <stdint.h>

#include "uq.h"
#include "uq_internal.hpp"

namespace {

constexpr int kHeadDim = 128;
constexpr int kPageSize = 16;
constexpr int kGroupSize = 32;
constexpr int kMaxGroup = 16;

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

uq_status check_desc(const uq_cache_desc* d) {
    if (d == nullptr) return UQ_ERR_INVALID_ARGUMENT;
    if (d->num_kv_heads < 1 || d->num_pages < 1) return UQ_ERR_INVALID_ARGUMENT;
    if (!(isfinite(d->c) && d->c > 0.0f)) return UQ_ERR_INVALID_ARGUMENT;
    if ((d->head_dim != 64 && d->head_dim != 128 && d->head_dim != 256) || d->page_size != kPageSize ||
        d->group_size != kGroupSize)
        return UQ_ERR_UNSUPPORTED;
    return UQ_OK;
}

// The calls that exist for head size 128 only (the decode step, cascade
// decode, the FP8-query form and uq_prepare_query).
uq_status require_128(const uq_cache_desc* d) { return d->head_dim == kHeadDim ? UQ_OK : UQ_ERR_UNSUPPORTED; }

uq_status from_hip(hipError_t e) { return e == hipSuccess ? UQ_OK : UQ_ERR_HIP; }

// Head size 64 runs two KV heads per block when the group size is at most 8
// and the KV heads pair up: then the grid has one block per pair.
bool paired_heads(const uq_cache_desc* desc, int32_t num_q_heads) {
    return desc->head_dim == 64 && desc->num_kv_heads % 2 == 0 && num_q_heads <= 8 * desc->num_kv_heads;
}
int32_t block_heads(const uq_cache_desc* desc, int32_t num_q_heads) {
    return paired_heads(desc, num_q_heads) ? desc->num_kv_heads / 2 : desc->num_kv_heads;
}

int32_t pick_partition(int32_t batch, int32_t num_kv_heads, int32_t max_context) {
    // The longest partition (fewest partials to merge, fewest per-block
    // prologues) that still gives every one of the 256 CUs at least two
    // blocks; between 1024 and 16384 tokens.
    const int64_t heads = int64_t(batch) * num_kv_heads;
    int32_t part = 16384;
    while (part > 1024 && heads * ((int64_t(max_context) + part - 1) / part) < 2 * uq::kNumCus) part /= 2;
    return part;
}

uq_status check_decode_common(const uq_cache_desc* desc, int32_t batch, int32_t num_q_heads, int32_t max_context,
                              int32_t partition_tokens) {
    uq_status s = check_desc(desc);
    if (s != UQ_OK) return s;
    if (batch < 1 || num_q_heads < 1 || max_context < 0 || partition_tokens < 0) return UQ_ERR_INVALID_ARGUMENT;
    if (num_q_heads % desc->num_kv_heads != 0) return UQ_ERR_INVALID_ARGUMENT;
    if (partition_tokens % 16 != 0) return UQ_ERR_INVALID_ARGUMENT;   // partitions are whole pages
    if (num_q_heads / desc->num_kv_heads > kMaxGroup) return UQ_ERR_UNSUPPORTED;
    if (batch > 65535 || desc->num_kv_heads > 65535) return UQ_ERR_UNSUPPORTED;
    return UQ_OK;
}

size_t align16(size_t x) { return (x + 15) & ~size_t(15); }

int64_t num_partitions(int32_t max_context, int32_t part) {
    return max_context > 0 ? (int64_t(max_context) + part - 1) / part : 1;
}

// Workspace of a decode call: the partial rows (accumulators, then the
// (max, sum) pairs); a cascade call (extra_slots > 0: its prefix
// partitions) adds its row list, 16 bytes per context row (partition,
// sequence) and per prefix row (column chunk, prefix partition).
size_t workspace_for(int32_t batch, int32_t num_q_heads, int32_t num_kv_heads, int32_t max_context, int32_t part,
                     int64_t extra_slots = 0, int32_t head_dim = kHeadDim) {
    const int64_t np_ctx = num_partitions(max_context, part);
    const size_t rows = align16(size_t(batch) * size_t(num_q_heads) * size_t(np_ctx + extra_slots) *
                                size_t(head_dim + 2) * sizeof(float));
    if (extra_slots <= 0) return rows;
    const int64_t chunks = (int64_t(batch) * (num_q_heads / num_kv_heads) + 15) / 16;
    return rows + size_t(np_ctx * batch + chunks * extra_slots) * 16;
}

// Fill the parameter block of the decode launches.  Workspace: the partial
// accumulators, then the (max, sum) pairs, then (cascade) the row list.
uq_status make_decode_params(const uq_cache_desc* desc, const void* q, uq_dtype q_dtype, int32_t batch,
                             int32_t num_q_heads, const uint8_t* kv_codes, const uint8_t* kv_scales,
                             const int32_t* page_table, int32_t max_pages_per_seq, const int32_t* context_lens,
                             int32_t max_context, float softmax_scale, int32_t partition_tokens, void* workspace,
                             size_t workspace_bytes, void* out, uq_dtype out_dtype, uq::DecodeParams& p,
                             int64_t extra_slots = 0) {
    const int32_t part = partition_tokens == 0 ? pick_partition(batch, block_heads(desc, num_q_heads), max_context)
                                               : partition_tokens;
    const size_t need =
        workspace_for(batch, num_q_heads, desc->num_kv_heads, max_context, part, extra_slots, desc->head_dim);
    if (workspace == nullptr) return UQ_ERR_INVALID_ARGUMENT;
    if (workspace_bytes < need) return UQ_ERR_WORKSPACE_TOO_SMALL;
    if (!aligned16(workspace)) return UQ_ERR_INVALID_ARGUMENT;
    const int64_t np_ctx = num_partitions(max_context, part);
    const int64_t np = np_ctx + extra_slots;
    // one linear grid of partitions x kv heads x sequences
    if (np * desc->num_kv_heads * batch > 0x7FFFFFFF) return UQ_ERR_UNSUPPORTED;
    p.q = q;
    p.q_dtype = int32_t(q_dtype);
    p.codes = const_cast<uint8_t*>(kv_codes);     // written only by the decode-step calls
    p.scales = const_cast<uint8_t*>(kv_scales);
    p.k_new = nullptr;
    p.v_new = nullptr;
    p.new_dtype = 0;
    p.c = desc->c;
    p.k_scale = 1.0f;
    p.v_scale = 1.0f;
    p.page_table = page_table;
    p.max_pages_per_seq = max_pages_per_seq;
    p.context_lens = context_lens;
    p.max_context = max_context;
    p.batch = batch;
    p.num_q_heads = num_q_heads;
    p.num_kv_heads = desc->num_kv_heads;
    p.group = num_q_heads / desc->num_kv_heads;
    p.num_pages = desc->num_pages;
    p.scale_log2 = float(double(softmax_scale) * 1.4426950408889634);
    p.partition_tokens = part;
    p.num_partitions = int32_t(np);
    char* ws = static_cast<char*>(workspace);
    const size_t acc_bytes = size_t(batch) * num_q_heads * size_t(np) * size_t(desc->head_dim) * sizeof(float);
    const size_t ml_bytes = size_t(batch) * num_q_heads * size_t(np) * 2 * sizeof(float);
    p.part_acc = reinterpret_cast<float*>(ws);
    p.part_ml = reinterpret_cast<float*>(ws + acc_bytes);
    p.cascade_rows = extra_slots > 0 ? reinterpret_cast<int4*>(ws + align16(acc_bytes + ml_bytes)) : nullptr;
    p.out = out;
    p.out_dtype = out_dtype == UQ_F32 ? 0 : 1;
    p.rotate_v = desc->rotate_v != 0;
    p.head_dim = desc->head_dim;
    p.kv_fmt = desc->head_dim == 64 ? (paired_heads(desc, num_q_heads) ? uq::kFp4d64x2 : uq::kFp4d64)
               : desc->head_dim == 256 ? uq::kFp4d256 : uq::kFp4;
    p.out_scale = 1.0f;
    p.prefix_pages = nullptr;
    p.prefix_lens = nullptr;
    p.prefix_tokens = 0;
    p.prefix_partition = 0;
    p.prefix_chunks = 0;
    p.prefix_blocks = 0;
    p.suffix_partitions = int32_t(np_ctx);
    p.allow_wave_parts = 1;
    p.wave_parts = 0;
    p.probe_sink = nullptr;
    return UQ_OK;
}

// Cascade decode: the prefix partition (tokens per prefix block; the
// default gives about 1024 prefix blocks, at least 32 tokens each) and the
// number of prefix partial slots per (sequence, query head).
int32_t prefix_partition(const uq_shared_prefix* pre, int32_t num_kv_heads, int32_t batch, int32_t group) {
    if (pre->partition_tokens > 0) return pre->partition_tokens;
    const int64_t chunks = (int64_t(batch) * group + 15) / 16;
    int64_t parts = (1024 + num_kv_heads * chunks - 1) / (num_kv_heads * chunks);
    parts = parts < 1 ? 1 : parts;
    int64_t pp = (int64_t(pre->num_tokens) + parts - 1) / parts;
    pp = (pp + 31) & ~int64_t(31);
    return int32_t(pp < 32 ? 32 : pp);
}

uq_status check_prefix(const uq_shared_prefix* pre) {
    if (pre == nullptr || pre->pages == nullptr || pre->lens == nullptr) return UQ_ERR_INVALID_ARGUMENT;
    if (pre->num_tokens < 16 || pre->num_tokens % 16 != 0) return UQ_ERR_INVALID_ARGUMENT;
    if (pre->partition_tokens < 0 || pre->partition_tokens % 32 != 0) return UQ_ERR_INVALID_ARGUMENT;
    return UQ_OK;
}

int64_t prefix_slots(const uq_shared_prefix* pre, int32_t num_kv_heads, int32_t batch, int32_t group) {
    const int32_t pp = prefix_partition(pre, num_kv_heads, batch, group);
    return (int64_t(pre->num_tokens) + pp - 1) / pp;
}

// Fill the cascade fields of a parameter block made with the prefix slots.
uq_status apply_prefix(const uq_shared_prefix* pre, uq::DecodeParams& p) {
    p.prefix_pages = pre->pages;
    p.prefix_lens = pre->lens;
    p.prefix_tokens = pre->num_tokens;
    p.prefix_partition = prefix_partition(pre, p.num_kv_heads, p.batch, p.group);
    p.prefix_chunks = int32_t((int64_t(p.batch) * p.group + 15) / 16);
    const int64_t blocks = int64_t(p.num_kv_heads) * p.prefix_chunks *
                           ((int64_t(pre->num_tokens) + p.prefix_partition - 1) / p.prefix_partition);
    if (blocks + int64_t(p.suffix_partitions) * p.num_kv_heads * p.batch > 0x7FFFFFFF) return UQ_ERR_UNSUPPORTED;
    p.prefix_blocks = int32_t(blocks);
    return UQ_OK;
}

uq_status check_split_args(const uq_cache_desc* desc, const void* q, uq_dtype q_dtype, int32_t batch,
                           int32_t num_q_heads, const uint8_t* kv_codes, const uint8_t* kv_scales,
                           const int32_t* page_table, int32_t max_pages_per_seq, const int32_t* context_lens,
                           int32_t max_context, float softmax_scale, int32_t partition_tokens) {
    uq_status s = check_decode_common(desc, batch, num_q_heads, max_context, partition_tokens);
    if (s != UQ_OK) return s;
    if (q == nullptr || kv_codes == nullptr || kv_scales == nullptr || page_table == nullptr || context_lens == nullptr)
        return UQ_ERR_INVALID_ARGUMENT;
    if (q_dtype != UQ_F32 && q_dtype != UQ_BF16 && q_dtype != UQ_F16 && q_dtype != UQ_FP8_E4M3)
        return UQ_ERR_UNSUPPORTED;
    if (q_dtype == UQ_FP8_E4M3 && desc->head_dim != kHeadDim) return UQ_ERR_UNSUPPORTED;
    if (max_pages_per_seq < 1) return UQ_ERR_INVALID_ARGUMENT;
    if (int64_t(max_context) > int64_t(max_pages_per_seq) * kPageSize) return UQ_ERR_INVALID_ARGUMENT;
    if (!(isfinite(softmax_scale) && softmax_scale > 0.0f)) return UQ_ERR_INVALID_ARGUMENT;
    if (!aligned16(q) || !aligned16(kv_codes) || !aligned16(kv_scales)) return UQ_ERR_INVALID_ARGUMENT;
    return UQ_OK;
}

// Comparison caches: the descriptor check and the FP4 descriptor with the
// same geometry (the decode set-up above is shared; no rotation).
// fp32 -> nearest BF16 (ties to even) of a finite value, as fp32.
float bf16_nearest(float x) {
    uint32_t u;
    memcpy(&u, &x, 4);
    u += 0x7FFFu + ((u >> 16) & 1u);
    u &= 0xFFFF0000u;
    float r;
    memcpy(&r, &u, 4);
    return r;
}

// The Ultra-TQ codebook tables: levels rounded to BF16 (finite, strictly
// ascending), the encoder's midpoints (c_j + c_{j+1}) / 2 in fp64 and the
// decoder's byte tables.  False for an unusable codebook.
bool tq_tables(const float* cb, uq::TqTables& t) {
    if (cb == nullptr) return false;
    float lv[16];
    for (int j = 0; j < 16; ++j) {
        if (!isfinite(cb[j])) return false;
        lv[j] = bf16_nearest(cb[j]);
        if (!isfinite(lv[j])) return false;
    }
    for (int j = 0; j < 15; ++j)
        if (!(lv[j] < lv[j + 1])) return false;
    for (int j = 0; j < 15; ++j) {
        // the midpoint must be exact in fp64 (adjacent levels within 2^44 of
        // each other): the encoder decides x > m_j n by the sign of an fma
        const double a = lv[j], b = lv[j + 1], s = a + b;
        if (s - a != b || s - b != a) return false;
        t.mid[j] = s * 0.5;
    }
    for (int w = 0; w < 4; ++w) {
        uint32_t hi = 0, lo = 0;
        for (int b = 0; b < 4; ++b) {
            uint32_t u;
            memcpy(&u, &lv[4 * w + b], 4);
            hi |= ((u >> 24) & 0xFFu) << (8 * b);
            lo |= ((u >> 16) & 0xFFu) << (8 * b);
        }
        t.lut[w] = hi;
        t.lut[4 + w] = lo;
    }
    return true;
}

uq_status check_ref_desc(const uq_ref_cache_desc* d) {
    if (d == nullptr) return UQ_ERR_INVALID_ARGUMENT;
    if (d->num_kv_heads < 1 || d->num_pages < 1) return UQ_ERR_INVALID_ARGUMENT;
    if (d->format != UQ_REF_FP8_E4M3 && d->format != UQ_REF_BF16 && d->format != UQ_REF_TQ4)
        return UQ_ERR_UNSUPPORTED;
    if (d->head_dim != kHeadDim || d->page_size != kPageSize) return UQ_ERR_UNSUPPORTED;
    if (d->format == UQ_REF_FP8_E4M3 &&
        !(isfinite(d->k_scale) && d->k_scale > 0.0f && isfinite(d->v_scale) && d->v_scale > 0.0f))
        return UQ_ERR_INVALID_ARGUMENT;
    if (d->format == UQ_REF_TQ4) {
        uq::TqTables t;
        if (!tq_tables(d->codebook, t)) return UQ_ERR_INVALID_ARGUMENT;
    }
    return UQ_OK;
}

uq_cache_desc geometry_of(const uq_ref_cache_desc* d) {
    uq_cache_desc g;
    g.num_kv_heads = d->num_kv_heads;
    g.head_dim = kHeadDim;
    g.page_size = kPageSize;
    g.group_size = kGroupSize;
    g.num_pages = d->num_pages;
    g.c = 0.156f;
    g.rotate_v = 0;
    return g;
}

int32_t ref_fmt(const uq_ref_cache_desc* d) {
    return d->format == UQ_REF_FP8_E4M3 ? uq::kFp8 : d->format == UQ_REF_TQ4 ? uq::kTq4 : uq::kBf16;
}

// Half of the bytes of one (page, kv head): the K tile, or for TQ4 half of
// the block that holds both.
int64_t ref_tile_bytes(const uq_ref_cache_desc* d) {
    return d->format == UQ_REF_FP8_E4M3 ? 2048 : d->format == UQ_REF_TQ4 ? uq::kTqBlock / 2 : 4096;
}

}  // namespace

// The partials of uq_decode_attention_noalloc: one array per GPU, placed by
// the module loader, never allocated by a call.  In host code `scratch` is a
// host-side stand-in for the symbol, not a device address: only the address
// hipGetSymbolAddress returns for the current device is ever passed to a
// kernel.
static __device__ __align__(256) uint8_t scratch[UQ_NOALLOC_SCRATCH_BYTES];

namespace {
constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch_ptr[kMaxDevices];
std::mutex g_scratch_mutex;

// The array's address on the current device, looked up once per device.
uq_status scratch_of_current_device(void** ptr) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0) return UQ_ERR_HIP;
    if (dev >= kMaxDevices) return UQ_ERR_UNSUPPORTED;
    void* p = g_scratch_ptr[dev].load(std::memory_order_acquire);
    if (p == nullptr) {
        std::lock_guard<std::mutex> lock(g_scratch_mutex);
        p = g_scratch_ptr[dev].load(std::memory_order_relaxed);
        if (p == nullptr) {
            if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) return UQ_ERR_HIP;
            g_scratch_ptr[dev].store(p, std::memory_order_release);
        }
    }
    *ptr = p;
    return UQ_OK;
}
}  // namespace

extern "C" {

const char* uq_status_string(uq_status s) {
    switch (s) {
        case UQ_OK: return "UQ_OK";
        case UQ_ERR_INVALID_ARGUMENT: return "UQ_ERR_INVALID_ARGUMENT";
        case UQ_ERR_UNSUPPORTED: return "UQ_ERR_UNSUPPORTED";
        case UQ_ERR_WORKSPACE_TOO_SMALL: return "UQ_ERR_WORKSPACE_TOO_SMALL";
        case UQ_ERR_HIP: return "UQ_ERR_HIP";
    }
    return "UQ_ERR_UNKNOWN";
}

int32_t uq_version(void) { return 100; }

uq_status uq_quantize_kv(const uq_cache_desc* desc, const void* k, const void* v, uq_dtype in_dtype,
                         int64_t num_tokens, int64_t token_stride, const int32_t* page_table, int32_t num_seqs,
                         int32_t max_pages_per_seq, const int64_t* slot_mapping, uint8_t* kv_codes,
                         uint8_t* kv_scales, void* stream) {
    uq_status s = check_desc(desc);
    if (s != UQ_OK) return s;
    if (in_dtype != UQ_F32 && in_dtype != UQ_BF16 && in_dtype != UQ_F16) return UQ_ERR_UNSUPPORTED;
    if (num_tokens < 0) return UQ_ERR_INVALID_ARGUMENT;
    if (k == nullptr || v == nullptr || slot_mapping == nullptr || kv_codes == nullptr || kv_scales == nullptr)
        return UQ_ERR_INVALID_ARGUMENT;
    if (token_stride < int64_t(desc->num_kv_heads) * desc->head_dim) return UQ_ERR_INVALID_ARGUMENT;
    const int64_t vec_elems = in_dtype == UQ_F32 ? 4 : 8;   // one 16-byte load
    if (token_stride % vec_elems != 0 || !aligned16(k) || !aligned16(v)) return UQ_ERR_INVALID_ARGUMENT;
    if (!aligned16(kv_codes) || !aligned16(kv_scales)) return UQ_ERR_INVALID_ARGUMENT;
    if (page_table != nullptr && (max_pages_per_seq < 1 || num_seqs < 1)) return UQ_ERR_INVALID_ARGUMENT;
    if (num_tokens == 0) return UQ_OK;
    uq::QuantizeParams p;
    p.k = k;
    p.v = v;
    p.num_tokens = num_tokens;
    p.token_stride = token_stride;
    p.slot_mapping = slot_mapping;
    p.page_table = page_table;
    p.max_pages_per_seq = max_pages_per_seq;
    p.num_seqs = page_table != nullptr ? num_seqs : 0;
    p.num_kv_heads = desc->num_kv_heads;
    p.num_pages = desc->num_pages;
    p.c = desc->c;
    p.rotate_v = desc->rotate_v != 0;
    p.codes = kv_codes;
    p.scales = kv_scales;
    p.head_dim = desc->head_dim;
    return from_hip(uq::launch_quantize_kv(p, int(in_dtype), static_cast<hipStream_t>(stream)));
}

uq_status uq_prepare_query(const uq_cache_desc* desc, const void* q, uq_dtype q_dtype, int64_t rows, uint8_t* q_fp8,
                           void* stream) {
    uq_status s = check_desc(desc);
    if (s != UQ_OK) return s;
    s = require_128(desc);
    if (s != UQ_OK) return s;
    if (q_dtype != UQ_F32 && q_dtype != UQ_BF16 && q_dtype != UQ_F16) return UQ_ERR_UNSUPPORTED;
    if (rows < 0 || q == nullptr || q_fp8 == nullptr) return UQ_ERR_INVALID_ARGUMENT;
    if (!aligned16(q) || (reinterpret_cast<uintptr_t>(q_fp8) & 7u) != 0) return UQ_ERR_INVALID_ARGUMENT;
    if (rows == 0) return UQ_OK;
    return from_hip(uq::launch_prepare_query(q, int(q_dtype), rows, q_fp8, static_cast<hipStream_t>(stream)));
}

uq_status uq_quantize_error(const void* x, uq_dtype dtype, int64_t rows, int64_t row_stride, int32_t rotate,
                            int32_t pow2_scale, int32_t num_c, const float* c_values, double* sums, void* stream) {
    if (dtype != UQ_F32 && dtype != UQ_BF16 && dtype != UQ_F16) return UQ_ERR_UNSUPPORTED;
    if (rows < 0 || num_c < 0 || num_c > uq::kMaxErrorConstants || row_stride < kHeadDim)
        return UQ_ERR_INVALID_ARGUMENT;
    if ((x == nullptr && rows > 0) || c_values == nullptr || sums == nullptr) return UQ_ERR_INVALID_ARGUMENT;
    if (rows == 0 || num_c == 0) return UQ_OK;
    const int64_t vec_elems = dtype == UQ_F32 ? 4 : 8;
    if (row_stride % vec_elems != 0 || !aligned16(x)) return UQ_ERR_INVALID_ARGUMENT;
    if (rows == 0 || num_c == 0) return UQ_OK;
    uq::ErrorParams p;
    p.x = x;
    p.rows = rows;
    p.row_stride = row_stride;
    p.rotate = rotate != 0;
    p.pow2 = pow2_scale != 0;
    p.num_c = num_c;
    p.c_values = c_values;
    p.sums = sums;
    return from_hip(uq::launch_quantize_error(p, int(dtype), static_cast<hipStream_t>(stream)));
}

int32_t uq_default_partition(const uq_cache_desc* desc, int32_t batch, int32_t num_q_heads, int32_t max_context) {
    if (check_decode_common(desc, batch, num_q_heads, max_context, 0) != UQ_OK) return 0;
    return pick_partition(batch, block_heads(desc, num_q_heads), max_context);
}

size_t uq_decode_workspace_bytes(const uq_cache_desc* desc, int32_t batch, int32_t num_q_heads, int32_t max_context,
                                 int32_t partition_tokens) {
    if (check_decode_common(desc, batch, num_q_heads, max_context, partition_tokens) != UQ_OK) return 0;
    const int32_t part = partition_tokens == 0 ? pick_partition(batch, block_heads(desc, num_q_heads), max_context)
                                               : partition_tokens;
    return workspace_for(batch, num_q_heads, desc->num_kv_heads, max_context, part, 0, desc->head_dim);
}

// Shared set-up of the decode entry points: validation and the parameter block.
static uq_status decode_setup(const uq_cache_desc* desc, const void* q, uq_dtype q_dtype, int32_t batch,
                              int32_t num_q_heads, const uint8_t* kv_codes, const uint8_t* kv_scales,
                              const int32_t* page_table, int32_t max_pages_per_seq, const int32_t* context_lens,
                              int32_t max_context, float softmax_scale, int32_t partition_tokens, void* workspace,
                              size_t workspace_bytes, void* out, uq_dtype out_dtype, uq::DecodeParams& p,
                              int64_t extra_slots = 0) {
    uq_status s = check_split_args(desc, q, q_dtype, batch, num_q_heads, kv_codes, kv_scales, page_table,
                                   max_pages_per_seq, context_lens, max_context, softmax_scale, partition_tokens);
    if (s != UQ_OK) return s;
    if (out == nullptr) return UQ_ERR_INVALID_ARGUMENT;
    if (out_dtype != UQ_F32 && out_dtype != UQ_BF16) return UQ_ERR_UNSUPPORTED;
    if (!aligned16(out)) return UQ_ERR_INVALID_ARGUMENT;
    return make_decode_params(desc, q, q_dtype, batch, num_q_heads, kv_codes, kv_scales, page_table, max_pages_per_seq,
                              context_lens, max_context, softmax_scale, partition_tokens, workspace, workspace_bytes,
                              out, out_dtype, p, extra_slots);
}

// The new-token arguments of the decode-step calls (head size 128).
static uq_status step_args(const void* k_new, const void* v_new, uq_dtype new_dtype, uq::DecodeParams& p) {
    if (p.head_dim != kHeadDim) return UQ_ERR_UNSUPPORTED;
    if (k_new == nullptr || v_new == nullptr) return UQ_ERR_INVALID_ARGUMENT;
    if (new_dtype != UQ_F32 && new_dtype != UQ_BF16 && new_dtype != UQ_F16) return UQ_ERR_UNSUPPORTED;
    if (!aligned16(k_new) || !aligned16(v_new)) return UQ_ERR_INVALID_ARGUMENT;
    p.k_new = k_new;
    p.v_new = v_new;
    p.new_dtype = int32_t(new_dtype);
    return UQ_OK;
}

uq_status uq_decode_attention(const uq_cache_desc* desc, const void* q, uq_dtype q_dtype, int32_t batch,
                              int32_t num_q_heads, const uint8_t* kv_codes, const uint8_t* kv_scales,
                              const int32_t* page_table, int32_t max_pages_per_seq, const int32_t* context_lens,
                              int32_t max_context, float softmax_scale, int32_t partition_tokens, void* workspace,
                              size_t workspace_bytes, void* out, uq_dtype out_dtype, void* stream) {
    uq::DecodeParams p;
    uq_status s = decode_setup(desc, q, q_dtype, batch, num_q_heads, kv_codes, kv_scales, page_table,
                               max_pages_per_seq, context_lens, max_context, softmax_scale, partition_tokens, workspace,
                               workspace_bytes, out, out_dtype, p);
    if (s != UQ_OK) return s;
    s = from_hip(uq::launch_decode_partials(p, static_cast<hipStream_t>(stream)));
    if (s != UQ_OK) return s;
    return from_hip(uq::launch_decode_merge(p, static_cast<hipStream_t>(stream)));
}

uq_status uq_decode_attention_scaled_pv(const uq_cache_desc* desc, const void* q, uq_dtype q_dtype, int32_t batch,
                                        int32_t num_q_heads, const uint8_t* kv_codes, const uint8_t* kv_scales,
                                        const int32_t* page_table, int32_t max_pages_per_seq,
                                        const int32_t* context_lens, int32_t max_context, float softmax_scale,
                                        int32_t partition_tokens, void* workspace, size_t workspace_bytes, void* out,
                                        uq_dtype out_dtype, void* stream) {
    uq::DecodeParams p;
    uq_status s = decode_setup(desc, q, q_dtype, batch, num_q_heads, kv_codes, kv_scales, page_table,
                               max_pages_per_seq, context_lens, max_context, softmax_scale, partition_tokens, workspace,
                               workspace_bytes, out, out_dtype, p);
    if (s != UQ_OK) return s;
    if (desc->head_dim != kHeadDim) return UQ_ERR_UNSUPPORTED;
    if (p.partition_tokens % 32 != 0) return UQ_ERR_INVALID_ARGUMENT;   // whole page pairs only
    p.allow_wave_parts = 0;   // the prototype's grid is one block per partition
    s = from_hip(uq::launch_decode_partials_mxpv(p, static_cast<hipStream_t>(stream)));
    if (s != UQ_OK) return s;
    return from_hip(uq::launch_decode_merge(p, static_cast<hipStream_t>(stream)));
}

uq_status uq_decode_partials(const uq_cache_desc* desc, const void* q, uq_dtype q_dtype, int32_t batch,
                             int32_t num_q_heads, const uint8_t* kv_codes, const uint8_t* kv_scales,
                             const int32_t* page_table, int32_t max_pages_per_seq, const int32_t* context_lens,
                             int32_t max_context, float softmax_scale, int32_t partition_tokens, void* workspace,
                             size_t workspace_bytes, void* out, uq_dtype out_dtype, void* stream) {
    uq::DecodeParams p;
    uq_status s = decode_setup(desc, q, q_dtype, batch, num_q_heads, kv_codes, kv_scales, page_table,
                               max_pages_per_seq, context_lens, max_context, softmax_scale, partition_tokens, workspace,
                               workspace_bytes, out, out_dtype, p);
    if (s != UQ_OK) return s;
    return from_hip(uq::launch_decode_partials(p, static_cast<hipStream_t>(stream)));
}

uq_status uq_decode_step(const uq_cache_desc* desc, const void* q, uq_dtype q_dtype, const void* k_new,
                         const void* v_new, uq_dtype new_dtype, int32_t batch, int32_t num_q_heads,
                         uint8_t* kv_codes, uint8_t* kv_scales, const int32_t* page_table, int32_t max_pages_per_seq,
                         const int32_t* context_lens, int32_t max_context, float softmax_scale,
                         int32_t partition_tokens, void* workspace, size_t workspace_bytes, void* out,
                         uq_dtype out_dtype, void* stream) {
    uq::DecodeParams p;
    uq_status s = decode_setup(desc, q, q_dtype, batch, num_q_heads, kv_codes, kv_scales, page_table,
                               max_pages_per_seq, context_lens, max_context, softmax_scale, partition_tokens, workspace,
                               workspace_bytes, out, out_dtype, p);
    if (s != UQ_OK) return s;
    s = step_args(k_new, v_new, new_dtype, p);
    if (s != UQ_OK) return s;
    s = from_hip(uq::launch_decode_partials(p, static_cast<hipStream_t>(stream)));
    if (s != UQ_OK) return s;
    return from_hip(uq::launch_decode_merge(p, static_cast<hipStream_t>(stream)));
}

uq_status uq_decode_step_partials(const uq_cache_desc* desc, const void* q, uq_dtype q_dtype, const void* k_new,
                                  const void* v_new, uq_dtype new_dtype, int32_t batch, int32_t num_q_heads,
                                  uint8_t* kv_codes, uint8_t* kv_scales, const int32_t* page_table,
                                  int32_t max_pages_per_seq, const int32_t* context_lens, int32_t max_context,
                                  float softmax_scale, int32_t partition_tokens, void* workspace,
                                  size_t workspace_bytes, void* out, uq_dtype out_dtype, void* stream) {
    uq::DecodeParams p;
    uq_status s = decode_setup(desc, q, q_dtype, batch, num_q_heads, kv_codes, kv_scales, page_table,
                               max_pages_per_seq, context_lens, max_context, softmax_scale, partition_tokens, workspace,
                               workspace_bytes, out, out_dtype, p);
    if (s != UQ_OK) return s;
    s = step_args(k_new, v_new, new_dtype, p);
    if (s != UQ_OK) return s;
    return from_hip(uq::launch_decode_partials(p, static_cast<hipStream_t>(stream)));
}

uq_status uq_decode_merge(const uq_cache_desc* desc, int32_t batch, int32_t num_q_heads, const int32_t* context_lens,
                          int32_t max_context, int32_t partition_tokens, const void* workspace, size_t workspace_bytes,
                          void* out, uq_dtype out_dtype, void* stream) {
    uq_status s = check_decode_common(desc, batch, num_q_heads, max_context, partition_tokens);
    if (s != UQ_OK) return s;
    if (context_lens == nullptr || out == nullptr) return UQ_ERR_INVALID_ARGUMENT;
    if (out_dtype != UQ_F32 && out_dtype != UQ_BF16) return UQ_ERR_UNSUPPORTED;
    if (!aligned16(out)) return UQ_ERR_INVALID_ARGUMENT;
    uq::DecodeParams p;
    s = make_decode_params(desc, nullptr, UQ_F32, batch, num_q_heads, nullptr, nullptr, nullptr, 1, context_lens,
                           max_context, 1.0f, partition_tokens, const_cast<void*>(workspace), workspace_bytes, out,
                           out_dtype, p);
    if (s != UQ_OK) return s;
    return from_hip(uq::launch_decode_merge(p, static_cast<hipStream_t>(stream)));
}

size_t uq_ref_cache_bytes(const uq_ref_cache_desc* desc) {
    if (check_ref_desc(desc) != UQ_OK) return 0;
    return size_t(desc->num_pages) * size_t(desc->num_kv_heads) * 2 * size_t(ref_tile_bytes(desc));
}

uq_status uq_ref_write_kv(const uq_ref_cache_desc* desc, const void* k, const void* v, uq_dtype in_dtype,
                          int64_t num_tokens, int64_t token_stride, const int32_t* page_table, int32_t num_seqs,
                          int32_t max_pages_per_seq, const int64_t* slot_mapping, uint8_t* cache, void* stream) {
    uq_status s = check_ref_desc(desc);
    if (s != UQ_OK) return s;
    if (in_dtype != UQ_F32 && in_dtype != UQ_BF16 && in_dtype != UQ_F16) return UQ_ERR_UNSUPPORTED;
    if (num_tokens < 0) return UQ_ERR_INVALID_ARGUMENT;
    if (k == nullptr || v == nullptr || slot_mapping == nullptr || cache == nullptr) return UQ_ERR_INVALID_ARGUMENT;
    if (token_stride < int64_t(desc->num_kv_heads) * kHeadDim) return UQ_ERR_INVALID_ARGUMENT;
    const int64_t vec_elems = in_dtype == UQ_F32 ? 4 : 8;
    if (token_stride % vec_elems != 0 || !aligned16(k) || !aligned16(v) || !aligned16(cache))
        return UQ_ERR_INVALID_ARGUMENT;
    if (page_table != nullptr && (max_pages_per_seq < 1 || num_seqs < 1)) return UQ_ERR_INVALID_ARGUMENT;
    if (num_tokens == 0) return UQ_OK;
    uq::RefWriteParams p;
    p.k = k;
    p.v = v;
    p.num_tokens = num_tokens;
    p.token_stride = token_stride;
    p.slot_mapping = slot_mapping;
    p.page_table = page_table;
    p.max_pages_per_seq = max_pages_per_seq;
    p.num_seqs = page_table != nullptr ? num_seqs : 0;
    p.num_kv_heads = desc->num_kv_heads;
    p.num_pages = desc->num_pages;
    p.k_scale = desc->format == UQ_REF_FP8_E4M3 ? desc->k_scale : 1.0f;
    p.v_scale = desc->format == UQ_REF_FP8_E4M3 ? desc->v_scale : 1.0f;
    p.kv_fmt = ref_fmt(desc);
    p.cache = cache;
    if (desc->format == UQ_REF_TQ4) tq_tables(desc->codebook, p.tq);
    return from_hip(uq::launch_write_kv_ref(p, int(in_dtype), static_cast<hipStream_t>(stream)));
}

size_t uq_ref_decode_workspace_bytes(const uq_ref_cache_desc* desc, int32_t batch, int32_t num_q_heads,
                                     int32_t max_context, int32_t partition_tokens) {
    if (check_ref_desc(desc) != UQ_OK) return 0;
    const uq_cache_desc g = geometry_of(desc);
    return uq_decode_workspace_bytes(&g, batch, num_q_heads, max_context, partition_tokens);
}

// Shared set-up of the comparison-cache decode calls: the FP4 set-up on the
// same geometry, then the format, the K scale folded into the exponent
// scale and the V scale applied to the output.
static uq_status ref_decode_setup(const uq_ref_cache_desc* desc, const void* q, uq_dtype q_dtype, int32_t batch,
                                  int32_t num_q_heads, const uint8_t* cache, const int32_t* page_table,
                                  int32_t max_pages_per_seq, const int32_t* context_lens, int32_t max_context,
                                  float softmax_scale, int32_t partition_tokens, void* workspace,
                                  size_t workspace_bytes, void* out, uq_dtype out_dtype, uq::DecodeParams& p,
                                  int64_t extra_slots = 0) {
    uq_status s = check_ref_desc(desc);
    if (s != UQ_OK) return s;
    if (q_dtype != UQ_F32 && q_dtype != UQ_BF16 && q_dtype != UQ_F16) return UQ_ERR_UNSUPPORTED;
    const uq_cache_desc g = geometry_of(desc);
    s = decode_setup(&g, q, q_dtype, batch, num_q_heads, cache, cache, page_table, max_pages_per_seq, context_lens,
                     max_context, softmax_scale, partition_tokens, workspace, workspace_bytes, out, out_dtype, p,
                     extra_slots);
    if (s != UQ_OK) return s;
    p.kv_fmt = ref_fmt(desc);
    p.scales = nullptr;
    if (desc->format == UQ_REF_TQ4) tq_tables(desc->codebook, p.tq);
    if (desc->format == UQ_REF_FP8_E4M3) {
        p.scale_log2 = float(double(softmax_scale) * double(desc->k_scale) * 1.4426950408889634);
        p.out_scale = desc->v_scale;
        p.k_scale = desc->k_scale;
        p.v_scale = desc->v_scale;
        if (!(isfinite(p.scale_log2) && p.scale_log2 > 0.0f)) return UQ_ERR_INVALID_ARGUMENT;
    }
    return UQ_OK;
}

uq_status uq_ref_decode_attention(const uq_ref_cache_desc* desc, const void* q, uq_dtype q_dtype, int32_t batch,
                                  int32_t num_q_heads, const uint8_t* cache, const int32_t* page_table,
                                  int32_t max_pages_per_seq, const int32_t* context_lens, int32_t max_context,
                                  float softmax_scale, int32_t partition_tokens, void* workspace,
                                  size_t workspace_bytes, void* out, uq_dtype out_dtype, void* stream) {
    uq::DecodeParams p;
    uq_status s = ref_decode_setup(desc, q, q_dtype, batch, num_q_heads, cache, page_table, max_pages_per_seq,
                                   context_lens, max_context, softmax_scale, partition_tokens, workspace,
                                   workspace_bytes, out, out_dtype, p);
    if (s != UQ_OK) return s;
    s = from_hip(uq::launch_decode_partials(p, static_cast<hipStream_t>(stream)));
    if (s != UQ_OK) return s;
    return from_hip(uq::launch_decode_merge(p, static_cast<hipStream_t>(stream)));
}

uq_status uq_ref_decode_partials(const uq_ref_cache_desc* desc, const void* q, uq_dtype q_dtype, int32_t batch,
                                 int32_t num_q_heads, const uint8_t* cache, const int32_t* page_table,
                                 int32_t max_pages_per_seq, const int32_t* context_lens, int32_t max_context,
                                 float softmax_scale, int32_t partition_tokens, void* workspace,
                                 size_t workspace_bytes, void* out, uq_dtype out_dtype, void* stream) {
    uq::DecodeParams p;
    uq_status s = ref_decode_setup(desc, q, q_dtype, batch, num_q_heads, cache, page_table, max_pages_per_seq,
                                   context_lens, max_context, softmax_scale, partition_tokens, workspace,
                                   workspace_bytes, out, out_dtype, p);
    if (s != UQ_OK) return s;
    return from_hip(uq::launch_decode_partials(p, static_cast<hipStream_t>(stream)));
}

uq_status uq_ref_decode_step(const uq_ref_cache_desc* desc, const void* q, uq_dtype q_dtype, const void* k_new,
                             const void* v_new, uq_dtype new_dtype, int32_t batch, int32_t num_q_heads,
                             uint8_t* cache, const int32_t* page_table, int32_t max_pages_per_seq,
                             const int32_t* context_lens, int32_t max_context, float softmax_scale,
                             int32_t partition_tokens, void* workspace, size_t workspace_bytes, void* out,
                             uq_dtype out_dtype, void* stream) {
    uq::DecodeParams p;
    uq_status s = ref_decode_setup(desc, q, q_dtype, batch, num_q_heads, cache, page_table, max_pages_per_seq,
                                   context_lens, max_context, softmax_scale, partition_tokens, workspace,
                                   workspace_bytes, out, out_dtype, p);
    if (s != UQ_OK) return s;
    s = step_args(k_new, v_new, new_dtype, p);
    if (s != UQ_OK) return s;
    s = from_hip(uq::launch_decode_partials(p, static_cast<hipStream_t>(stream)));
    if (s != UQ_OK) return s;
    return from_hip(uq::launch_decode_merge(p, static_cast<hipStream_t>(stream)));
}

uq_status uq_ref_decode_step_partials(const uq_ref_cache_desc* desc, const void* q, uq_dtype q_dtype,
                                      const void* k_new, const void* v_new, uq_dtype new_dtype, int32_t batch,
                                      int32_t num_q_heads, uint8_t* cache, const int32_t* page_table,
                                      int32_t max_pages_per_seq, const int32_t* context_lens, int32_t max_context,
                                      float softmax_scale, int32_t partition_tokens, void* workspace,
                                      size_t workspace_bytes, void* out, uq_dtype out_dtype, void* stream) {
    uq::DecodeParams p;
    uq_status s = ref_decode_setup(desc, q, q_dtype, batch, num_q_heads, cache, page_table, max_pages_per_seq,
                                   context_lens, max_context, softmax_scale, partition_tokens, workspace,
                                   workspace_bytes, out, out_dtype, p);
    if (s != UQ_OK) return s;
    s = step_args(k_new, v_new, new_dtype, p);
    if (s != UQ_OK) return s;
    return from_hip(uq::launch_decode_partials(p, static_cast<hipStream_t>(stream)));
}

uq_status uq_ref_decode_merge(const uq_ref_cache_desc* desc, int32_t batch, int32_t num_q_heads,
                              const int32_t* context_lens, int32_t max_context, int32_t partition_tokens,
                              const void* workspace, size_t workspace_bytes, void* out, uq_dtype out_dtype,
                              void* stream) {
    uq_status s = check_ref_desc(desc);
    if (s != UQ_OK) return s;
    const uq_cache_desc g = geometry_of(desc);
    s = check_decode_common(&g, batch, num_q_heads, max_context, partition_tokens);
    if (s != UQ_OK) return s;
    if (context_lens == nullptr || out == nullptr) return UQ_ERR_INVALID_ARGUMENT;
    if (out_dtype != UQ_F32 && out_dtype != UQ_BF16) return UQ_ERR_UNSUPPORTED;
    if (!aligned16(out)) return UQ_ERR_INVALID_ARGUMENT;
    uq::DecodeParams p;
    s = make_decode_params(&g, nullptr, UQ_F32, batch, num_q_heads, nullptr, nullptr, nullptr, 1, context_lens,
                           max_context, 1.0f, partition_tokens, const_cast<void*>(workspace), workspace_bytes, out,
                           out_dtype, p);
    if (s != UQ_OK) return s;
    p.kv_fmt = ref_fmt(desc);
    if (desc->format == UQ_REF_FP8_E4M3) p.out_scale = desc->v_scale;
    return from_hip(uq::launch_decode_merge(p, static_cast<hipStream_t>(stream)));
}

// ---------------------------------------------------------------- cascade decode

static int32_t group_of(int32_t num_q_heads, int32_t num_kv_heads) {
    return num_kv_heads > 0 && num_q_heads % num_kv_heads == 0 ? num_q_heads / num_kv_heads : 1;
}

size_t uq_decode_cascade_workspace_bytes(int32_t num_kv_heads, int32_t batch, int32_t num_q_heads,
                                         int32_t max_context, int32_t partition_tokens,
                                         const uq_shared_prefix* prefix) {
    if (check_prefix(prefix) != UQ_OK) return 0;
    uq_cache_desc d;
    d.num_kv_heads = num_kv_heads;
    d.head_dim = kHeadDim;
    d.page_size = kPageSize;
    d.group_size = kGroupSize;
    d.num_pages = 1;
    d.c = 0.156f;
    d.rotate_v = 0;
    if (check_decode_common(&d, batch, num_q_heads, max_context, partition_tokens) != UQ_OK) return 0;
    const int32_t part = partition_tokens == 0 ? pick_partition(batch, num_kv_heads, max_context) : partition_tokens;
    return workspace_for(batch, num_q_heads, num_kv_heads, max_context, part,
                         prefix_slots(prefix, num_kv_heads, batch, group_of(num_q_heads, num_kv_heads)));
}

static uq_status cascade_finish_setup(const void* k_new, const void* v_new, uq_dtype new_dtype,
                                      const uq_shared_prefix* prefix, uq::DecodeParams& p) {
    if (k_new != nullptr || v_new != nullptr) {
        const uq_status s = step_args(k_new, v_new, new_dtype, p);
        if (s != UQ_OK) return s;
    }
    return apply_prefix(prefix, p);
}

static uq_status cascade_setup(const uq_cache_desc* desc, const void* q, uq_dtype q_dtype, const void* k_new,
                               const void* v_new, uq_dtype new_dtype, int32_t batch, int32_t num_q_heads,
                               uint8_t* kv_codes, uint8_t* kv_scales, const int32_t* page_table,
                               int32_t max_pages_per_seq, const int32_t* context_lens, int32_t max_context,
                               const uq_shared_prefix* prefix, float softmax_scale, int32_t partition_tokens,
                               void* workspace, size_t workspace_bytes, void* out, uq_dtype out_dtype,
                               uq::DecodeParams& p) {
    uq_status s = check_prefix(prefix);
    if (s != UQ_OK) return s;
    s = check_desc(desc);
    if (s != UQ_OK) return s;
    s = require_128(desc);
    if (s != UQ_OK) return s;
    s = decode_setup(desc, q, q_dtype, batch, num_q_heads, kv_codes, kv_scales, page_table, max_pages_per_seq,
                     context_lens, max_context, softmax_scale, partition_tokens, workspace, workspace_bytes, out,
                     out_dtype, p, prefix_slots(prefix, desc->num_kv_heads, batch, group_of(num_q_heads, desc->num_kv_heads)));
    if (s != UQ_OK) return s;
    return cascade_finish_setup(k_new, v_new, new_dtype, prefix, p);
}

uq_status uq_decode_cascade(const uq_cache_desc* desc, const void* q, uq_dtype q_dtype, const void* k_new,
                            const void* v_new, uq_dtype new_dtype, int32_t batch, int32_t num_q_heads,
                            uint8_t* kv_codes, uint8_t* kv_scales, const int32_t* page_table,
                            int32_t max_pages_per_seq, const int32_t* context_lens, int32_t max_context,
                            const uq_shared_prefix* prefix, float softmax_scale, int32_t partition_tokens,
                            void* workspace, size_t workspace_bytes, void* out, uq_dtype out_dtype, void* stream) {
    uq::DecodeParams p;
    uq_status s = cascade_setup(desc, q, q_dtype, k_new, v_new, new_dtype, batch, num_q_heads, kv_codes, kv_scales,
                                page_table, max_pages_per_seq, context_lens, max_context, prefix, softmax_scale,
                                partition_tokens, workspace, workspace_bytes, out, out_dtype, p);
    if (s != UQ_OK) return s;
    s = from_hip(uq::launch_decode_partials(p, static_cast<hipStream_t>(stream)));
    if (s != UQ_OK) return s;
    return from_hip(uq::launch_decode_merge(p, static_cast<hipStream_t>(stream)));
}

uq_status uq_decode_cascade_partials(const uq_cache_desc* desc, const void* q, uq_dtype q_dtype, const void* k_new,
                                     const void* v_new, uq_dtype new_dtype, int32_t batch, int32_t num_q_heads,
                                     uint8_t* kv_codes, uint8_t* kv_scales, const int32_t* page_table,
                                     int32_t max_pages_per_seq, const int32_t* context_lens, int32_t max_context,
                                     const uq_shared_prefix* prefix, float softmax_scale, int32_t partition_tokens,
                                     void* workspace, size_t workspace_bytes, void* out, uq_dtype out_dtype,
                                     void* stream) {
    uq::DecodeParams p;
    uq_status s = cascade_setup(desc, q, q_dtype, k_new, v_new, new_dtype, batch, num_q_heads, kv_codes, kv_scales,
                                page_table, max_pages_per_seq, context_lens, max_context, prefix, softmax_scale,
                                partition_tokens, workspace, workspace_bytes, out, out_dtype, p);
    if (s != UQ_OK) return s;
    return from_hip(uq::launch_decode_partials(p, static_cast<hipStream_t>(stream)));
}

// Shared set-up of the two cascade merge calls.
static uq_status cascade_merge_setup(const uq_cache_desc* g, int32_t batch, int32_t num_q_heads,
                                     const int32_t* context_lens, int32_t max_context, const uq_shared_prefix* prefix,
                                     int32_t partition_tokens, const void* workspace, size_t workspace_bytes,
                                     void* out, uq_dtype out_dtype, uq::DecodeParams& p) {
    uq_status s = check_prefix(prefix);
    if (s != UQ_OK) return s;
    s = check_decode_common(g, batch, num_q_heads, max_context, partition_tokens);
    if (s != UQ_OK) return s;
    if (context_lens == nullptr || out == nullptr) return UQ_ERR_INVALID_ARGUMENT;
    if (out_dtype != UQ_F32 && out_dtype != UQ_BF16) return UQ_ERR_UNSUPPORTED;
    if (!aligned16(out)) return UQ_ERR_INVALID_ARGUMENT;
    s = make_decode_params(g, nullptr, UQ_F32, batch, num_q_heads, nullptr, nullptr, nullptr, 1, context_lens,
                           max_context, 1.0f, partition_tokens, const_cast<void*>(workspace), workspace_bytes, out,
                           out_dtype, p, prefix_slots(prefix, g->num_kv_heads, batch, num_q_heads / g->num_kv_heads));
    if (s != UQ_OK) return s;
    return apply_prefix(prefix, p);
}

uq_status uq_decode_cascade_merge(const uq_cache_desc* desc, int32_t batch, int32_t num_q_heads,
                                  const int32_t* context_lens, int32_t max_context, const uq_shared_prefix* prefix,
                                  int32_t partition_tokens, const void* workspace, size_t workspace_bytes, void* out,
                                  uq_dtype out_dtype, void* stream) {
    uq_status s = check_desc(desc);
    if (s != UQ_OK) return s;
    s = require_128(desc);
    if (s != UQ_OK) return s;
    uq::DecodeParams p;
    s = cascade_merge_setup(desc, batch, num_q_heads, context_lens, max_context, prefix, partition_tokens, workspace,
                            workspace_bytes, out, out_dtype, p);
    if (s != UQ_OK) return s;
    return from_hip(uq::launch_decode_merge(p, static_cast<hipStream_t>(stream)));
}

static uq_status ref_cascade_setup(const uq_ref_cache_desc* desc, const void* q, uq_dtype q_dtype, const void* k_new,
                                   const void* v_new, uq_dtype new_dtype, int32_t batch, int32_t num_q_heads,
                                   uint8_t* cache, const int32_t* page_table, int32_t max_pages_per_seq,
                                   const int32_t* context_lens, int32_t max_context, const uq_shared_prefix* prefix,
                                   float softmax_scale, int32_t partition_tokens, void* workspace,
                                   size_t workspace_bytes, void* out, uq_dtype out_dtype, uq::DecodeParams& p) {
    uq_status s = check_prefix(prefix);
    if (s != UQ_OK) return s;
    s = check_ref_desc(desc);
    if (s != UQ_OK) return s;
    s = ref_decode_setup(desc, q, q_dtype, batch, num_q_heads, cache, page_table, max_pages_per_seq, context_lens,
                         max_context, softmax_scale, partition_tokens, workspace, workspace_bytes, out, out_dtype, p,
                         prefix_slots(prefix, desc->num_kv_heads, batch, group_of(num_q_heads, desc->num_kv_heads)));
    if (s != UQ_OK) return s;
    return cascade_finish_setup(k_new, v_new, new_dtype, prefix, p);
}

uq_status uq_ref_decode_cascade(const uq_ref_cache_desc* desc, const void* q, uq_dtype q_dtype, const void* k_new,
                                const void* v_new, uq_dtype new_dtype, int32_t batch, int32_t num_q_heads,
                                uint8_t* cache, const int32_t* page_table, int32_t max_pages_per_seq,
                                const int32_t* context_lens, int32_t max_context, const uq_shared_prefix* prefix,
                                float softmax_scale, int32_t partition_tokens, void* workspace,
                                size_t workspace_bytes, void* out, uq_dtype out_dtype, void* stream) {
    uq::DecodeParams p;
    uq_status s = ref_cascade_setup(desc, q, q_dtype, k_new, v_new, new_dtype, batch, num_q_heads, cache, page_table,
                                    max_pages_per_seq, context_lens, max_context, prefix, softmax_scale,
                                    partition_tokens, workspace, workspace_bytes, out, out_dtype, p);
    if (s != UQ_OK) return s;
    s = from_hip(uq::launch_decode_partials(p, static_cast<hipStream_t>(stream)));
    if (s != UQ_OK) return s;
    return from_hip(uq::launch_decode_merge(p, static_cast<hipStream_t>(stream)));
}

uq_status uq_ref_decode_cascade_partials(const uq_ref_cache_desc* desc, const void* q, uq_dtype q_dtype,
                                         const void* k_new, const void* v_new, uq_dtype new_dtype, int32_t batch,
                                         int32_t num_q_heads, uint8_t* cache, const int32_t* page_table,
                                         int32_t max_pages_per_seq, const int32_t* context_lens,
                                         int32_t max_context, const uq_shared_prefix* prefix, float softmax_scale,
                                         int32_t partition_tokens, void* workspace, size_t workspace_bytes,
                                         void* out, uq_dtype out_dtype, void* stream) {
    uq::DecodeParams p;
    uq_status s = ref_cascade_setup(desc, q, q_dtype, k_new, v_new, new_dtype, batch, num_q_heads, cache, page_table,
                                    max_pages_per_seq, context_lens, max_context, prefix, softmax_scale,
                                    partition_tokens, workspace, workspace_bytes, out, out_dtype, p);
    if (s != UQ_OK) return s;
    return from_hip(uq::launch_decode_partials(p, static_cast<hipStream_t>(stream)));
}

uq_status uq_ref_decode_cascade_merge(const uq_ref_cache_desc* desc, int32_t batch, int32_t num_q_heads,
                                      const int32_t* context_lens, int32_t max_context,
                                      const uq_shared_prefix* prefix, int32_t partition_tokens,
                                      const void* workspace, size_t workspace_bytes, void* out, uq_dtype out_dtype,
                                      void* stream) {
    uq_status s = check_ref_desc(desc);
    if (s != UQ_OK) return s;
    const uq_cache_desc g = geometry_of(desc);
    uq::DecodeParams p;
    s = cascade_merge_setup(&g, batch, num_q_heads, context_lens, max_context, prefix, partition_tokens, workspace,
                            workspace_bytes, out, out_dtype, p);
    if (s != UQ_OK) return s;
    p.kv_fmt = ref_fmt(desc);
    if (desc->format == UQ_REF_FP8_E4M3) p.out_scale = desc->v_scale;
    return from_hip(uq::launch_decode_merge(p, static_cast<hipStream_t>(stream)));
}

uq_status uq_decode_attention_noalloc(const uq_cache_desc* desc, const void* q, uq_dtype q_dtype, int32_t batch,
                                      int32_t num_q_heads, const uint8_t* kv_codes, const uint8_t* kv_scales,
                                      const int32_t* page_table, int32_t max_pages_per_seq,
                                      const int32_t* context_lens, int32_t max_context, float softmax_scale,
                                      int32_t partition_tokens, void* out, uq_dtype out_dtype, void* stream) {
    // every host-side check of uq_decode_attention, the size bound included
    // (WORKSPACE_TOO_SMALL), before the first HIP call: an aligned stand-in
    // address takes the array's place until its device address is known
    uq::DecodeParams p;
    void* const stand_in = reinterpret_cast<void*>(uintptr_t(256));
    uq_status s = decode_setup(desc, q, q_dtype, batch, num_q_heads, kv_codes, kv_scales, page_table,
                               max_pages_per_seq, context_lens, max_context, softmax_scale, partition_tokens,
                               stand_in, UQ_NOALLOC_SCRATCH_BYTES, out, out_dtype, p);
    if (s != UQ_OK) return s;
    void* base = nullptr;
    s = scratch_of_current_device(&base);
    if (s != UQ_OK) return s;
    // the same parameter block with the array's device address
    s = decode_setup(desc, q, q_dtype, batch, num_q_heads, kv_codes, kv_scales, page_table, max_pages_per_seq,
                     context_lens, max_context, softmax_scale, partition_tokens, base, UQ_NOALLOC_SCRATCH_BYTES, out,
                     out_dtype, p);
    if (s != UQ_OK) return s;
    s = from_hip(uq::launch_decode_partials(p, static_cast<hipStream_t>(stream)));
    if (s != UQ_OK) return s;
    return from_hip(uq::launch_decode_merge(p, static_cast<hipStream_t>(stream)));
}

uq_status uq_probe_stream_read(const void* buf, size_t bytes, uint32_t* sink, void* stream) {
    if (buf == nullptr || sink == nullptr || bytes == 0 || bytes % 16 != 0) return UQ_ERR_INVALID_ARGUMENT;
    if (!aligned16(buf) || (reinterpret_cast<uintptr_t>(sink) & 3u) != 0) return UQ_ERR_INVALID_ARGUMENT;
    return from_hip(uq::launch_stream_read_probe(buf, int64_t(bytes / 16), sink, UQ_PROBE_STREAM_BLOCKS,
                                                 static_cast<hipStream_t>(stream)));
}

uq_status uq_probe_page_gather(const uq_cache_desc* desc, int32_t batch, int32_t num_q_heads, const uint8_t* kv_codes,
                               const uint8_t* kv_scales, const int32_t* page_table, int32_t max_pages_per_seq,
                               const int32_t* context_lens, int32_t max_context, int32_t partition_tokens,
                               uint32_t* sink, size_t sink_words, void* stream) {
    // the decode call's own checks (the sink stands in for the query, the
    // output and the workspace, which the probe does not touch)
    uq::DecodeParams p;
    const size_t ws = uq_decode_workspace_bytes(desc, batch, num_q_heads, max_context, partition_tokens);
    uq_status s = decode_setup(desc, sink, UQ_F32, batch, num_q_heads, kv_codes, kv_scales, page_table,
                               max_pages_per_seq, context_lens, max_context, 1.0f, partition_tokens, sink, ws, sink,
                               UQ_F32, p);
    if (s != UQ_OK) return s;
    if (sink_words < size_t(uq::probe_words(p))) return UQ_ERR_WORKSPACE_TOO_SMALL;
    return from_hip(uq::launch_gather_probe(p, sink, static_cast<hipStream_t>(stream)));
}

uq_status uq_probe_page_gather_cascade(const uq_cache_desc* desc, int32_t batch, int32_t num_q_heads,
                                       const uint8_t* kv_codes, const uint8_t* kv_scales, const int32_t* page_table,
                                       int32_t max_pages_per_seq, const int32_t* context_lens, int32_t max_context,
                                       const uq_shared_prefix* prefix, int32_t partition_tokens, void* workspace,
                                       size_t workspace_bytes, uint32_t* sink, size_t sink_words, void* stream) {
    // the cascade call's own checks (the sink stands in for the query and the
    // output; the workspace receives the row list)
    uq::DecodeParams p;
    uq_status s = cascade_setup(desc, sink, UQ_F32, nullptr, nullptr, UQ_F32, batch, num_q_heads,
                                const_cast<uint8_t*>(kv_codes), const_cast<uint8_t*>(kv_scales), page_table,
                                max_pages_per_seq, context_lens, max_context, prefix, 1.0f, partition_tokens, workspace,
                                workspace_bytes, sink, UQ_F32, p);
    if (s != UQ_OK) return s;
    if (sink_words < size_t(uq::probe_words(p))) return UQ_ERR_WORKSPACE_TOO_SMALL;
    return from_hip(uq::launch_gather_probe(p, sink, static_cast<hipStream_t>(stream)));
}

uq_status uq_probe_mfma(int32_t kind, const void* a, const void* b, const uint8_t* scale_a, const uint8_t* scale_b,
                        int32_t n, float* d, void* stream) {
    if (kind < 0 || kind > 3 || n < 1 || n > 65535) return UQ_ERR_INVALID_ARGUMENT;
    if (a == nullptr || b == nullptr || d == nullptr) return UQ_ERR_INVALID_ARGUMENT;
    if (kind != 2 && (scale_a == nullptr || scale_b == nullptr)) return UQ_ERR_INVALID_ARGUMENT;
    if (!aligned16(a) || !aligned16(b) || !aligned16(d)) return UQ_ERR_INVALID_ARGUMENT;
    return from_hip(uq::launch_mfma_probe(kind, a, b, scale_a, scale_b, n, d, static_cast<hipStream_t>(stream)));
}

uq_status uq_time_next_launch(void* start_event, void* stop_event) {
    if ((start_event == nullptr) != (stop_event == nullptr)) return UQ_ERR_INVALID_ARGUMENT;
    uq::time_next_launch(static_cast<hipEvent_t>(start_event), static_cast<hipEvent_t>(stop_event));
    return UQ_OK;
}

}  // extern "C"
