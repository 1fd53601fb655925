/*
 * uq.h -- C ABI of libuq: FP4 (E2M1 + UE8M0) KV-cache decode attention for
 * AMD Instinct MI355X (gfx950), after "UltraQuant" (arXiv 2606.20474).
 *
 * The library implements the two halves of the paper's Algorithm 1:
 *   Write  (uq_quantize_kv)      rotate K (and V when rotate_v) with the
 *                                fixed d-point Walsh-Hadamard transform,
 *                                pick one UE8M0 exponent per 32 channels,
 *                                round every element onto the E2M1 grid and
 *                                store 2 codes per byte + 1 scale byte.
 *   Decode (uq_decode_attention) rotate the query, cast it to FP8 E4M3 once,
 *                                compute QK^T on the block-scaled FP8 x FP4
 *                                MFMA with the stored UE8M0 bytes as operand
 *                                scales, convert V through the hardware
 *                                FP4 -> BF16 path, and run softmax attention
 *                                split over context partitions, then merge.
 *
 * Conventions shared by every call
 * --------------------------------
 *  - All pointers except `desc` and the host-side scalars are DEVICE
 *    pointers on the current HIP device.  `stream` is a hipStream_t (NULL =
 *    the default stream).  Every call only enqueues work on `stream`; none
 *    synchronises.  The library allocates nothing and keeps no pointer after
 *    a call returns (except the two events of uq_time_next_launch, held for
 *    the calling thread's next launch); the caller owns every buffer.  Calls
 *    are thread-safe.
 *  - Arguments are validated on the host before any HIP call: a failed
 *    check returns its status and enqueues nothing.  Device-resident
 *    indices (page ids, slots, context lengths) cannot be checked without a
 *    synchronisation; kernels clamp them so that no access leaves the pools
 *    (an out-of-range page id reads page 0, an out-of-range slot is
 *    skipped), but such results are unspecified.
 *  - Supported shape: head_dim d = 64, 128 or 256, page_size 16,
 *    group_size 32, up to 16 query heads per KV head.  Other values return
 *    UQ_ERR_UNSUPPORTED.  The paper's layers use d = 128; the decode step,
 *    cascade decode, the pre-cast FP8 query, uq_prepare_query and the
 *    comparison caches are d = 128 calls (UNSUPPORTED for 64 and 256).
 *    Sizes written 128 below are d for head sizes 64 and 256.
 *  - Inputs must be finite.  Attention stays finite and accurate for scores
 *    (q.k * softmax_scale * log2 e) of any magnitude up to 1e30, as long as
 *    the fp32 products themselves do not overflow; only tokens inside a
 *    context are read, so every one of them must have been written.
 *
 * Cache format (the "pools")
 * --------------------------
 * One tile holds one (page, kv head, K or V): 16 tokens x d channels.
 *   kv_codes  : uint8 [num_pages][num_kv_heads][2 (K=0, V=1)][8 d]
 *   kv_scales : uint8 [num_pages][num_kv_heads][2 (K=0, V=1)][d/32 groups][16 tokens]
 * 17 bytes per 32 elements = 4.25 bits per element (paper, "Cache Layout");
 * 17 d / 16 bytes (136 at d = 128) per token and kv head for K and V together.
 * Inside a code tile (8 d bytes), for token t (0..15) and channel ch
 * (0..d-1), the even channel of a pair in the low nibble:
 *   K: byte ((ch/32)*16 + t)*16 + (ch%32)/2
 *      ([group][token][16 bytes] -- one lane of the QK MFMA reads one
 *       token's 32-channel group as 16 contiguous bytes, and its scale byte
 *       sits at the same [group][token] index: the scale layout matches the
 *       operand layout of the block-scaled MFMA, paper "Kernel
 *       Implementation in vLLM")
 *   V: byte ((t/4)*(d/8) + ch/8)*16 + (t%4)*4 + (ch%8)/2
 *      ([token/4][channel/8][token%4][4 bytes] -- one lane of the PV step
 *       reads 4 tokens x 8 channels as 16 contiguous bytes)
 * A code is sign(1) | E2M1 magnitude index(3) over {0,.5,1,1.5,2,3,4,6};
 * a scale byte is E + 127 and the element value is code * 2^(byte-127)
 * (paper, "Dequantization").
 */
#ifndef UQ_H_
#define UQ_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* The enumerations are 32-bit integers on both sides of the ABI; a C caller
 * may pass any int32_t value (out-of-range values are rejected, and
 * uq_status_string names them UQ_ERR_UNKNOWN), so C++ gives them that
 * underlying type explicitly. */
#ifdef __cplusplus
#define UQ_ENUM_BASE : int32_t
#else
#define UQ_ENUM_BASE
#endif

typedef enum uq_status UQ_ENUM_BASE {
    UQ_OK = 0,
    UQ_ERR_INVALID_ARGUMENT = 1,   /* null pointer, negative size, inconsistent shape */
    UQ_ERR_UNSUPPORTED = 2,        /* valid request outside the supported shapes */
    UQ_ERR_WORKSPACE_TOO_SMALL = 3,
    UQ_ERR_HIP = 4                 /* a HIP launch failed (hipGetLastError) */
} uq_status;

typedef enum uq_dtype UQ_ENUM_BASE {
    UQ_F32 = 0,
    UQ_BF16 = 1,
    UQ_F16 = 2,
    UQ_FP8_E4M3 = 3                /* OCP e4m3fn */
} uq_dtype;

typedef struct uq_cache_desc {
    int32_t num_kv_heads;   /* >= 1 */
    int32_t head_dim;       /* 64, 128 or 256 */
    int32_t page_size;      /* must be 16 */
    int32_t group_size;     /* must be 32 */
    int64_t num_pages;      /* pages in the pools, >= 1 */
    float c;                /* global scale constant, finite and > 0; the paper deploys 0.156 */
    int32_t rotate_v;       /* 0: V stored unrotated (Algorithm 1 as printed); 1: V rotated like K */
} uq_cache_desc;

/* Human-readable name of a status code; never NULL. */
const char *uq_status_string(uq_status s);

/* Library version, major*10000 + minor*100 + patch. */
int32_t uq_version(void);

/*
 * uq_quantize_kv -- quantize-on-write (Algorithm 1, "Write").
 *   k, v          : [num_tokens][num_kv_heads][128] of in_dtype (F32, BF16 or
 *                   F16); token t starts at element t * token_stride, heads
 *                   are contiguous inside a token (token_stride >=
 *                   num_kv_heads * 128).
 *   slot_mapping  : int64 [num_tokens].  With page_table == NULL it holds the
 *                   physical slot page * 16 + offset (vLLM convention).  With
 *                   a page table it holds the logical slot
 *                   seq * (max_pages_per_seq * 16) + position, and the page
 *                   is page_table[seq][position / 16].  Negative = padding,
 *                   skipped; a slot beyond the pool (or a sequence index
 *                   >= num_seqs) is skipped too.
 *   page_table    : int32 [num_seqs][max_pages_per_seq] or NULL.
 *   k, v must be 16-byte aligned and token_stride a multiple of 16 bytes.
 *   kv_codes, kv_scales : the pools described above; only the slots named
 *                   by slot_mapping are written.  Two tokens of one call
 *                   naming the same slot race: the slot's bytes are then
 *                   unspecified (possibly a mix of both tokens).
 * Per token and head the K vector is always rotated, V only with rotate_v.
 * Codes and scale bytes are a pure function of the inputs and `c`.
 * Errors: INVALID_ARGUMENT for null k/v/slot_mapping/pools, num_tokens < 0,
 * token_stride too small or misaligned, non-finite or non-positive c,
 * num_seqs < 1 or max_pages_per_seq < 1 with a page table; UNSUPPORTED for other head_dim/page/group sizes or
 * an unknown in_dtype.  num_tokens == 0 is a no-op.
 */
uq_status uq_quantize_kv(const uq_cache_desc *desc, const void *k, const void *v, uq_dtype in_dtype,
                         int64_t num_tokens, int64_t token_stride, const int32_t *page_table, int32_t num_seqs,
                         int32_t max_pages_per_seq, const int64_t *slot_mapping, uint8_t *kv_codes,
                         uint8_t *kv_scales, void *stream);

/*
 * uq_prepare_query -- the query half of Algorithm 1, "Decode":
 * q8 = e4m3fn(R q) for `rows` 128-vectors (round to nearest even, saturate
 * at +-448, no query scale).  q: [rows][128] F32/BF16/F16; q_fp8: [rows][128]
 * bytes.  uq_decode_attention does this itself; this entry point exposes the
 * step for callers that cache the FP8 query and for tests.
 */
uq_status uq_prepare_query(const uq_cache_desc *desc, const void *q, uq_dtype q_dtype, int64_t rows,
                           uint8_t *q_fp8, void *stream);

/*
 * Workspace needed by uq_decode_attention for these sizes: per (sequence,
 * query head, partition) 128 fp32 accumulators, a running max and a running
 * sum.  partition_tokens == 0 selects the library's default partition for
 * the shape.  Returns 0 for invalid arguments.
 */
size_t uq_decode_workspace_bytes(const uq_cache_desc *desc, int32_t batch, int32_t num_q_heads,
                                 int32_t max_context, int32_t partition_tokens);

/* Partition length (tokens) the library picks when partition_tokens == 0:
 * the longest (1024 .. 16384) that still gives the 256 compute units two
 * blocks each.  A block serves one KV head, or two at head size 64 when the
 * group size is at most 8 and num_kv_heads is even (the kernel then treats
 * the pair as one 128-channel head with a block-diagonal query operand). */
int32_t uq_default_partition(const uq_cache_desc *desc, int32_t batch, int32_t num_q_heads, int32_t max_context);

/*
 * uq_decode_attention -- decode attention over the FP4 cache (Algorithm 1,
 * "Decode"), one new query token per sequence: one launch of the partition
 * kernel, plus one launch of the merge kernel when a context can span more
 * than one partition (max_context > partition).  The partition kernel runs
 * one block of 4 waves per (partition, kv head, sequence), the waves sharing
 * the partition's pages, or -- when the launch has at least 2048 blocks of
 * W partitions each (head size 128, no shared prefix; W = 8 where that many
 * blocks of 8 exist and there are 16 partitions or more, else 4) -- one
 * wave per partition, a block taking W consecutive partitions of one
 * sequence and kv head and reducing their partials into one before the
 * merge.  The result does not depend on the grid beyond rounding.
 *   q             : [batch][num_q_heads][128].  F32/BF16/F16: rotated and
 *                   cast to FP8 inside the call.  FP8_E4M3: already
 *                   prepared by uq_prepare_query.
 *   page_table    : int32 [batch][max_pages_per_seq], physical page ids.
 *   context_lens  : int32 [batch] on the device; tokens 0..len-1 attend.
 *   max_context   : host-side upper bound of every context_lens[b]
 *                   (<= max_pages_per_seq * 16); sizes the grid without a
 *                   device read.  Lengths above it are clamped to it.
 *   softmax_scale : multiplies q.k (usually 1/sqrt(128)); finite and > 0.
 *   partition_tokens : context tokens per split-context partition, a
 *                   multiple of 16 (whole pages), or 0 for the default.
 *   workspace     : >= uq_decode_workspace_bytes(...) bytes of device
 *                   memory, 16-byte aligned, no initial contents required.
 *                   Calls that share a workspace must not run concurrently.
 *   out           : [batch][num_q_heads][128] F32 or BF16.  With rotate_v
 *                   the output is rotated back (o <- R o), so it is in the
 *                   same basis as an unrotated V.  An empty context gives 0.
 * Query head h reads kv head h / (num_q_heads / num_kv_heads).
 * Errors: INVALID_ARGUMENT for null pointers, batch/num_q_heads < 1,
 * num_q_heads % num_kv_heads != 0, max_context < 0 or above
 * max_pages_per_seq * 16, partition_tokens not a multiple of 16, a
 * non-finite or non-positive softmax_scale, misaligned q/pools/workspace/out; UNSUPPORTED
 * for more than 16 query heads per kv head or unsupported dtypes;
 * WORKSPACE_TOO_SMALL.
 */
uq_status uq_decode_attention(const uq_cache_desc *desc, const void *q, uq_dtype q_dtype, int32_t batch,
                              int32_t num_q_heads, const uint8_t *kv_codes, const uint8_t *kv_scales,
                              const int32_t *page_table, int32_t max_pages_per_seq, const int32_t *context_lens,
                              int32_t max_context, float softmax_scale, int32_t partition_tokens,
                              void *workspace, size_t workspace_bytes, void *out, uq_dtype out_dtype,
                              void *stream);

/*
 * The two launches of uq_decode_attention, for callers that time or overlap
 * them.  uq_decode_partials runs the partition kernel: each block writes
 * a partial (running max, running sum, 128 accumulators per query head) of
 * its partition (its W partitions on the wave grid) into the workspace, or
 * the final output when it holds the whole context.  uq_decode_merge
 * merges the partials into `out` (a no-op when max_context <= partition).  Called back
 * to back on one stream with the same arguments they are exactly
 * uq_decode_attention; the arguments, validation and errors are the same.
 */
uq_status uq_decode_partials(const uq_cache_desc *desc, const void *q, uq_dtype q_dtype, int32_t batch,
                             int32_t num_q_heads, const uint8_t *kv_codes, const uint8_t *kv_scales,
                             const int32_t *page_table, int32_t max_pages_per_seq, const int32_t *context_lens,
                             int32_t max_context, float softmax_scale, int32_t partition_tokens,
                             void *workspace, size_t workspace_bytes, void *out, uq_dtype out_dtype,
                             void *stream);

/*
 * uq_decode_step -- one decode step of Algorithm 1 in one call: write each
 * sequence's new K and V token into the FP4 cache ("Write"), then decode
 * attention over the context that now ends with it ("Decode").
 *   k_new, v_new : [batch][num_kv_heads][128] rows of new_dtype (F32, BF16
 *                  or F16), 16-byte aligned.  Sequence b's token is
 *                  quantised exactly as uq_quantize_kv does and stored at
 *                  position len_b - 1, len_b = min(context_lens[b],
 *                  max_context), through page_table; it is part of the
 *                  attended context.  A sequence with len_b <= 0 writes
 *                  nothing.  The page holding position len_b - 1 must not
 *                  be a page another sequence of the call reads.
 *   kv_codes, kv_scales : the pools, read and (one token per sequence and
 *                  kv head) written.
 * The write is done inside the partition kernel by the block that reads
 * that page, so the step costs the launches of uq_decode_attention.
 * Every other argument, the output and the errors are those of
 * uq_decode_attention (plus INVALID_ARGUMENT for null or misaligned
 * k_new/v_new and UNSUPPORTED for other new_dtype).
 * uq_decode_step_partials is its first launch; uq_decode_merge with the
 * same arguments finishes it.
 */
uq_status uq_decode_step(const uq_cache_desc *desc, const void *q, uq_dtype q_dtype, const void *k_new,
                         const void *v_new, uq_dtype new_dtype, int32_t batch, int32_t num_q_heads,
                         uint8_t *kv_codes, uint8_t *kv_scales, const int32_t *page_table, int32_t max_pages_per_seq,
                         const int32_t *context_lens, int32_t max_context, float softmax_scale,
                         int32_t partition_tokens, void *workspace, size_t workspace_bytes, void *out,
                         uq_dtype out_dtype, void *stream);
uq_status uq_decode_step_partials(const uq_cache_desc *desc, const void *q, uq_dtype q_dtype, const void *k_new,
                                  const void *v_new, uq_dtype new_dtype, int32_t batch, int32_t num_q_heads,
                                  uint8_t *kv_codes, uint8_t *kv_scales, const int32_t *page_table,
                                  int32_t max_pages_per_seq, const int32_t *context_lens, int32_t max_context,
                                  float softmax_scale, int32_t partition_tokens, void *workspace,
                                  size_t workspace_bytes, void *out, uq_dtype out_dtype, void *stream);

uq_status uq_decode_merge(const uq_cache_desc *desc, int32_t batch, int32_t num_q_heads,
                          const int32_t *context_lens, int32_t max_context, int32_t partition_tokens,
                          const void *workspace, size_t workspace_bytes, void *out, uq_dtype out_dtype,
                          void *stream);

/*
 * uq_quantize_error -- calibration of the scale constant c (section
 * "Constant-Optimized Scaling": c is chosen once, offline, to minimise the
 * reconstruction error of the E2M1 grid on rotated key rows).  For each
 * candidate c_values[i], every row of x (128 channels, rotated first when
 * `rotate`) is quantised per 32-channel group with the scale
 * s = 2^round(log2(c m)) of the cache format (pow2_scale = 1) or the
 * continuous s = c m of the paper's fitting objective (pow2_scale = 0),
 * decoded back to code * s, and
 *   sums[2 i]     += sum over rows and channels of (x - decoded)^2,
 *   sums[2 i + 1] += sum of x^2 (the same for every i).
 * The sums accumulate (zero them before the first call; several calls can
 * cover one large set).  x: F32/BF16/F16 rows, row_stride elements apart,
 * 16-byte aligned; c_values: num_c floats (device), finite and > 0;
 * sums: 2 * num_c doubles (device).
 * rows = 0 launches nothing (x may then be NULL).
 * Errors: INVALID_ARGUMENT for NULL pointers, rows < 0, num_c outside
 * [0, 256], row_stride < 128 or misaligned rows; UNSUPPORTED for other
 * dtypes.  Asynchronous on `stream`; the library keeps no pointer.
 */
uq_status uq_quantize_error(const void *x, uq_dtype dtype, int64_t rows, int64_t row_stride, int32_t rotate,
                            int32_t pow2_scale, int32_t num_c, const float *c_values, double *sums, void *stream);

/* ------------------------------------------------------------------------
 * Cascade decode over a shared prefix.
 *
 * Many sequences of a batch often begin with the same pages (a shared system
 * prompt or document: the prefix reuse the paper's agent traces show,
 * section "Introduction" and the MiniMax-like workload).  The cascade calls
 * read those pages once per KV head for all sequences together: a prefix
 * block takes 16 (sequence, query head) pairs as the 16 query columns of
 * its matrix instructions, whatever the group size, and the context blocks
 * start each sequence after its prefix.  The two kinds of partial results
 * are merged per (sequence, query head) as split contexts are.  The output
 * is the attention over the same tokens as uq_decode_attention; only the
 * order of the floating-point sums differs.
 * ---------------------------------------------------------------------- */

typedef struct uq_shared_prefix {
    const int32_t *pages;     /* [num_tokens / 16] physical page ids of the shared prefix (device) */
    const int32_t *lens;      /* [batch] (device): the first lens[b] tokens of sequence b are the first
                                 lens[b] tokens of the shared prefix; a multiple of 16, at most num_tokens
                                 and below context_lens[b] (larger values are clamped to that).  The
                                 tokens from lens[b] on are read through page_table as usual. */
    int32_t num_tokens;       /* prefix length in tokens, a positive multiple of 16 */
    int32_t partition_tokens; /* prefix tokens per prefix block, a multiple of 32, or 0 for the default */
} uq_shared_prefix;

/* Workspace of the cascade calls (FP4 and comparison caches): the partial
 * rows of the context and prefix partitions (rounded up to 16 bytes), then
 * the dispatch list of the partition kernel, 16 bytes per (context
 * partition, sequence) and per (chunk of 16 query columns, prefix
 * partition); 0 for invalid arguments. */
size_t uq_decode_cascade_workspace_bytes(int32_t num_kv_heads, int32_t batch, int32_t num_q_heads,
                                         int32_t max_context, int32_t partition_tokens,
                                         const uq_shared_prefix *prefix);

/*
 * uq_decode_cascade -- uq_decode_attention (k_new == v_new == NULL) or
 * uq_decode_step (both given) with a shared prefix.  The new token of a
 * step is written at position len_b - 1, which lies after lens[b].
 * Arguments, output and errors are those of uq_decode_step, plus
 * INVALID_ARGUMENT for a NULL prefix, pages or lens, a num_tokens that is not
 * a positive multiple of 16, a prefix partition_tokens that is not a multiple of 32,
 * or only one of k_new, v_new.  uq_decode_cascade_partials is its first
 * part and uq_decode_cascade_merge (with the same prefix and partition)
 * its second.  The first part is two launches: a one-block kernel lists the
 * (context partition, sequence) rows in the workspace, the ones with the
 * most tokens first, then the prefix rows, and the partition kernel's
 * blocks take their rows from that list, so that the longest blocks start
 * first and short ones fill the end; the order changes no result.
 */
uq_status uq_decode_cascade(const uq_cache_desc *desc, const void *q, uq_dtype q_dtype, const void *k_new,
                            const void *v_new, uq_dtype new_dtype, int32_t batch, int32_t num_q_heads,
                            uint8_t *kv_codes, uint8_t *kv_scales, const int32_t *page_table,
                            int32_t max_pages_per_seq, const int32_t *context_lens, int32_t max_context,
                            const uq_shared_prefix *prefix, float softmax_scale, int32_t partition_tokens,
                            void *workspace, size_t workspace_bytes, void *out, uq_dtype out_dtype, void *stream);
uq_status uq_decode_cascade_partials(const uq_cache_desc *desc, const void *q, uq_dtype q_dtype, const void *k_new,
                                     const void *v_new, uq_dtype new_dtype, int32_t batch, int32_t num_q_heads,
                                     uint8_t *kv_codes, uint8_t *kv_scales, const int32_t *page_table,
                                     int32_t max_pages_per_seq, const int32_t *context_lens, int32_t max_context,
                                     const uq_shared_prefix *prefix, float softmax_scale, int32_t partition_tokens,
                                     void *workspace, size_t workspace_bytes, void *out, uq_dtype out_dtype,
                                     void *stream);
uq_status uq_decode_cascade_merge(const uq_cache_desc *desc, int32_t batch, int32_t num_q_heads,
                                  const int32_t *context_lens, int32_t max_context, const uq_shared_prefix *prefix,
                                  int32_t partition_tokens, const void *workspace, size_t workspace_bytes, void *out,
                                  uq_dtype out_dtype, void *stream);

/* ------------------------------------------------------------------------
 * Plain comparison caches.
 *
 * The paper measures the FP4 path against a hardware FP8 KV cache and a
 * BF16 KV cache (section "Performance Results").  These calls build both
 * with the same paging and the same decode kernel as the FP4 cache (the
 * same staging ring, online softmax, PV and merge), so a comparison between
 * them measures the cache format.  FP8 and BF16 rotate nothing.
 *
 * Pool layout (one buffer, caller-owned, uq_ref_cache_bytes bytes):
 * [num_pages][num_kv_heads][K, V][tile], tile = 16 tokens x 128 channels in
 * the lane order the decode kernel reads:
 *   FP8  (2048 B): K at ((c%64)/16 * 16 + t) * 32 + c%16 + (c >= 64 ? 16 : 0);
 *                  V at ((t/4) * 16 + c/8) * 32 + (t%4) * 8 + c%8.
 *   BF16 (4096 B): K at ((c/8) * 16 + t) * 16 + 2 * (c%8);
 *                  V at ((t/4) * 16 + c/8) * 64 + (t%4) * 16 + 2 * (c%8).
 * (t = token within the page, c = channel; FP8 entries are one byte, BF16
 * entries two, little endian.)
 *
 * TQ4 is the codebook encoding UltraQuant replaces (appendix "Calibrated LUT
 * int4 KV Encoding (Ultra-TQ)", its algorithm): K is rotated by the same
 * R as the FP4 cache, its norm n (the l2 norm of the rotated fp32 key,
 * rounded once to fp32) is stored per token and each rotated channel x is
 * coded to the index of the codebook level c_j (rounded to BF16) nearest to
 * x / n, ties to the lower index: the number of midpoints m_j = (c_j +
 * c_{j+1}) / 2 with x > m_j n, compared exactly (index 0 when n = 0); the
 * decoded key is n * c[idx].  A codebook must be 16 finite, strictly
 * ascending values whose adjacent BF16 levels lie within 2^44 of each other
 * (so that each m_j is exact in fp64), else INVALID_ARGUMENT.  V is not
 * rotated: per 32-channel group,
 * z = bf16(min), s = bf16(max(max - z, 0) / 15), code = clamp(rint((x - z)
 * / s), 0, 15) (0 when s = 0), decoded as bf16(fma(s, code, z)).  Decode
 * attention rotates the query and rounds it to BF16.  The block of one
 * (page, kv head) is 2368 bytes:
 *   [0, 1024)     K indices, (t, c) at 16 * (t + 16 * ((c%32)/8)) + 4 * (c/32)
 *                 + (c%8)/2;
 *   [1024, 2048)  V codes at 1024 + 16 * (c/8 + 16 * (t/4)) + 4 * (t%4) + (c%8)/2;
 *                 (low nibble = even channel in both);
 *   [2048, 2112)  K norms, fp32, token t at 2048 + 4 t;
 *   [2112, 2368)  V (s, z) as two BF16 (s in the low half), token t and
 *                 group g at 2112 + 16 * (4 * (t/4) + g) + 4 * (t%4).
 * ---------------------------------------------------------------------- */

typedef enum uq_ref_format UQ_ENUM_BASE {
    UQ_REF_FP8_E4M3 = 1, /* OCP E4M3 (no infinities), one scale per tensor */
    UQ_REF_BF16 = 2,
    UQ_REF_TQ4 = 3       /* the Ultra-TQ codebook cache (see below) */
} uq_ref_format;

typedef struct uq_ref_cache_desc {
    int32_t num_kv_heads;
    int32_t head_dim;  /* must be 128 */
    int32_t page_size; /* must be 16 */
    int32_t format;    /* uq_ref_format */
    int64_t num_pages;
    float k_scale;     /* FP8: stored byte = e4m3(x / k_scale), value = byte * k_scale;  */
    float v_scale;     /* finite and > 0.  Ignored for BF16 and TQ4. */
    const float *codebook; /* TQ4: 16 finite key levels (host memory, read during each
                              call), strictly ascending once rounded to BF16.  Ignored
                              for FP8 and BF16. */
} uq_ref_cache_desc;

/* Bytes of the pool of a comparison cache; 0 for an invalid descriptor. */
size_t uq_ref_cache_bytes(const uq_ref_cache_desc *desc);

/*
 * uq_ref_write_kv -- write K and V rows into a comparison cache: FP8 bytes
 * are e4m3(x / scale) rounded to nearest even and saturated at +-448; BF16
 * is round-to-nearest-even; TQ4 as described above.  Arguments, slot addressing (physical slots, or
 * logical slots through page_table), skipped slots and errors are those of
 * uq_quantize_kv; `cache` must be 16-byte aligned.  A TQ4 descriptor whose
 * codebook is NULL, non-finite or not strictly ascending in BF16 is
 * INVALID_ARGUMENT (for every call taking the descriptor).
 */
uq_status uq_ref_write_kv(const uq_ref_cache_desc *desc, const void *k, const void *v, uq_dtype in_dtype,
                          int64_t num_tokens, int64_t token_stride, const int32_t *page_table, int32_t num_seqs,
                          int32_t max_pages_per_seq, const int64_t *slot_mapping, uint8_t *cache, void *stream);

/* Workspace of uq_ref_decode_attention; 0 for invalid arguments. */
size_t uq_ref_decode_workspace_bytes(const uq_ref_cache_desc *desc, int32_t batch, int32_t num_q_heads,
                                     int32_t max_context, int32_t partition_tokens);

/*
 * uq_ref_decode_attention -- decode attention over a comparison cache.  q is
 * F32, BF16 or F16 (never pre-cast).  FP8 cache: the query is cast to E4M3
 * (nearest even, saturating) and q.k runs on the FP8 x FP8 matrix
 * instruction; the scores are multiplied by softmax_scale * k_scale and the
 * output by v_scale.  BF16 cache: the query is cast to BF16 and q.k runs on
 * BF16 matrix instructions.  TQ4 cache: the rotated query is cast to BF16,
 * the K indices are decoded through the BF16 levels, q.k runs on BF16
 * matrix instructions and each score is multiplied by its token's norm; V
 * is decoded to BF16 values.  Every other argument, the output and the
 * errors are those of uq_decode_attention.  uq_ref_decode_partials and
 * uq_ref_decode_merge are its two launches, as for the FP4 cache.
 */
uq_status uq_ref_decode_attention(const uq_ref_cache_desc *desc, const void *q, uq_dtype q_dtype, int32_t batch,
                                  int32_t num_q_heads, const uint8_t *cache, const int32_t *page_table,
                                  int32_t max_pages_per_seq, const int32_t *context_lens, int32_t max_context,
                                  float softmax_scale, int32_t partition_tokens, void *workspace,
                                  size_t workspace_bytes, void *out, uq_dtype out_dtype, void *stream);
uq_status uq_ref_decode_partials(const uq_ref_cache_desc *desc, const void *q, uq_dtype q_dtype, int32_t batch,
                                 int32_t num_q_heads, const uint8_t *cache, const int32_t *page_table,
                                 int32_t max_pages_per_seq, const int32_t *context_lens, int32_t max_context,
                                 float softmax_scale, int32_t partition_tokens, void *workspace,
                                 size_t workspace_bytes, void *out, uq_dtype out_dtype, void *stream);
/* The decode step over a comparison cache: uq_decode_step with the token
 * stored as uq_ref_write_kv stores it. */
uq_status uq_ref_decode_step(const uq_ref_cache_desc *desc, const void *q, uq_dtype q_dtype, const void *k_new,
                             const void *v_new, uq_dtype new_dtype, int32_t batch, int32_t num_q_heads,
                             uint8_t *cache, const int32_t *page_table, int32_t max_pages_per_seq,
                             const int32_t *context_lens, int32_t max_context, float softmax_scale,
                             int32_t partition_tokens, void *workspace, size_t workspace_bytes, void *out,
                             uq_dtype out_dtype, void *stream);
uq_status uq_ref_decode_step_partials(const uq_ref_cache_desc *desc, const void *q, uq_dtype q_dtype,
                                      const void *k_new, const void *v_new, uq_dtype new_dtype, int32_t batch,
                                      int32_t num_q_heads, uint8_t *cache, const int32_t *page_table,
                                      int32_t max_pages_per_seq, const int32_t *context_lens, int32_t max_context,
                                      float softmax_scale, int32_t partition_tokens, void *workspace,
                                      size_t workspace_bytes, void *out, uq_dtype out_dtype, void *stream);
/* Cascade decode over a comparison cache: uq_decode_cascade with the cache
 * and token format of uq_ref_decode_step. */
uq_status uq_ref_decode_cascade(const uq_ref_cache_desc *desc, const void *q, uq_dtype q_dtype, const void *k_new,
                                const void *v_new, uq_dtype new_dtype, int32_t batch, int32_t num_q_heads,
                                uint8_t *cache, const int32_t *page_table, int32_t max_pages_per_seq,
                                const int32_t *context_lens, int32_t max_context, const uq_shared_prefix *prefix,
                                float softmax_scale, int32_t partition_tokens, void *workspace,
                                size_t workspace_bytes, void *out, uq_dtype out_dtype, void *stream);
uq_status uq_ref_decode_cascade_partials(const uq_ref_cache_desc *desc, const void *q, uq_dtype q_dtype,
                                         const void *k_new, const void *v_new, uq_dtype new_dtype, int32_t batch,
                                         int32_t num_q_heads, uint8_t *cache, const int32_t *page_table,
                                         int32_t max_pages_per_seq, const int32_t *context_lens,
                                         int32_t max_context, const uq_shared_prefix *prefix, float softmax_scale,
                                         int32_t partition_tokens, void *workspace, size_t workspace_bytes,
                                         void *out, uq_dtype out_dtype, void *stream);
uq_status uq_ref_decode_cascade_merge(const uq_ref_cache_desc *desc, int32_t batch, int32_t num_q_heads,
                                      const int32_t *context_lens, int32_t max_context,
                                      const uq_shared_prefix *prefix, int32_t partition_tokens,
                                      const void *workspace, size_t workspace_bytes, void *out, uq_dtype out_dtype,
                                      void *stream);
uq_status uq_ref_decode_merge(const uq_ref_cache_desc *desc, int32_t batch, int32_t num_q_heads,
                              const int32_t *context_lens, int32_t max_context, int32_t partition_tokens,
                              const void *workspace, size_t workspace_bytes, void *out, uq_dtype out_dtype,
                              void *stream);

/* ------------------------------------------------------------------------
 * uq_decode_attention_scaled_pv -- uq_decode_attention with PV on the
 * block-scaled matrix instruction (Algorithm 1, Decode, "PV via FP4/scale
 * path"; section "UltraQuant Kernel Ladder"): a prototype kept for
 * measurement against the default BF16 PV path.  QK^T and the softmax are
 * the default kernel's; PV runs on v_mfma_scale_f32_16x16x128_f8f6f4 with
 * the raw E2M1 V codes as one operand and P, scaled per (token, channel
 * group) by V's UE8M0 scale and split into four FP8 terms, as the other
 * (the instruction's scales are per 32-token block and cannot carry V's
 * per-token scales).  Head size 128 only; V scale bytes up to 135
 * (|V| < 6 * 2^8) keep the FP8 terms in range.  Arguments, outputs and
 * errors as uq_decode_attention, plus UNSUPPORTED for other head sizes and
 * INVALID_ARGUMENT for a partition_tokens that is not a multiple of 32.
 * ---------------------------------------------------------------------- */
uq_status uq_decode_attention_scaled_pv(const uq_cache_desc *desc, const void *q, uq_dtype q_dtype, int32_t batch,
                                        int32_t num_q_heads, const uint8_t *kv_codes, const uint8_t *kv_scales,
                                        const int32_t *page_table, int32_t max_pages_per_seq,
                                        const int32_t *context_lens, int32_t max_context, float softmax_scale,
                                        int32_t partition_tokens, void *workspace, size_t workspace_bytes, void *out,
                                        uq_dtype out_dtype, void *stream);

/* ------------------------------------------------------------------------
 * uq_decode_attention_noalloc -- uq_decode_attention for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc.  The partition partials go to a device
 * array the library holds for the life of the process (one per GPU, made at
 * module load; UQ_NOALLOC_SCRATCH_BYTES bytes) instead of a caller's
 * workspace.  The call makes no hipMalloc, hipFree or other allocating
 * call: its first call on a device looks the array's address up once
 * (hipGetSymbolAddress) with that device current.
 *   Arguments, layouts, launches, numerics and errors are those of
 *   uq_decode_attention without the workspace pair: the output is the same,
 *   bit for bit, for the same arguments.  The stream must belong to the
 *   current device.
 *   WORKSPACE_TOO_SMALL when the call needs more than the array holds, i.e.
 *   uq_decode_workspace_bytes(desc, batch, num_q_heads, max_context,
 *   partition_tokens) > UQ_NOALLOC_SCRATCH_BYTES (checked on the host before
 *   anything is enqueued); UQ_ERR_HIP if the address lookup fails.
 *   Every call on a GPU shares that GPU's array: calls that overlap on one GPU
 *   (other streams, other host threads) race and must be serialised by the
 *   caller.  Nothing in the array needs to start at zero: every partial the
 *   merge reads is written by the same call first.
 * ---------------------------------------------------------------------- */
#define UQ_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)
uq_status uq_decode_attention_noalloc(const uq_cache_desc *desc, const void *q, uq_dtype q_dtype, int32_t batch,
                                      int32_t num_q_heads, const uint8_t *kv_codes, const uint8_t *kv_scales,
                                      const int32_t *page_table, int32_t max_pages_per_seq,
                                      const int32_t *context_lens, int32_t max_context, float softmax_scale,
                                      int32_t partition_tokens, void *out, uq_dtype out_dtype, void *stream);

/* ------------------------------------------------------------------------
 * Measurement probes (diagnostics, not part of the method; section
 * "Kernel-Level Roofline Analysis" measures against the HBM roof, and these
 * give the share of it this GPU actually delivers to the access patterns of
 * this library, and the arithmetic of its matrix instructions).
 *
 * uq_probe_stream_read -- read `bytes` of device memory at `buf` once
 *   (UQ_PROBE_STREAM_BLOCKS blocks, each streaming its own contiguous share
 *   with non-temporal 16-byte loads), XOR-folding them into one checksum
 *   word per block in `sink`.  Its kernel time is the time a plain stream
 *   of that many bytes takes.
 *   buf 16-byte aligned, bytes > 0 and a multiple of 16; sink: at least
 *   UQ_PROBE_STREAM_BLOCKS uint32 words of device memory.
 *   Errors: INVALID_ARGUMENT otherwise.
 *
 * uq_probe_page_gather -- the FP4 decode kernel's memory traffic alone:
 *   the partition launch of uq_decode_attention for these arguments, run
 *   as a probe: its grid (one block per partition, or one wave per
 *   partition on the grid the library picks for many partitions; head
 *   sizes 64, 128 and 256), page walk through page_table, page-id copies
 *   and 2-slot LDS ring filled by the same copy instructions with the same
 *   cache policy, every staged byte read back into registers, and no query
 *   prologue, arithmetic or partial rows: each wave writes one uint32 XOR
 *   checksum of what it staged to sink[W * block + wave] (0 for a wave
 *   without pages; W, the waves per block, is 8 on a one-wave-per-partition
 *   grid of blocks of 8 partitions, else 4).  Arguments as
 *   uq_decode_attention; sink_words >= 4 x partitions x num_kv_heads x
 *   batch (partitions = ceil(max_context / partition), the partition being
 *   partition_tokens or, for 0, the library's default for the shape) always
 *   suffices: W words per block of the launch are written; sink 16-byte
 *   aligned.
 *   Errors: those of uq_decode_attention's argument checks;
 *   WORKSPACE_TOO_SMALL for a short sink.
 *
 * uq_probe_page_gather_cascade -- the same probe of uq_decode_cascade's
 *   partition launch: the row list is written to `workspace` (sized as for
 *   uq_decode_cascade) and the context and shared-prefix blocks stage their
 *   pages as the cascade kernel does (the prefix pages with the default
 *   cache policy).  sink_words >= 4 x (context blocks + prefix blocks),
 *   context blocks = partitions x num_kv_heads x batch, prefix blocks =
 *   num_kv_heads x ceil(batch x group / 16) x prefix partitions; rows
 *   without work leave their 4 words 0.  Errors: those of
 *   uq_decode_cascade's argument checks; WORKSPACE_TOO_SMALL for a short
 *   sink.
 *
 * uq_probe_mfma -- n independent one-wave products D = A x B of one matrix
 *   instruction on given operand bytes, in the instruction's lane layout:
 *   a, b: [n][64 lanes][32 bytes] (an FP4 operand uses the first 16 bytes of
 *   a lane: 32 E2M1 codes, k order = nibble order, low nibble first; a BF16
 *   operand the first 16: 8 values); scale_a, scale_b: [n][64] UE8M0 bytes,
 *   lane 16 j + i scaling row (A) or column (B) i over k-block j of 32;
 *   d: [n][64][4] floats, lane l element r = D[4 (l / 16) + r][l % 16].
 *   kind 0: v_mfma_scale_f32_16x16x128_f8f6f4 with A FP4 E2M1, B FP8 E4M3
 *   (the QK^T instruction of the decode kernel); kind 1: the same with A and
 *   B FP8 E4M3 (the FP8-KV comparator's); kind 2:
 *   v_mfma_f32_16x16x32_bf16 (scales unused, may be NULL); kind 3: the
 *   scaled instruction with A FP8 E4M3, B FP4 E2M1.  Lane l of an operand
 *   holds row (A) or column (B) l % 16; k = 32 (l / 16) + e for FP4 element
 *   e; for FP8 bytes 0..15 are k = 16 (l / 16) + e, bytes 16..31 are k = 64
 *   + 16 (l / 16) + e - 16; for BF16 k = 8 (l / 16) + e.
 *   Errors: INVALID_ARGUMENT for null or misaligned pointers, n < 1 or
 *   n > 65535, an unknown kind.
 * ---------------------------------------------------------------------- */
#define UQ_PROBE_STREAM_BLOCKS 2048
uq_status uq_probe_stream_read(const void *buf, size_t bytes, uint32_t *sink, void *stream);
uq_status uq_probe_page_gather(const uq_cache_desc *desc, int32_t batch, int32_t num_q_heads,
                               const uint8_t *kv_codes, const uint8_t *kv_scales, const int32_t *page_table,
                               int32_t max_pages_per_seq, const int32_t *context_lens, int32_t max_context,
                               int32_t partition_tokens, uint32_t *sink, size_t sink_words, void *stream);
uq_status uq_probe_page_gather_cascade(const uq_cache_desc *desc, int32_t batch, int32_t num_q_heads,
                                       const uint8_t *kv_codes, const uint8_t *kv_scales, const int32_t *page_table,
                                       int32_t max_pages_per_seq, const int32_t *context_lens, int32_t max_context,
                                       const uq_shared_prefix *prefix, int32_t partition_tokens, void *workspace,
                                       size_t workspace_bytes, uint32_t *sink, size_t sink_words, void *stream);
uq_status uq_probe_mfma(int32_t kind, const void *a, const void *b, const uint8_t *scale_a, const uint8_t *scale_b,
                        int32_t n, float *d, void *stream);

/* ------------------------------------------------------------------------
 * Kernel timing (benchmarks).
 *
 * HIP events recorded on the stream around a call also count the command
 * processor's dispatch and completion latency (a few microseconds).  After
 * uq_time_next_launch(start, stop), the next launch of the decode partition
 * kernel (by uq_decode_attention, uq_decode_partials,
 * uq_decode_step(_partials), the cascade calls or their comparison-cache
 * forms), of the quantize-on-write kernel (uq_quantize_kv) or of a bandwidth
 * probe (uq_probe_stream_read, uq_probe_page_gather(_cascade)) made from the calling
 * host thread is dispatched with hipExtLaunchKernel, which sets
 * `start` and `stop` (hipEvent_t, created by the caller, not owned by the
 * library) to that kernel's own start and end; hipEventElapsedTime(start,
 * stop) is then the kernel's duration.  The setting is used by that one
 * launch and then cleared (a call that fails its checks launches nothing
 * and leaves it); NULL, NULL clears it.  Errors: INVALID_ARGUMENT when
 * exactly one of the two is NULL.
 * ---------------------------------------------------------------------- */
uq_status uq_time_next_launch(void *start_event, void *stop_event);

#ifdef __cplusplus
}
#endif

#endif /* UQ_H_ */
