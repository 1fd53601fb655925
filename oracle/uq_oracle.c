/*
 * uq_oracle.c -- plain, slow CPU oracle for the UltraQuant FP4 KV-cache path.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link, load or
 * call this file; only the test suite, the smoke check and the benchmark's
 * CPU-baseline leg use it.  It shares no code, header, table or constant
 * generator with the HIP library: every rule below is written out from the
 * paper (arXiv 2606.20474, "UltraQuant") and from the cache-format
 * specification in include/uq.h.
 *
 * What it computes (each function cites the passage it follows):
 *   - the fixed Walsh-Hadamard rotation R = H_128 / sqrt(128)
 *       (section "Ultra-TurboQuant": a fixed WHT spreads outliers;
 *        Algorithm 1, Write: K <- R.K; Decode: Q <- R.Q),
 *   - per-32-channel UE8M0 exponent E = round(log2(c * m)), m = max|x|
 *       (section "Constant-Optimized Scaling"; Algorithm 1, Write),
 *   - FP4 E2M1 nearest-level rounding q(x / 2^E) onto
 *       F = {0, +-0.5, +-1, +-1.5, +-2, +-3, +-4, +-6}
 *       (section "Constant-Optimized Scaling", the definition of q),
 *   - packing 2 codes per byte + 1 scale byte per group
 *       (section "Cache Layout": 17 bytes per 32 elements),
 *   - dequantisation value = code * 2^(byte - 127)
 *       (section "Dequantization", its single equation),
 *   - the FP8 E4M3 query cast (Algorithm 1, Decode),
 *   - softmax attention over the dequantised cache, in fp64,
 *   - the round-trip error sum(z - s q(z / s))^2 behind the offline choice
 *       of c (section "Constant-Optimized Scaling", the c* equation).
 *
 * Readings where the paper is silent (the same list is kept with the design
 * notes of the repository):
 *   R1 the rotation is Sylvester H_128 with no sign diagonal, evaluated in
 *      fp32 as an in-place butterfly with stage widths 1,2,4,...,64, pair
 *      (i, i+h) -> (x_i + x_{i+h}, x_i - x_{i+h}), then one fp32 multiply by
 *      fl32(1/sqrt(128)).  Codes are integers decided from these fp32 values,
 *      so the order is part of the format.
 *   R2 "round(log2(y))" is nearest-integer rounding in the log domain
 *      (threshold at significand sqrt(2)); y = fl32(c * m) is one fp32
 *      multiply.  m = 0 gives E = -127.  E is clamped to [-127, 127], so the
 *      byte E + 127 is never the UE8M0 NaN byte 255.
 *   R3 ties in q go to the level with an even E2M1 code; values beyond 6
 *      saturate to 6; the sign bit of x is kept even when |code| = 0.
 *   R4 FP8 E4M3 is the OCP "fn" variant (bias 7, no infinities, max 448),
 *      round-to-nearest-even, saturating; no query scale.
 *   R5 K is always rotated; V is rotated iff rotate_v (Algorithm 1 rotates
 *      keys only; rotate_v = 0 is that mode).  With rotate_v the attention
 *      output is mapped back by R (R is symmetric and orthonormal).
 *
 * Built with: gcc -O2 -std=gnu11 -fopenmp -ffp-contract=off -shared -fPIC
 * -lquadmath (no -ffast-math: fp32 results must follow IEEE
 * round-to-nearest-even; binary128 gives the Ultra-TQ norm and index their
 * exact reference values).
 */
#include <math.h>
#include <omp.h>
#include <quadmath.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define UQO_D 128          /* head dimension of the fixed-size entry points */
#define UQO_DMAX 256       /* largest head dimension of the _d entry points (64, 128, 256) */
#define UQO_GROUP 32       /* channels per scale group */
#define UQO_NGROUP 4       /* groups per 128-channel head vector */
#define UQO_PAGE 16        /* tokens per page */

/* Threads the OpenMP loops of this file use. */
int uqo_num_threads(void) { return omp_get_max_threads(); }

/* The E2M1 magnitudes, indexed by the low 3 bits of a code (section
 * "Constant-Optimized Scaling", the set F). */
static const double kE2M1Mag[8] = {0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0};

/* ---------------------------------------------------------------------- */
/* Rotation (section "Ultra-TurboQuant"; Algorithm 1), reading R1, for a    */
/* head vector of d = 64, 128 or 256 channels: R = H_d / sqrt(d).           */
/* ---------------------------------------------------------------------- */
void uqo_wht_f32(float *x, int64_t n_vec, int d) {
    const float inv_sqrt = (float)(1.0 / sqrt((double)d));
    for (int64_t v = 0; v < n_vec; ++v) {
        float *p = x + v * d;
        for (int h = 1; h < d; h <<= 1) {
            for (int i = 0; i < d; ++i) {
                if (i & h) continue;
                float a = p[i], b = p[i + h];
                p[i] = a + b;
                p[i + h] = a - b;
            }
        }
        for (int i = 0; i < d; ++i) p[i] = p[i] * inv_sqrt;
    }
}
void uqo_wht128_f32(float *x, int64_t n_vec) { uqo_wht_f32(x, n_vec, UQO_D); }

/* Exact rotation in fp64: y = H_d x / sqrt(d), H[i][j] = (-1)^popcount(i&j). */
void uqo_wht_f64(const double *x, double *y, int d) {
    const double inv_sqrt = 1.0 / sqrt((double)d);
    for (int i = 0; i < d; ++i) {
        double s = 0.0;
        for (int j = 0; j < d; ++j)
            s += (__builtin_popcount((unsigned)(i & j)) & 1) ? -x[j] : x[j];
        y[i] = s * inv_sqrt;
    }
}
void uqo_wht128_f64(const double *x, double *y) { uqo_wht_f64(x, y, UQO_D); }

/* ---------------------------------------------------------------------- */
/* Scale exponent (section "Constant-Optimized Scaling"), reading R2.       */
/* ---------------------------------------------------------------------- */
int uqo_scale_exponent(float m, float c) {
    float y = c * m;                 /* one fp32 multiply */
    if (!(y > 0.0f)) return -127;    /* m = 0 (all-zero group) */
    int e;
    double f = frexp((double)y, &e); /* y = f * 2^e, f in [0.5, 1) */
    /* log2(y) = (e - 1) + log2(2f); round to nearest: +1 iff 2f >= sqrt(2).
     * 2f has 24 significant bits, so it never equals sqrt(2); the double
     * nearest to sqrt(2) separates the same fp32 neighbours. */
    int E = (e - 1) + ((2.0 * f >= sqrt(2.0)) ? 1 : 0);
    if (E < -127) E = -127;
    if (E > 127) E = 127;
    return E;
}

/* ---------------------------------------------------------------------- */
/* E2M1 rounding q(.) (section "Constant-Optimized Scaling"), reading R3.  */
/* Returns the 4-bit code: bit 3 = sign, bits 0-2 = index into F.           */
/* ---------------------------------------------------------------------- */
uint8_t uqo_e2m1_encode(float x, int E) {
    double t = ldexp((double)x, -E);   /* x / 2^E, exact in fp64 */
    double a = fabs(t);
    int best = 0;
    double best_d = fabs(a - kE2M1Mag[0]);
    for (int k = 1; k < 8; ++k) {
        double d = fabs(a - kE2M1Mag[k]);
        if (d < best_d || (d == best_d && (k % 2) == 0)) {
            best = k;
            best_d = d;
        }
    }
    return (uint8_t)((signbit(x) ? 8 : 0) | best);
}

/* Dequantisation (section "Dequantization"): code * 2^(byte - 127). */
double uqo_e2m1_value(uint8_t code, int scale_byte) {
    double mag = kE2M1Mag[code & 7];
    double v = ldexp(mag, scale_byte - 127);
    return (code & 8) ? -v : v;
}

/* ---------------------------------------------------------------------- */
/* FP8 E4M3 (OCP fn) encode / decode (Algorithm 1, Decode), reading R4.     */
/* ---------------------------------------------------------------------- */
double uqo_e4m3_value(uint8_t b) {
    int s = b >> 7, e = (b >> 3) & 15, m = b & 7;
    if (e == 15 && m == 7) return NAN;
    double v = (e == 0) ? ldexp((double)m / 8.0, -6) : ldexp(1.0 + (double)m / 8.0, e - 7);
    return s ? -v : v;
}

uint8_t uqo_e4m3_encode(float x) {
    if (isnan(x)) return 0x7F;
    if (isinf(x)) return (uint8_t)((signbit(x) ? 0x80 : 0) | 0x7E);
    double a = fabs((double)x);
    /* nearest among the 127 finite non-negative encodings 0x00..0x7E; the
     * byte order is the numeric order, ties go to the even byte (even
     * mantissa); anything above 448 lands on 448 (saturation). */
    int best = 0;
    double best_d = fabs(a - uqo_e4m3_value(0));
    for (int k = 1; k <= 0x7E; ++k) {
        double d = fabs(a - uqo_e4m3_value((uint8_t)k));
        if (d < best_d || (d == best_d && (k % 2) == 0)) {
            best = k;
            best_d = d;
        }
    }
    return (uint8_t)((signbit(x) ? 0x80 : 0) | best);
}

/* Query preparation (Algorithm 1, Decode): q8 = e4m3(R q), per d-vector. */
static void prepare_query_row(const float *q, uint8_t *q8, int d) {
    float tmp[UQO_DMAX];
    memcpy(tmp, q, sizeof(float) * (size_t)d);
    uqo_wht_f32(tmp, 1, d);
    for (int i = 0; i < d; ++i) q8[i] = uqo_e4m3_encode(tmp[i]);
}

void uqo_prepare_query_d(const float *q, int64_t rows, uint8_t *q8, int d) {
#pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < rows; ++r) prepare_query_row(q + r * d, q8 + r * d, d);
}
void uqo_prepare_query(const float *q, int64_t rows, uint8_t *q8) { uqo_prepare_query_d(q, rows, q8, UQO_D); }

/* ---------------------------------------------------------------------- */
/* Quantise one head vector of d channels (Algorithm 1, Write): optional    */
/* rotation, per-group exponent, per-element code.  codes[d] holds one code */
/* per byte, scale_bytes[d / 32] one byte per group.                        */
/* ---------------------------------------------------------------------- */
void uqo_quantize_vector_d(const float *x_in, int d, float c, int rotate, uint8_t *codes, uint8_t *scale_bytes) {
    float x[UQO_DMAX];
    memcpy(x, x_in, sizeof(float) * (size_t)d);
    if (rotate) uqo_wht_f32(x, 1, d);
    for (int g = 0; g < d / UQO_GROUP; ++g) {
        float m = 0.0f;
        for (int i = 0; i < UQO_GROUP; ++i) {
            float a = fabsf(x[g * UQO_GROUP + i]);
            if (a > m) m = a;
        }
        int E = uqo_scale_exponent(m, c);
        scale_bytes[g] = (uint8_t)(E + 127);
        for (int i = 0; i < UQO_GROUP; ++i) codes[g * UQO_GROUP + i] = uqo_e2m1_encode(x[g * UQO_GROUP + i], E);
    }
}
void uqo_quantize_vector(const float *x_in, float c, int rotate, uint8_t *codes, uint8_t *scale_bytes) {
    uqo_quantize_vector_d(x_in, UQO_D, c, rotate, codes, scale_bytes);
}

/* Batch form over n_vec contiguous d-vectors. */
void uqo_quantize_vectors_d(const float *x, int64_t n_vec, int d, float c, int rotate, uint8_t *codes,
                            uint8_t *scale_bytes) {
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n_vec; ++i)
        uqo_quantize_vector_d(x + i * d, d, c, rotate, codes + i * d, scale_bytes + i * (d / UQO_GROUP));
}
void uqo_quantize_vectors(const float *x, int64_t n_vec, float c, int rotate, uint8_t *codes, uint8_t *scale_bytes) {
    uqo_quantize_vectors_d(x, n_vec, UQO_D, c, rotate, codes, scale_bytes);
}

/* ---------------------------------------------------------------------- */
/* Page layout (the cache format of include/uq.h), for head size d.         */
/* Written out here from that specification, independently of the library. */
/*   codes  pool: [num_pages][num_kv_heads][2 = K,V][8 d bytes]             */
/*   scales pool: [num_pages][num_kv_heads][2 = K,V][d/32 groups][16 tokens]*/
/*   K tile byte of (token t, channel c): ((c/32)*16 + t)*16 + (c%32)/2     */
/*   V tile byte of (token t, channel c):                                   */
/*        ((t/4)*(d/8) + c/8)*16 + (t%4)*4 + (c%8)/2                        */
/*   even channel in the low nibble, odd channel in the high nibble.         */
/* ---------------------------------------------------------------------- */
static inline int64_t tile_index(int64_t page, int num_kv_heads, int head, int kv) {
    return (page * num_kv_heads + head) * 2 + kv;
}
static inline int code_byte_offset(int kv, int t, int ch, int d) {
    if (kv == 0) return ((ch / 32) * 16 + t) * 16 + (ch % 32) / 2;
    return ((t / 4) * (d / 8) + ch / 8) * 16 + (t % 4) * 4 + (ch % 8) / 2;
}

void uqo_store_vector_d(uint8_t *codes_pool, uint8_t *scales_pool, int num_kv_heads, int64_t page, int head, int kv,
                        int t, const uint8_t *codes, const uint8_t *scale_bytes, int d) {
    int64_t ti = tile_index(page, num_kv_heads, head, kv);
    uint8_t *ct = codes_pool + ti * (8 * d);
    uint8_t *st = scales_pool + ti * (d / 2);
    for (int ch = 0; ch < d; ++ch) {
        int off = code_byte_offset(kv, t, ch, d);
        if (ch % 2 == 0) ct[off] = (uint8_t)((ct[off] & 0xF0) | (codes[ch] & 0x0F));
        else ct[off] = (uint8_t)((ct[off] & 0x0F) | ((codes[ch] & 0x0F) << 4));
    }
    for (int g = 0; g < d / UQO_GROUP; ++g) st[g * UQO_PAGE + t] = scale_bytes[g];
}
void uqo_store_vector(uint8_t *codes_pool, uint8_t *scales_pool, int num_kv_heads, int64_t page, int head, int kv,
                      int t, const uint8_t *codes, const uint8_t *scale_bytes) {
    uqo_store_vector_d(codes_pool, scales_pool, num_kv_heads, page, head, kv, t, codes, scale_bytes, UQO_D);
}

void uqo_load_vector_d(const uint8_t *codes_pool, const uint8_t *scales_pool, int num_kv_heads, int64_t page,
                       int head, int kv, int t, uint8_t *codes, uint8_t *scale_bytes, int d) {
    int64_t ti = tile_index(page, num_kv_heads, head, kv);
    const uint8_t *ct = codes_pool + ti * (8 * d);
    const uint8_t *st = scales_pool + ti * (d / 2);
    for (int ch = 0; ch < d; ++ch) {
        uint8_t b = ct[code_byte_offset(kv, t, ch, d)];
        codes[ch] = (ch % 2 == 0) ? (b & 0x0F) : (b >> 4);
    }
    for (int g = 0; g < d / UQO_GROUP; ++g) scale_bytes[g] = st[g * UQO_PAGE + t];
}
void uqo_load_vector(const uint8_t *codes_pool, const uint8_t *scales_pool, int num_kv_heads, int64_t page, int head,
                     int kv, int t, uint8_t *codes, uint8_t *scale_bytes) {
    uqo_load_vector_d(codes_pool, scales_pool, num_kv_heads, page, head, kv, t, codes, scale_bytes, UQO_D);
}

/* ---------------------------------------------------------------------- */
/* Quantize-on-write (Algorithm 1, Write) into the paged pools.             */
/* k, v: [num_tokens][num_kv_heads][d] fp32 with a token stride in floats;   */
/* slot_mapping[t] = page * 16 + offset, negative = skip.  Returns the      */
/* number of tokens written.                                                 */
/* ---------------------------------------------------------------------- */
int64_t uqo_quantize_kv_d(const float *k, const float *v, int64_t num_tokens, int num_kv_heads, int64_t token_stride,
                          const int64_t *slot_mapping, int64_t num_pages, float c, int rotate_v, uint8_t *codes_pool,
                          uint8_t *scales_pool, int d) {
    int64_t written = 0;
#pragma omp parallel for schedule(static) reduction(+ : written)
    for (int64_t t = 0; t < num_tokens; ++t) {
        int64_t slot = slot_mapping[t];
        if (slot < 0 || slot >= num_pages * UQO_PAGE) continue;
        int64_t page = slot / UQO_PAGE;
        int off = (int)(slot % UQO_PAGE);
        for (int h = 0; h < num_kv_heads; ++h) {
            uint8_t codes[UQO_DMAX], sb[UQO_DMAX / UQO_GROUP];
            uqo_quantize_vector_d(k + t * token_stride + (int64_t)h * d, d, c, 1, codes, sb);
            uqo_store_vector_d(codes_pool, scales_pool, num_kv_heads, page, h, 0, off, codes, sb, d);
            uqo_quantize_vector_d(v + t * token_stride + (int64_t)h * d, d, c, rotate_v, codes, sb);
            uqo_store_vector_d(codes_pool, scales_pool, num_kv_heads, page, h, 1, off, codes, sb, d);
        }
        written += 1;
    }
    return written;
}
int64_t uqo_quantize_kv(const float *k, const float *v, int64_t num_tokens, int num_kv_heads, int64_t token_stride,
                        const int64_t *slot_mapping, int64_t num_pages, float c, int rotate_v, uint8_t *codes_pool,
                        uint8_t *scales_pool) {
    return uqo_quantize_kv_d(k, v, num_tokens, num_kv_heads, token_stride, slot_mapping, num_pages, c, rotate_v,
                             codes_pool, scales_pool, UQO_D);
}

/* Dequantise one stored vector to fp64 (section "Dequantization"). */
void uqo_dequant_vector_d(const uint8_t *codes_pool, const uint8_t *scales_pool, int num_kv_heads, int64_t page,
                          int head, int kv, int t, double *out, int d) {
    uint8_t codes[UQO_DMAX], sb[UQO_DMAX / UQO_GROUP];
    uqo_load_vector_d(codes_pool, scales_pool, num_kv_heads, page, head, kv, t, codes, sb, d);
    for (int ch = 0; ch < d; ++ch) out[ch] = uqo_e2m1_value(codes[ch], sb[ch / UQO_GROUP]);
}
void uqo_dequant_vector(const uint8_t *codes_pool, const uint8_t *scales_pool, int num_kv_heads, int64_t page,
                        int head, int kv, int t, double *out) {
    uqo_dequant_vector_d(codes_pool, scales_pool, num_kv_heads, page, head, kv, t, out, UQO_D);
}

/* ---------------------------------------------------------------------- */
/* Decode attention over the paged cache, fp64 (Algorithm 1, Decode).       */
/*   q: [batch][num_q_heads][d] fp32 (rotated and cast to FP8 here),        */
/*   page_table: [batch][max_pages_per_seq], context_lens: [batch].         */
/*   Query head h reads KV head h / (num_q_heads / num_kv_heads).           */
/*   out: [batch][num_q_heads][d] fp64; an empty context gives zeros.       */
/* Plain definition: s_j = scale * <q8, k_j>, p = softmax(s), o = sum p_j v_j */
/* then o <- R o when V was stored rotated.                                  */
/* ---------------------------------------------------------------------- */
void uqo_decode_attention_d(const float *q, int batch, int num_q_heads, int num_kv_heads, const uint8_t *codes_pool,
                            const uint8_t *scales_pool, const int32_t *page_table, int max_pages_per_seq,
                            const int32_t *context_lens, double softmax_scale, int rotate_v, double *out, int d) {
    const int G = num_q_heads / num_kv_heads;
#pragma omp parallel for schedule(dynamic) collapse(2)
    for (int b = 0; b < batch; ++b) {
        for (int hq = 0; hq < num_q_heads; ++hq) {
            const int hk = hq / G;
            const int ctx = context_lens[b];
            double *o = out + ((int64_t)b * num_q_heads + hq) * d;
            for (int i = 0; i < d; ++i) o[i] = 0.0;
            if (ctx <= 0) continue;
            uint8_t q8[UQO_DMAX];
            prepare_query_row(q + ((int64_t)b * num_q_heads + hq) * d, q8, d);
            double qd[UQO_DMAX];
            for (int i = 0; i < d; ++i) qd[i] = uqo_e4m3_value(q8[i]);
            double *s = (double *)malloc(sizeof(double) * (size_t)ctx);
            double kv[UQO_DMAX];
            double smax = -INFINITY;
            for (int j = 0; j < ctx; ++j) {
                int64_t page = page_table[(int64_t)b * max_pages_per_seq + j / UQO_PAGE];
                uqo_dequant_vector_d(codes_pool, scales_pool, num_kv_heads, page, hk, 0, j % UQO_PAGE, kv, d);
                double dot = 0.0;
                for (int i = 0; i < d; ++i) dot += qd[i] * kv[i];
                s[j] = softmax_scale * dot;
                if (s[j] > smax) smax = s[j];
            }
            double denom = 0.0;
            double acc[UQO_DMAX];
            for (int i = 0; i < d; ++i) acc[i] = 0.0;
            for (int j = 0; j < ctx; ++j) {
                double p = exp(s[j] - smax);
                denom += p;
                int64_t page = page_table[(int64_t)b * max_pages_per_seq + j / UQO_PAGE];
                uqo_dequant_vector_d(codes_pool, scales_pool, num_kv_heads, page, hk, 1, j % UQO_PAGE, kv, d);
                for (int i = 0; i < d; ++i) acc[i] += p * kv[i];
            }
            free(s);
            for (int i = 0; i < d; ++i) acc[i] /= denom;
            if (rotate_v) uqo_wht_f64(acc, o, d);
            else memcpy(o, acc, sizeof(double) * (size_t)d);
        }
    }
}
void uqo_decode_attention(const float *q, int batch, int num_q_heads, int num_kv_heads, const uint8_t *codes_pool,
                          const uint8_t *scales_pool, const int32_t *page_table, int max_pages_per_seq,
                          const int32_t *context_lens, double softmax_scale, int rotate_v, double *out) {
    uqo_decode_attention_d(q, batch, num_q_heads, num_kv_heads, codes_pool, scales_pool, page_table,
                           max_pages_per_seq, context_lens, softmax_scale, rotate_v, out, UQO_D);
}

/* ---------------------------------------------------------------------- */
/* Round-trip error of the encoder, for the offline fit of c (section      */
/* "Constant-Optimized Scaling": c* = argmin_c E[(z - c m q(z/(c m)))^2]   */
/* over rotated key rows).  Per row of 128 (rotated by R first when         */
/* `rotate`), per group of 32 with absmax m, for each c_values[i]:          */
/*   pow2 = 1  the cache's own rule: s = 2^E, E = uqo_scale_exponent(m, c), */
/*             decoded value F[code] * 2^E;                                 */
/*   pow2 = 0  the continuous scale of the fitting objective: s = fl32(c m),*/
/*             code = q(fl32(z / s)), decoded value F[code] * s.            */
/* sums[2i] += sum of (z - decoded)^2 and sums[2i+1] += sum of z^2, both in */
/* fp64 over all rows and channels.  Groups with m = 0 add nothing.         */
/* ---------------------------------------------------------------------- */
static void error_row(const float *x_in, int rotate, int pow2, int num_c, const float *c_values, double *acc) {
    float x[UQO_D];
    memcpy(x, x_in, sizeof(x));
    if (rotate) uqo_wht128_f32(x, 1);
    for (int g = 0; g < UQO_NGROUP; ++g) {
        const float *z = x + g * UQO_GROUP;
        float m = 0.0f;
        for (int i = 0; i < UQO_GROUP; ++i) {
            float a = fabsf(z[i]);
            if (a > m) m = a;
        }
        if (m == 0.0f) continue;
        double energy = 0.0;
        for (int i = 0; i < UQO_GROUP; ++i) energy += (double)z[i] * (double)z[i];
        for (int k = 0; k < num_c; ++k) {
            double err = 0.0;
            if (pow2) {
                int E = uqo_scale_exponent(m, c_values[k]);
                for (int i = 0; i < UQO_GROUP; ++i) {
                    double d = (double)z[i] - uqo_e2m1_value(uqo_e2m1_encode(z[i], E), E + 127);
                    err += d * d;
                }
            } else {
                float s = c_values[k] * m;             /* one fp32 multiply */
                for (int i = 0; i < UQO_GROUP; ++i) {
                    float t = z[i] / s;                /* one fp32 division */
                    double d = (double)z[i] - uqo_e2m1_value(uqo_e2m1_encode(t, 0), 127) * (double)s;
                    err += d * d;
                }
            }
            acc[2 * k] += err;
            acc[2 * k + 1] += energy;
        }
    }
}

void uqo_quantize_error(const float *x, int64_t rows, int rotate, int pow2, int num_c, const float *c_values,
                        double *sums) {
#pragma omp parallel
    {
        double *acc = (double *)calloc((size_t)(2 * num_c), sizeof(double));
#pragma omp for schedule(static)
        for (int64_t r = 0; r < rows; ++r) error_row(x + r * UQO_D, rotate, pow2, num_c, c_values, acc);
#pragma omp critical
        for (int k = 0; k < 2 * num_c; ++k) sums[k] += acc[k];
        free(acc);
    }
}

/* ====================================================================== */
/* Ultra-TQ comparison cache: the codebook encoding UltraQuant replaces    */
/* (appendix "Calibrated LUT int4 KV Encoding (Ultra-TQ)", its algorithm,  */
/* and section "Calibrated Centroids").  Readings where the paper leaves    */
/* the details open (kept with the design notes too):                       */
/*   T1 K is rotated by R, V is not.  K's block is the whole head vector    */
/*      (the production per-token l2 norm); V's blocks are the 32-channel  */
/*      groups.                                                             */
/*   T2 the norm n is the l2 norm of the fp32 rotated key, rounded once to  */
/*      fp32: the squares (exact) are summed in binary128 -- exactly, when  */
/*      the key's nonzero magnitudes lie within 2^29 of each other, else to */
/*      113 bits -- and the square root is taken in binary128, then rounded */
/*      to fp32 (nearest even).                                             */
/*   T3 the 16 levels are used as BF16 (round to nearest even), the matrix  */
/*      operand type; the K index is that of the level nearest to x / n,    */
/*      ties to the lower one, i.e. the number of midpoints                 */
/*      m_j = (c_j + c_{j+1}) / 2 below x / n, each comparison x > m_j n    */
/*      made exactly (binary128, where m_j and m_j n are exact).  A zero    */
/*      key (n = 0) has index 0 in every channel.  The dequantised key is   */
/*      n * c[idx], exact.                                                  */
/*   T4 V per group: zero z = bf16(min), scale s = bf16(max(max - z, 0) /  */
/*      15) (fp32 subtract and divide), code = clamp(rint((x - z) / s),    */
/*      0, 15), or 0 when s = 0; the dequantised value is                  */
/*      bf16(fma(s, code, z)), the BF16 operand of the PV product.          */
/*   T5 the query is R q rounded to BF16.                                    */
/* Cache block per (page, kv head), 2368 bytes:                             */
/*   [0, 1024)     K indices: (token t, channel c) at byte                  */
/*                 16 * (t + 16 * ((c % 32) / 8)) + 4 * (c / 32) + (c % 8)/2*/
/*   [1024, 2048)  V codes: 1024 + 16 * (c / 8 + 16 * (t / 4)) + 4 * (t % 4)*/
/*                 + (c % 8) / 2                                            */
/*   (low nibble = even channel in both)                                     */
/*   [2048, 2112)  K norms, fp32, token t at 2048 + 4 t                      */
/*   [2112, 2368)  V (s, z) BF16 pairs, s in the low half: token t, group g */
/*                 at 2112 + 16 * (4 * (t / 4) + g) + 4 * (t % 4)            */
/* ====================================================================== */
#define UQO_TQ_BLOCK 2368

static float f32_of_bits(uint32_t u) { float f; memcpy(&f, &u, 4); return f; }
static uint32_t bits_of_f32(float f) { uint32_t u; memcpy(&u, &f, 4); return u; }

/* fp32 -> nearest BF16 (ties to even), as the fp32 value it stands for. */
float uqo_bf16_rne(float x) {
    uint32_t u = bits_of_f32(x);
    if (isnan(x)) return x;
    uint32_t lsb = (u >> 16) & 1u;
    u += 0x7FFFu + lsb;
    return f32_of_bits(u & 0xFFFF0000u);
}

/* The 16 levels as BF16 and their 15 midpoints (exact in binary128). */
static void tq_tables(const float *levels, float lv[16], __float128 mid[15]) {
    for (int j = 0; j < 16; ++j) lv[j] = uqo_bf16_rne(levels[j]);
    for (int j = 0; j < 15; ++j) mid[j] = ((__float128)lv[j] + (__float128)lv[j + 1]) / 2;
}

/* Reading T2: fl32(sqrt(sum of x_i^2)). */
float uqo_tq4_norm(const float x[UQO_D]) {
    __float128 s = 0;
    for (int c = 0; c < UQO_D; ++c) s += (__float128)x[c] * (__float128)x[c];
    return (float)sqrtq(s);
}

/* Reading T3: index of the level nearest to x / n (ties to the lower). */
int uqo_tq4_index(float x, float n, const float *levels) {
    float lv[16];
    __float128 mid[15];
    tq_tables(levels, lv, mid);
    if (!(n > 0.0f)) return 0;
    int idx = 0;
    for (int j = 0; j < 15; ++j) idx += (__float128)x > mid[j] * (__float128)n;
    return idx;
}

/* Encode one token's K and V (128 channels each) per readings T1-T4. */
void uqo_tq4_encode_vector(const float *k_in, const float *v, const float *levels, uint8_t kidx[UQO_D], float *norm,
                           uint8_t vcode[UQO_D], float s_out[UQO_NGROUP], float z_out[UQO_NGROUP]) {
    float x[UQO_D];
    memcpy(x, k_in, sizeof(x));
    uqo_wht128_f32(x, 1);
    const float n = uqo_tq4_norm(x);
    *norm = n;
    for (int c = 0; c < UQO_D; ++c) kidx[c] = (uint8_t)uqo_tq4_index(x[c], n, levels);
    for (int g = 0; g < UQO_NGROUP; ++g) {
        const float *vg = v + g * UQO_GROUP;
        float mn = vg[0], mx = vg[0];
        for (int i = 1; i < UQO_GROUP; ++i) {
            if (vg[i] < mn) mn = vg[i];
            if (vg[i] > mx) mx = vg[i];
        }
        const float z = uqo_bf16_rne(mn);
        float d = mx - z;
        if (!(d > 0.0f)) d = 0.0f;
        const float s = uqo_bf16_rne(d / 15.0f);
        s_out[g] = s;
        z_out[g] = z;
        for (int i = 0; i < UQO_GROUP; ++i) {
            int code = 0;
            if (s > 0.0f) {
                float r = rintf((vg[i] - z) / s);
                code = r < 0.0f ? 0 : r > 15.0f ? 15 : (int)r;
            }
            vcode[g * UQO_GROUP + i] = (uint8_t)code;
        }
    }
}

static int tq_k_byte(int t, int c) { return 16 * (t + 16 * ((c % 32) / 8)) + 4 * (c / 32) + (c % 8) / 2; }
static int tq_v_byte(int t, int c) { return 1024 + 16 * (c / 8 + 16 * (t / 4)) + 4 * (t % 4) + (c % 8) / 2; }
static int tq_meta_byte(int t, int g) { return 2112 + 16 * (4 * (t / 4) + g) + 4 * (t % 4); }

static void put_nibble(uint8_t *b, int c, uint8_t code) {
    if (c & 1) *b = (uint8_t)((*b & 0x0F) | (code << 4));
    else *b = (uint8_t)((*b & 0xF0) | (code & 0x0F));
}
static uint8_t get_nibble(const uint8_t *b, int c) { return (c & 1) ? (uint8_t)(*b >> 4) : (uint8_t)(*b & 0x0F); }

/* Write tokens into the Ultra-TQ cache through physical slots (page * 16 +
 * offset; negative or out-of-pool slots write nothing).  k, v: rows of
 * num_kv_heads * 128 floats, token_stride floats apart.  Returns the number
 * of (token, head) vectors written. */
int64_t uqo_tq4_write(const float *k, const float *v, int64_t num_tokens, int num_kv_heads, int64_t token_stride,
                      const int64_t *slots, int64_t num_pages, const float *levels, uint8_t *cache) {
    int64_t written = 0;
    for (int64_t t = 0; t < num_tokens; ++t) {
        const int64_t slot = slots[t];
        if (slot < 0 || slot / UQO_PAGE >= num_pages) continue;
        const int64_t page = slot / UQO_PAGE;
        const int off = (int)(slot % UQO_PAGE);
        for (int h = 0; h < num_kv_heads; ++h) {
            uint8_t kidx[UQO_D], vcode[UQO_D];
            float n, s[UQO_NGROUP], z[UQO_NGROUP];
            uqo_tq4_encode_vector(k + t * token_stride + h * UQO_D, v + t * token_stride + h * UQO_D, levels, kidx, &n,
                                  vcode, s, z);
            uint8_t *blk = cache + (page * num_kv_heads + h) * UQO_TQ_BLOCK;
            for (int c = 0; c < UQO_D; ++c) {
                put_nibble(blk + tq_k_byte(off, c), c, kidx[c]);
                put_nibble(blk + tq_v_byte(off, c), c, vcode[c]);
            }
            memcpy(blk + 2048 + 4 * off, &n, 4);
            for (int g = 0; g < UQO_NGROUP; ++g) {
                uint32_t w = (bits_of_f32(s[g]) >> 16) | (bits_of_f32(z[g]) & 0xFFFF0000u);
                memcpy(blk + tq_meta_byte(off, g), &w, 4);
            }
            ++written;
        }
    }
    return written;
}

/* Read back one token's indices, codes, norm and (s, z) from the cache. */
void uqo_tq4_load(const uint8_t *cache, int num_kv_heads, int64_t page, int head, int t, uint8_t kidx[UQO_D],
                  float *norm, uint8_t vcode[UQO_D], float s[UQO_NGROUP], float z[UQO_NGROUP]) {
    const uint8_t *blk = cache + (page * num_kv_heads + head) * UQO_TQ_BLOCK;
    for (int c = 0; c < UQO_D; ++c) {
        kidx[c] = get_nibble(blk + tq_k_byte(t, c), c);
        vcode[c] = get_nibble(blk + tq_v_byte(t, c), c);
    }
    memcpy(norm, blk + 2048 + 4 * t, 4);
    for (int g = 0; g < UQO_NGROUP; ++g) {
        uint32_t w;
        memcpy(&w, blk + tq_meta_byte(t, g), 4);
        s[g] = f32_of_bits(w << 16);
        z[g] = f32_of_bits(w & 0xFFFF0000u);
    }
}

/* Dequantise one token (algorithm's Decode, reading T3/T4): K = n * c[idx]
 * (the rotated key), V = bf16(fma(s, code, z)). */
void uqo_tq4_dequant(const uint8_t *cache, int num_kv_heads, int64_t page, int head, int t, const float *levels,
                     double kout[UQO_D], double vout[UQO_D]) {
    float lv[16];
    __float128 mid[15];
    tq_tables(levels, lv, mid);
    uint8_t kidx[UQO_D], vcode[UQO_D];
    float n, s[UQO_NGROUP], z[UQO_NGROUP];
    uqo_tq4_load(cache, num_kv_heads, page, head, t, kidx, &n, vcode, s, z);
    for (int c = 0; c < UQO_D; ++c) {
        kout[c] = (double)n * (double)lv[kidx[c]];
        vout[c] = (double)uqo_bf16_rne(fmaf(s[c / UQO_GROUP], (float)vcode[c], z[c / UQO_GROUP]));
    }
}

/* Decode attention over the Ultra-TQ cache (its algorithm, Decode): the
 * query rotated and rounded to BF16 (T5), scores scale * <q, K> over the
 * dequantised rotated keys, softmax and the weighted sum of the (unrotated)
 * dequantised values, all in fp64. */
void uqo_tq4_decode_attention(const float *q, int batch, int num_q_heads, int num_kv_heads, const uint8_t *cache,
                              const int32_t *page_table, int max_pages_per_seq, const int32_t *context_lens,
                              double softmax_scale, const float *levels, double *out) {
    const int G = num_q_heads / num_kv_heads;
#pragma omp parallel for collapse(2) schedule(dynamic)
    for (int b = 0; b < batch; ++b) {
        for (int hq = 0; hq < num_q_heads; ++hq) {
            double *o = out + ((int64_t)b * num_q_heads + hq) * UQO_D;
            const int ctx = context_lens[b];
            memset(o, 0, UQO_D * sizeof(double));
            if (ctx <= 0) continue;
            float qr[UQO_D];
            memcpy(qr, q + ((int64_t)b * num_q_heads + hq) * UQO_D, sizeof(qr));
            uqo_wht128_f32(qr, 1);
            double qb[UQO_D];
            for (int c = 0; c < UQO_D; ++c) qb[c] = (double)uqo_bf16_rne(qr[c]);
            const int hk = hq / G;
            double *sc = (double *)malloc((size_t)ctx * sizeof(double));
            double mx = -INFINITY;
            double kv[UQO_D], vv[UQO_D];
            for (int j = 0; j < ctx; ++j) {
                const int64_t page = page_table[(int64_t)b * max_pages_per_seq + j / UQO_PAGE];
                uqo_tq4_dequant(cache, num_kv_heads, page, hk, j % UQO_PAGE, levels, kv, vv);
                double d = 0.0;
                for (int c = 0; c < UQO_D; ++c) d += qb[c] * kv[c];
                sc[j] = softmax_scale * d;
                if (sc[j] > mx) mx = sc[j];
            }
            double l = 0.0;
            for (int j = 0; j < ctx; ++j) {
                const int64_t page = page_table[(int64_t)b * max_pages_per_seq + j / UQO_PAGE];
                uqo_tq4_dequant(cache, num_kv_heads, page, hk, j % UQO_PAGE, levels, kv, vv);
                const double p = exp(sc[j] - mx);
                l += p;
                for (int c = 0; c < UQO_D; ++c) o[c] += p * vv[c];
            }
            for (int c = 0; c < UQO_D; ++c) o[c] /= l;
            free(sc);
        }
    }
}
