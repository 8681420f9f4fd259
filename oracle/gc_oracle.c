/*
 * gc_oracle.c - plain, slow fp64 CPU oracle for prefix-cached prefill
 * attention over a paged KV pool, and for the KV append that precedes it.
 *
 * TEST INFRASTRUCTURE. Only the test suite, the package smoke check and the
 * benchmark's CPU-baseline leg may load this library. The product path (the
 * HIP library under paper_2505_23970_amd/ and its Python binding) shares no
 * code with it and never calls it.
 *
 * What is computed, and from which passage:
 *   GreenCache, §2.2 "Caching for LLM Serving", Fig. 1a (prefix_cache): when a
 *   request's context is found in the cache, the system joins the cached
 *   tokens' KV with the new tokens' KV and processes them together; the new
 *   tokens' KV is saved for later requests (step 1), the cached KV is reused
 *   (step 2). Matching is exact on tokens (§8 Related Work, "Caching for LLM", contrasted
 *   with semantic caching), so reused KV is bit-identical to recomputed KV and
 *   the result must equal a full recomputation over prefix + new tokens.
 *   §2.1 "LLM Serving Process": serving is Transformer-based and the prefill
 *   phase processes the whole prompt. The paper never writes the attention
 *   formula, so the textbook causal scaled-dot-product attention is used (a
 *   reading, not a statement of the paper: consecutive query heads share a KV
 *   head, the cached prefix is fully visible, a new token sees itself and the
 *   new tokens before it; the scale is a caller argument): for new token i of
 *   request r (logical
 *   position P_r + i) and query head h with KV head kvh = h / (Hq / Hkv),
 *       x_j = scale * <q, k_j>            for j = 0 .. P_r + i (inclusive)
 *       m = max_j x_j,  w_j = exp(x_j - m),  l = sum_j w_j
 *       o   = sum_j (w_j / l) * v_j
 *       lse = m + ln l
 *   Every bf16 input is widened exactly to double; sums run in increasing j.
 *
 * Pool layout (the interface's definition, not the paper's; the paper cites
 * PagedAttention for the KV cache, §2.1):
 *   k_pool bf16 [num_blocks][Hkv][page][D]   (key slot `off` of a page is row off)
 *   v_pool bf16 [num_blocks][Hkv][D][page]   (value pages are stored transposed)
 *   logical key j of request r lives in block block_tables[r][j / page],
 *   slot j % page.
 *
 * 8-bit pools (the low-precision variant: the paper serves its 70B model with
 * 8-bit weights, §6 "Experimental setup"; storing the cache in 8 bits halves
 * its footprint). Each pool element is an OCP 8-bit floating-point E4M3 code
 * times one scale per pool (k_scale for keys, v_scale for values):
 *   code = sign bit, 4 exponent bits (bias 7), 3 mantissa bits; exponent field
 *   0 holds the subnormals m/8 * 2^-6; S.1111.111 is NaN; no infinities; the
 *   largest magnitude is 448.
 * Storing a bf16 value x: v = fl32(x * inv) with inv = fl32(1 / scale), then
 * the code nearest to v after clamping to [-448, 448], ties to the even code;
 * the sign bit is v's (so -0 is stored as 0x80). The attention over 8-bit
 * pools dequantises every element first (code value * scale, exact in
 * double) and then follows the formula above unchanged.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define GCO_OK 0
#define GCO_ERR_ARG (-1)
#define GCO_ERR_TABLE (-2)
#define GCO_ERR_NOMEM (-3)

/* bf16 is the upper half of an IEEE binary32; the widening is exact. */
static double widen(uint16_t b) {
    uint32_t u = ((uint32_t)b) << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

void gco_widen_bf16(int64_t n, const uint16_t* src, double* dst) {
    for (int64_t i = 0; i < n; ++i) dst[i] = widen(src[i]);
}

/* Physical block of logical key j of request r, or -1 if the table does not
 * cover it or names a block outside the pool. */
static int64_t block_of(const int32_t* block_tables, int max_blocks, int num_blocks,
                        int r, int64_t j, int page) {
    int64_t lp = j / page;
    if (lp >= max_blocks) return -1;
    int32_t blk = block_tables[(int64_t)r * max_blocks + lp];
    if (blk < 0 || blk >= num_blocks) return -1;
    return blk;
}

/* Value of an E4M3 code (NaN for S.1111.111). */
double gco_e4m3_value(uint8_t code) {
    int e = (code >> 3) & 15, m = code & 7;
    double mag;
    if (e == 15 && m == 7) return NAN;
    if (e == 0)
        mag = ldexp((double)m / 8.0, -6);
    else
        mag = ldexp(1.0 + (double)m / 8.0, e - 7);
    return (code & 0x80) ? -mag : mag;
}

/* Code stored for the fp32 value v (see the header): nearest code by brute
 * force over the 127 finite non-negative codes, ties to the even code. */
uint8_t gco_e4m3_encode(float v) {
    if (isnan(v)) return 0x7F;
    double a = fabs((double)v);
    if (a > 448.0) a = 448.0;
    int best = 0;
    double best_d = INFINITY;
    for (int c = 0; c < 127; ++c) {
        double d = fabs(gco_e4m3_value((uint8_t)c) - a);
        if (d < best_d || (d == best_d && (c & 1) == 0)) {
            best_d = d;
            best = c;
        }
    }
    return (uint8_t)(best | (signbit(v) ? 0x80 : 0));
}

/* fl32(x * inv) for a bf16 x: the exact product fits a double, so rounding it
 * to float once is the correctly rounded fp32 product. */
static float scaled32(uint16_t x, float inv) {
    return (float)(widen(x) * (double)inv);
}

void gco_quantize_e4m3(int64_t n, const uint16_t* x, float inv, uint8_t* out) {
    for (int64_t i = 0; i < n; ++i) out[i] = gco_e4m3_encode(scaled32(x[i], inv));
}

/* One key/value element as a double: bf16 pools widen exactly; 8-bit pools
 * dequantise (code value times the pool's scale). */
static double kv_elem(const void* pool, int kv8, double scale, int64_t idx) {
    if (kv8) return gco_e4m3_value(((const uint8_t*)pool)[idx]) * scale;
    return widen(((const uint16_t*)pool)[idx]);
}

/*
 * KV append (§2.2, step 1: the new tokens' KV is saved into the cache pool).
 * New token i of request r (packed row cu_r + i of k_new/v_new, where cu_r is
 * the sum of the earlier requests' new_lens) takes logical position P_r + i
 * and is copied bit for bit into its page slot. No other pool byte changes.
 * Returns GCO_ERR_TABLE, leaving the pools untouched, if any target slot is
 * not covered by the block table or names a block outside the pool.
 */
static int kv_append_core(int batch, const int32_t* prefix_lens, const int32_t* new_lens,
                          const int32_t* block_tables, int max_blocks, int num_blocks,
                          int num_kv_heads, int head_dim, int page,
                          const uint16_t* k_new, const uint16_t* v_new,
                          void* k_pool, void* v_pool, int kv8, float k_inv, float v_inv) {
    if (batch < 0 || num_kv_heads <= 0 || head_dim <= 0 || page <= 0) return GCO_ERR_ARG;
    /* check every target first so that a bad table changes nothing */
    for (int r = 0; r < batch; ++r) {
        for (int i = 0; i < new_lens[r]; ++i) {
            if (block_of(block_tables, max_blocks, num_blocks, r,
                         (int64_t)prefix_lens[r] + i, page) < 0)
                return GCO_ERR_TABLE;
        }
    }
    int64_t token = 0;
    for (int r = 0; r < batch; ++r) {
        for (int i = 0; i < new_lens[r]; ++i, ++token) {
            int64_t pos = (int64_t)prefix_lens[r] + i;
            int64_t blk = block_of(block_tables, max_blocks, num_blocks, r, pos, page);
            int64_t off = pos % page;
            for (int h = 0; h < num_kv_heads; ++h) {
                const uint16_t* ks = k_new + (token * num_kv_heads + h) * head_dim;
                const uint16_t* vs = v_new + (token * num_kv_heads + h) * head_dim;
                for (int c = 0; c < head_dim; ++c) {
                    int64_t kidx = ((blk * num_kv_heads + h) * page + off) * head_dim + c;
                    int64_t vidx = ((blk * num_kv_heads + h) * head_dim + c) * page + off;
                    if (kv8) {
                        ((uint8_t*)k_pool)[kidx] = gco_e4m3_encode(scaled32(ks[c], k_inv));
                        ((uint8_t*)v_pool)[vidx] = gco_e4m3_encode(scaled32(vs[c], v_inv));
                    } else {
                        ((uint16_t*)k_pool)[kidx] = ks[c];
                        ((uint16_t*)v_pool)[vidx] = vs[c];
                    }
                }
            }
        }
    }
    return GCO_OK;
}

int gco_kv_append(int batch, const int32_t* prefix_lens, const int32_t* new_lens,
                  const int32_t* block_tables, int max_blocks, int num_blocks,
                  int num_kv_heads, int head_dim, int page,
                  const uint16_t* k_new, const uint16_t* v_new,
                  uint16_t* k_pool, uint16_t* v_pool) {
    return kv_append_core(batch, prefix_lens, new_lens, block_tables, max_blocks, num_blocks,
                          num_kv_heads, head_dim, page, k_new, v_new, k_pool, v_pool, 0, 1.f, 1.f);
}

/* The same append into 8-bit pools: each element is quantised as in the header,
 * with k_inv = fl32(1 / k_scale) and v_inv = fl32(1 / v_scale). */
int gco_kv_append_e4m3(int batch, const int32_t* prefix_lens, const int32_t* new_lens,
                       const int32_t* block_tables, int max_blocks, int num_blocks,
                       int num_kv_heads, int head_dim, int page,
                       const uint16_t* k_new, const uint16_t* v_new, float k_inv, float v_inv,
                       uint8_t* k_pool, uint8_t* v_pool) {
    return kv_append_core(batch, prefix_lens, new_lens, block_tables, max_blocks, num_blocks,
                          num_kv_heads, head_dim, page, k_new, v_new, k_pool, v_pool, 1, k_inv, v_inv);
}

/*
 * Attention of the new tokens (§2.2, step 2; §2.1 prefill). Computes the rows
 * listed in `rows` (row = token * Hq + head, token indexing the packed new
 * tokens), or all T * Hq rows in order when rows == NULL.
 * out: double [num_rows][head_dim]; lse: double [num_rows] or NULL.
 * num_threads <= 0 leaves the OpenMP default.
 * Returns GCO_ERR_TABLE if a key the rows need is not covered by the table.
 */
static int attention_core(int batch, const int32_t* prefix_lens, const int32_t* new_lens,
                          const int32_t* block_tables, int max_blocks, int num_blocks,
                          int num_q_heads, int num_kv_heads, int head_dim, int page,
                          const uint16_t* q, const void* k_pool, const void* v_pool,
                          int kv8, double k_scale, double v_scale,
                          double scale, int64_t num_rows, const int64_t* rows,
                          double* out, double* lse, int num_threads) {
    if (batch < 0 || num_q_heads <= 0 || num_kv_heads <= 0 || head_dim <= 0 || page <= 0)
        return GCO_ERR_ARG;
    if (num_q_heads % num_kv_heads != 0) return GCO_ERR_ARG;
    const int group = num_q_heads / num_kv_heads;
    int64_t total_tokens = 0;
    for (int r = 0; r < batch; ++r) total_tokens += new_lens[r];
    if (rows == NULL) num_rows = total_tokens * num_q_heads;
    int status = GCO_OK;

#ifdef _OPENMP
    if (num_threads > 0) omp_set_num_threads(num_threads);
#pragma omp parallel for schedule(dynamic, 1)
#endif
    for (int64_t k = 0; k < num_rows; ++k) {
        int64_t row = rows ? rows[k] : k;
        int64_t token = row / num_q_heads;
        int h = (int)(row % num_q_heads);
        if (token < 0 || token >= total_tokens) {
#ifdef _OPENMP
#pragma omp atomic write
#endif
            status = GCO_ERR_ARG;
            continue;
        }
        /* which request owns this packed token, and its index inside it */
        int r = 0;
        int64_t first = 0;
        while (token >= first + new_lens[r]) {
            first += new_lens[r];
            ++r;
        }
        int64_t i = token - first;
        int kvh = h / group;
        int64_t nkeys = (int64_t)prefix_lens[r] + i + 1;  /* keys 0 .. P_r + i */

        double* qv = (double*)malloc(sizeof(double) * head_dim);
        double* x = (double*)malloc(sizeof(double) * nkeys);
        if (!qv || !x) {
            free(qv);
            free(x);
#ifdef _OPENMP
#pragma omp atomic write
#endif
            status = GCO_ERR_NOMEM;
            continue;
        }
        for (int c = 0; c < head_dim; ++c)
            qv[c] = widen(q[(token * num_q_heads + h) * head_dim + c]);

        int bad = 0;
        for (int64_t j = 0; j < nkeys; ++j) {
            int64_t blk = block_of(block_tables, max_blocks, num_blocks, r, j, page);
            if (blk < 0) { bad = 1; break; }
            int64_t krow = ((blk * num_kv_heads + kvh) * page + j % page) * head_dim;
            double dot = 0.0;
            for (int c = 0; c < head_dim; ++c) dot += qv[c] * kv_elem(k_pool, kv8, k_scale, krow + c);
            x[j] = scale * dot;
        }
        if (bad) {
            free(qv);
            free(x);
#ifdef _OPENMP
#pragma omp atomic write
#endif
            status = GCO_ERR_TABLE;
            continue;
        }
        double m = x[0];
        for (int64_t j = 1; j < nkeys; ++j)
            if (x[j] > m) m = x[j];
        double l = 0.0;
        for (int64_t j = 0; j < nkeys; ++j) {
            x[j] = exp(x[j] - m);  /* x now holds the weights w_j */
            l += x[j];
        }
        double* o = out + k * head_dim;
        for (int c = 0; c < head_dim; ++c) o[c] = 0.0;
        for (int64_t j = 0; j < nkeys; ++j) {
            int64_t blk = block_of(block_tables, max_blocks, num_blocks, r, j, page);
            double p = x[j] / l;
            for (int c = 0; c < head_dim; ++c)
                o[c] += p * kv_elem(v_pool, kv8, v_scale, ((blk * num_kv_heads + kvh) * head_dim + c) * page + j % page);
        }
        if (lse) lse[k] = m + log(l);
        free(qv);
        free(x);
    }
    return status;
}

int gco_attention(int batch, const int32_t* prefix_lens, const int32_t* new_lens,
                  const int32_t* block_tables, int max_blocks, int num_blocks,
                  int num_q_heads, int num_kv_heads, int head_dim, int page,
                  const uint16_t* q, const uint16_t* k_pool, const uint16_t* v_pool,
                  double scale, int64_t num_rows, const int64_t* rows,
                  double* out, double* lse, int num_threads) {
    return attention_core(batch, prefix_lens, new_lens, block_tables, max_blocks, num_blocks,
                          num_q_heads, num_kv_heads, head_dim, page, q, k_pool, v_pool, 0, 1.0, 1.0,
                          scale, num_rows, rows, out, lse, num_threads);
}

/* Attention over 8-bit pools (dequantised first, see the header). */
int gco_attention_e4m3(int batch, const int32_t* prefix_lens, const int32_t* new_lens,
                       const int32_t* block_tables, int max_blocks, int num_blocks,
                       int num_q_heads, int num_kv_heads, int head_dim, int page,
                       const uint16_t* q, const uint8_t* k_pool, const uint8_t* v_pool,
                       double k_scale, double v_scale,
                       double scale, int64_t num_rows, const int64_t* rows,
                       double* out, double* lse, int num_threads) {
    return attention_core(batch, prefix_lens, new_lens, block_tables, max_blocks, num_blocks,
                          num_q_heads, num_kv_heads, head_dim, page, q, k_pool, v_pool, 1, k_scale,
                          v_scale, scale, num_rows, rows, out, lse, num_threads);
}

/* Number of OpenMP threads a parallel region would use (1 without OpenMP). */
int gco_max_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
