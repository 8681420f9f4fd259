/*
 * greencache.h - C ABI of the MI355X (gfx950) prefix-cached prefill path.
 *
 * GreenCache (arXiv 2505.23970) keeps the KV of earlier requests' context and
 * reuses it: when a request's context prefix is found in the cache, the
 * cached tokens' KV is joined with the new tokens' KV and both are processed
 * together, and the new tokens' KV is saved for later requests (§2.2
 * "Caching for LLM Serving", Fig. 1a, steps 1 and 2). This library is that
 * step on one GPU: it appends the new (suffix) tokens' K/V into a paged KV
 * pool and runs causal attention of the new tokens' queries over the cached
 * prefix plus the new tokens. Cache lookup, token matching, eviction and
 * sizing belong to the caller (the paper's cache manager, §5.5).
 *
 * Attention computed (the paper states no formula; textbook causal scaled
 * dot-product attention with grouped KV heads, §2.1 prefill): for new token i
 * of request r at logical position P_r + i and query head h, with
 * kvh = h / (Hq / Hkv),
 *     o = sum_{j <= P_r + i} softmax_j(scale * <q, k_j>) * v_j,
 *     lse = ln sum_{j <= P_r + i} exp(scale * <q, k_j>).
 *
 * Conventions shared by every entry point
 *   - All buffers belong to the caller. The library allocates no device or
 *     host memory and keeps no mutable global state; entry points are
 *     thread-safe. Work is enqueued on `stream` and the call returns without
 *     waiting; host arrays are only read during the call, device arrays must
 *     stay alive until the stream has run the work.
 *   - bf16 tensors are passed as pointers to IEEE bfloat16 bit patterns.
 *   - Packed new tokens: row t of q / k_new / v_new / out is new token
 *     t - cu_r of request r, where cu_r = new_lens[0] + ... + new_lens[r-1].
 *     T = sum of new_lens.
 *   - Pool layout (value pages are stored transposed so that the attention
 *     kernel reads both operands of its matrix products with 16-byte loads):
 *       k_pool  bf16 [num_blocks][num_kv_heads][page_size][head_dim]
 *       v_pool  bf16 [num_blocks][num_kv_heads][head_dim][page_size]
 *     Logical key j of request r lives in block block_tables[r][j / page_size],
 *     slot j % page_size.
 *   - Supported: head_dim 64 or 128; page_size 16; num_q_heads a multiple of
 *     num_kv_heads with num_q_heads / num_kv_heads <= 128.
 *   - Errors detectable on the host are returned before anything is enqueued
 *     and leave every buffer untouched. A block id outside [0, num_blocks) in
 *     a table entry the batch needs is not checked on the host: the kernels
 *     never access memory through such an id (append writes nothing there;
 *     attention skips the page or reads block 0 in its place), so a bad id
 *     never causes an out-of-bounds access, but the result is then undefined. Two requests appending into the same slot race.
 *     GC_ERR_HIP reports a failed launch; the HIP error is not cleared.
 *   - batch == 0 or T == 0: GC_OK, nothing is enqueued.
 */
#ifndef GREENCACHE_H
#define GREENCACHE_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum gc_status {
    GC_OK = 0,
    GC_ERR_NULL_ARG = -1,    /* a required pointer is NULL */
    GC_ERR_BAD_SHAPE = -2,   /* negative length, Hq % Hkv != 0, non-positive sizes, bad scale */
    GC_ERR_UNSUPPORTED = -3, /* head_dim not 64/128, page_size != 16, Hq/Hkv > 128, Hkv > 65535,
                                small tiles forced with Hq/Hkv > 16 */
    GC_ERR_BLOCK_TABLE = -4, /* ceil((P_r + n_r) / page_size) > max_blocks_per_seq */
    GC_ERR_WORKSPACE = -5,   /* workspace NULL or smaller than required */
    GC_ERR_HIP = -6,         /* a HIP launch or runtime call failed */
    GC_ERR_LENGTHS = -7      /* the device length arrays disagree with the host's
                                (reported by gc_prefix_prefill_plan_status) */
} gc_status;

/* Model and pool geometry. */
typedef struct gc_geometry {
    int32_t num_q_heads;        /* Hq */
    int32_t num_kv_heads;       /* Hkv */
    int32_t head_dim;           /* D */
    int32_t page_size;          /* keys per pool block (16) */
    int32_t num_blocks;         /* blocks in each pool */
    int32_t max_blocks_per_seq; /* row length of block_tables */
} gc_geometry;

/* One ragged batch of requests whose prefixes hit the cache (P_r may be 0: a
 * miss is a plain causal prefill). Host and device copies of the lengths
 * must hold the same values. */
typedef struct gc_batch {
    int32_t batch;                   /* B >= 0 */
    const int32_t* prefix_lens_host; /* [B] cached tokens already in the pool, P_r >= 0 */
    const int32_t* new_lens_host;    /* [B] new tokens, n_r >= 0 */
    const int32_t* prefix_lens_dev;  /* [B] device copy of prefix_lens_host */
    const int32_t* cu_new_lens_dev;  /* [B+1] device: 0, n_0, n_0+n_1, ..., T */
    const int32_t* block_tables_dev; /* [B][max_blocks_per_seq] device, physical block ids */
} gc_batch;

/* Tilings of the attention call (gc_plan_options.tiling). */
typedef enum gc_tiling {
    GC_TILES_AUTO = 0,    /* small tiles when every request has n_r * Hq / Hkv <= 16
                             (decode-like batches); otherwise wide or prefill tiles,
                             by the amount of work (see gc_prefix_prefill_plan) */
    GC_TILES_PREFILL = 1, /* 128 query rows x 64 keys per tile, staged through LDS */
    GC_TILES_SMALL = 2,   /* 16 query rows x 32 keys per wavefront, read straight from
                             global memory; needs Hq / Hkv <= 16 */
    GC_TILES_WIDE = 3     /* 256 query rows x 64 keys per workgroup of 8 wavefronts,
                             staged through LDS (twice the rows per copied K/V tile) */
} gc_tiling;

/* Work-split and tiling options of the attention call. Pass NULL for the defaults. */
typedef struct gc_plan_options {
    /* 0: automatic. > 0: split the keys of every query tile into chunks of this
     * many key tiles (64 keys with prefill tiles, 32 with small tiles), merged
     * by log-sum-exp. < 0: never split. */
    int32_t kv_split_tiles;
    int32_t tiling;          /* a gc_tiling value; other values: GC_ERR_BAD_SHAPE */
    int32_t reserved[6];     /* must be zero */
} gc_plan_options;

/*
 * Save the new tokens' K/V into the pool (§2.2, step 1: the processed
 * request's KV is stored for reuse). For every request r, new token i and KV
 * head h, the head_dim values of k_new[cu_r + i][h] and v_new[cu_r + i][h] are
 * copied bit for bit to slot (P_r + i) % page_size of block
 * block_tables[r][(P_r + i) / page_size]. No other pool byte changes.
 *   k_new, v_new : bf16 [T][Hkv][D], device memory or pinned host memory
 *                  (hipHostMalloc), which the kernel reads directly over PCIe
 *   k_pool, v_pool: device bf16 pools (layout above), updated in place
 * Call it before the attention call, which reads the new tokens' K/V from the
 * pool. The same call restores a cached prefix loaded back from the cache's
 * host tier (§2.2: on a hit the stored KV is brought back before the new
 * tokens are processed): pass prefix_lens = 0 and new_lens = the cached
 * lengths, with k_new / v_new pointing at the cached K/V in pinned host memory.
 */
gc_status gc_kv_append(const gc_geometry* geo, const gc_batch* batch,
                       const void* k_new, const void* v_new,
                       void* k_pool, void* v_pool, hipStream_t stream);

/*
 * Device workspace, in bytes, that the attention call needs for this batch and
 * these options (work list plus split-KV partial results). Writes *bytes.
 */
gc_status gc_prefix_prefill_workspace_size(const gc_geometry* geo, const gc_batch* batch,
                                           const gc_plan_options* opts, size_t* bytes);

/*
 * Build the attention work list in `workspace` on the device from the device
 * length arrays (one small kernel; no host-to-device copy). A plan stays valid
 * for every later gc_prefix_prefill_run with the same batch and options, so a
 * serving loop plans once per batch and runs once per layer.
 */
gc_status gc_prefix_prefill_plan(const gc_geometry* geo, const gc_batch* batch,
                                 const gc_plan_options* opts,
                                 void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * Whether the last plan written into `workspace` (by gc_prefix_prefill_plan,
 * gc_prefix_prefill_attention[_fp8] or gc_prefix_prefill_prepare[_fp8]) was
 * built from device lengths that agree with the host's. The planner checks on
 * the device that cu_new_lens_dev starts at 0, never decreases and ends at the
 * host's T, that every prefix_lens_dev entry is >= 0, that every request's
 * keys fit its block-table row, and that the work-item, merge and partial
 * counts equal those the host derived from the host lengths. When any check
 * fails the plan holds no work: a run on it enqueues kernels that write nothing
 * (out and lse keep their contents), and nothing is accessed out of bounds.
 * The check result is an int32 at byte offset 0 of the workspace (0: agree,
 * 1: disagree). This call waits for `stream` (the plan must have been enqueued
 * on it), reads that word and returns GC_OK or GC_ERR_LENGTHS; GC_ERR_NULL_ARG
 * for a NULL workspace, GC_ERR_WORKSPACE for workspace_bytes < 4, GC_ERR_HIP if
 * the copy or the wait fails. It is the one entry point that blocks the host.
 * (§2.2: the caller owns the lookup that produces the lengths; the library
 * rejects a batch whose two copies disagree, visibly.)
 */
gc_status gc_prefix_prefill_plan_status(const void* workspace, size_t workspace_bytes,
                                        hipStream_t stream);

/*
 * Attention of the new tokens over the cached prefix plus the new tokens
 * (§2.2, step 2), using a plan made by gc_prefix_prefill_plan on the same
 * stream for the same batch and options.
 *   q     : device bf16 [T][Hq][D]
 *   scale : softmax scale, finite and > 0 (callers pass 1/sqrt(D))
 *   out   : device bf16 [T][Hq][D], rounded to nearest even
 *   lse   : device fp32 [T][Hq] natural-log log-sum-exp, or NULL
 * The pools must already hold every key of every request (prefix and new).
 * The workspace also holds state that runs update (split-KV partials, and the work
 * queues of large wide-tile launches, which the plan clears and every run leaves
 * cleared): runs that share a workspace must be ordered (one stream, or waited for).
 */
gc_status gc_prefix_prefill_run(const gc_geometry* geo, const gc_batch* batch,
                                const gc_plan_options* opts,
                                const void* q, const void* k_pool, const void* v_pool,
                                float scale, void* out, float* lse,
                                void* workspace, size_t workspace_bytes, hipStream_t stream);

/* gc_prefix_prefill_plan followed by gc_prefix_prefill_run. */
gc_status gc_prefix_prefill_attention(const gc_geometry* geo, const gc_batch* batch,
                                      const gc_plan_options* opts,
                                      const void* q, const void* k_pool, const void* v_pool,
                                      float scale, void* out, float* lse,
                                      void* workspace, size_t workspace_bytes,
                                      hipStream_t stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc): gc_prefix_prefill_attention
 * without a workspace argument. The plan and the split-KV partials go to a
 * static device array of GC_NOALLOC_SCRATCH_BYTES bytes that the library holds
 * on every GPU it runs on until the process ends; this call allocates nothing
 * (no hipMalloc, hipFree or allocating library routine). Arguments, layouts,
 * results and errors are those of gc_prefix_prefill_attention, plus
 * GC_ERR_WORKSPACE (nothing enqueued) when the batch's workspace
 * (gc_prefix_prefill_workspace_size) exceeds GC_NOALLOC_SCRATCH_BYTES. Every
 * word the kernels read is written by the same call's plan first, so nothing
 * needs clearing between calls. All calls on one GPU share its array: calls
 * whose work overlaps on one GPU (two streams, or two host threads) race and
 * must be serialised by the caller; calls in one stream are ordered.
 */
#define GC_NOALLOC_SCRATCH_BYTES (64u << 20)
gc_status gc_prefix_prefill_attention_noalloc(const gc_geometry* geo, const gc_batch* batch,
                                              const gc_plan_options* opts,
                                              const void* q, const void* k_pool, const void* v_pool,
                                              float scale, void* out, float* lse, hipStream_t stream);

/*
 * gc_kv_append followed by gc_prefix_prefill_plan, as one launch: the two are
 * independent (the plan reads only the lengths), so one launch overlaps them
 * and saves a kernel boundary in a step that appends and attends once per
 * batch. Arguments, layouts and errors are those of the two calls (the pool
 * pointers are required); nothing is enqueued if any check fails. Then call
 * gc_prefix_prefill_run on the same stream.
 */
gc_status gc_prefix_prefill_prepare(const gc_geometry* geo, const gc_batch* batch,
                                    const gc_plan_options* opts, const void* k_new,
                                    const void* v_new, void* k_pool, void* v_pool,
                                    void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * gc_kv_append and gc_prefix_prefill_run fused (§2.2: the new tokens are
 * processed together with the reused prefix and their KV is saved for later
 * requests). With prefill tiles one launch does both: the attention reads every
 * key at or past P_r straight from k_new / v_new instead of the pool (so it does
 * not wait for the append, and the append's workgroups run in the same launch
 * after the attention's). With small tiles (decode-like batches), whose kernel
 * reads every key from the pool, the append is enqueued first as its own launch.
 *   q, k_new, v_new: device bf16 [T][Hq][D], [T][Hkv][D], [T][Hkv][D]
 *   k_pool, v_pool : device bf16 pools, updated in place exactly as by
 *                    gc_kv_append
 *   other arguments: as gc_prefix_prefill_run (a plan made by
 *                    gc_prefix_prefill_plan for this batch and these options
 *                    must be in the workspace)
 * Pools, out and lse are bit for bit those of gc_kv_append followed by
 * gc_prefix_prefill_run. A pool page that receives new tokens must not be read
 * as part of another request's prefix in the same batch (with the separate calls
 * such a read would see the appended tokens, here it may not). Errors as the two
 * calls, plus GC_ERR_UNSUPPORTED when a request's new rows span 2 GiB or more
 * (n_r * Hkv * D * 2 bytes > 2^31 - 1); nothing is enqueued if any check fails.
 */
gc_status gc_prefix_prefill_run_with_append(const gc_geometry* geo, const gc_batch* batch,
                                            const gc_plan_options* opts, const void* q,
                                            const void* k_new, const void* v_new,
                                            void* k_pool, void* v_pool, float scale,
                                            void* out, float* lse, void* workspace,
                                            size_t workspace_bytes, hipStream_t stream);

/*
 * 8-bit KV pools. The paper serves its 70B model with 8-bit weights (§6
 * "Experimental setup"); storing the context cache in 8 bits likewise halves
 * the memory a cached token takes, so twice the context fits a given pool, and
 * halves the bytes the memory-bound (decode-like) attention reads.
 *   Pool layout: as above with one byte per element,
 *     k_pool8  uint8 [num_blocks][num_kv_heads][page_size][head_dim]
 *     v_pool8  uint8 [num_blocks][num_kv_heads][head_dim][page_size]
 *   Each byte is an OCP 8-bit floating-point E4M3 code (sign, 4 exponent bits
 *   with bias 7, 3 mantissa bits; subnormals m/8 * 2^-6; S.1111.111 is NaN; no
 *   infinities; magnitudes up to 448) and stands for code_value * scale, with
 *   one scale for the key pool (k_scale) and one for the value pool (v_scale).
 *   Scales must be finite, > 0 and have a finite fl32(1 / scale); otherwise
 *   GC_ERR_BAD_SHAPE.
 */

/*
 * gc_kv_append into 8-bit pools: element x (bf16) of a new token's key is
 * stored as the E4M3 code nearest to v = fl32(x * fl32(1 / k_scale)) after
 * clamping v to [-448, 448], ties to the even code, -0 as 0x80 (values use
 * v_scale). A NaN input is stored as a NaN code. Slots, ordering, host/device
 * sources and errors as gc_kv_append.
 */
gc_status gc_kv_append_fp8(const gc_geometry* geo, const gc_batch* batch,
                           const void* k_new, const void* v_new, float k_scale, float v_scale,
                           void* k_pool8, void* v_pool8, hipStream_t stream);

/*
 * gc_prefix_prefill_run over 8-bit pools: the same attention with every key
 * and value element dequantised first (code value * scale). Plans, workspaces,
 * tilings and options are the bf16 ones (gc_prefix_prefill_plan and
 * gc_prefix_prefill_workspace_size serve both).
 */
gc_status gc_prefix_prefill_run_fp8(const gc_geometry* geo, const gc_batch* batch,
                                    const gc_plan_options* opts,
                                    const void* q, const void* k_pool8, const void* v_pool8,
                                    float k_scale, float v_scale, float scale, void* out,
                                    float* lse, void* workspace, size_t workspace_bytes,
                                    hipStream_t stream);

/* gc_prefix_prefill_plan followed by gc_prefix_prefill_run_fp8. */
gc_status gc_prefix_prefill_attention_fp8(const gc_geometry* geo, const gc_batch* batch,
                                          const gc_plan_options* opts,
                                          const void* q, const void* k_pool8, const void* v_pool8,
                                          float k_scale, float v_scale, float scale, void* out,
                                          float* lse, void* workspace, size_t workspace_bytes,
                                          hipStream_t stream);

/* gc_prefix_prefill_prepare over 8-bit pools (gc_kv_append_fp8 + plan, one launch). */
gc_status gc_prefix_prefill_prepare_fp8(const gc_geometry* geo, const gc_batch* batch,
                                        const gc_plan_options* opts, const void* k_new,
                                        const void* v_new, float k_scale, float v_scale,
                                        void* k_pool8, void* v_pool8, void* workspace,
                                        size_t workspace_bytes, hipStream_t stream);

/*
 * Calibration, not part of the attention path: read every byte of `buf`
 * (device memory, `bytes` a multiple of 16) once as a streaming reduction,
 * writing GC_READ_PROBE_SINK_WORDS 32-bit words to `sink` (device). Timing it
 * gives the sustained HBM read rate that the memory-bound attention cases are
 * also reported against (the nominal 8 TB/s is not reached by a read stream).
 */
#define GC_READ_PROBE_SINK_WORDS (2048 * 256)
gc_status gc_read_bandwidth_probe(const void* buf, size_t bytes, void* sink, hipStream_t stream);

/*
 * Calibration, not part of the attention path: a register-only loop of
 * independent bf16 matrix-core products (v_mfma_f32_32x32x16_bf16, 32768 flops
 * each) on every SIMD: GC_MFMA_PROBE_PRODUCTS_PER_ITERATION products per
 * iteration over the whole launch. Every operand element is 1; it writes
 * GC_MFMA_PROBE_SINK_FLOATS floats to `sink` (device), each 4096 * iterations
 * (exact while that is below 2^24). Timing it gives the sustained bf16 MFMA rate that the
 * compute-bound attention cases are also reported against (the nominal 2.5
 * PFLOP/s assumes the peak clock). iterations < 0: GC_ERR_BAD_SHAPE;
 * iterations == 0: GC_OK, nothing enqueued.
 */
#define GC_MFMA_PROBE_SINK_FLOATS (1024 * 256)
#define GC_MFMA_PROBE_PRODUCTS_PER_ITERATION (1024 * 4 * 16)
gc_status gc_mfma_peak_probe(int32_t iterations, void* sink, hipStream_t stream);

/* Static, NUL-terminated description of a status code. */
const char* gc_status_string(gc_status status);

#ifdef __cplusplus
}
#endif

#endif /* GREENCACHE_H */
