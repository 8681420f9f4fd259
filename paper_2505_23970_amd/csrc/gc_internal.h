// Internal declarations shared by the host library and the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gc {

// Attention tiling, prefill path: a workgroup of 4 wavefronts owns 128 query
// rows (query heads of one KV head stacked over consecutive new tokens) and
// walks the request's keys in tiles of 64 (four 16-key pool pages).
constexpr int kRowsPerWave = 32;
constexpr int kWaves = 4;
constexpr int kBlockM = kRowsPerWave * kWaves;  // 128
constexpr int kBlockN = 64;
// Small-tile (decode) path: one wavefront owns 16 query rows and walks the keys
// in tiles of 32 (two pages), straight from global memory.
constexpr int kDecM = 16;
constexpr int kDecN = 32;
constexpr int kDecWaves = 4;                    // independent wavefronts per workgroup
constexpr int kPage = 16;
constexpr int kAttnThreads = kWaves * 64;
// Wide prefill tiles: 8 wavefronts, 256 query rows per work item (one workgroup
// per CU; every K/V tile copied into LDS feeds twice the rows).
constexpr int kWideWaves = 8;
constexpr int kWideM = kRowsPerWave * kWideWaves;  // 256
constexpr int kPlanThreads = 256;
constexpr int kAppendThreads = 256;
constexpr int kCostBuckets = 2048;  // counting-sort buckets of the work list (cost in tiles)
constexpr int kCombineThreads = 256;  // threads per split-merge workgroup
constexpr int kPlanLdsBatch = 512;    // batches up to this size are planned from LDS copies
constexpr int kProbeBlocks = 2048;    // read-probe grid
constexpr int kProbeThreads = 256;
constexpr int kMfmaProbeBlocks = 1024;   // matrix-core probe grid: four workgroups per CU
constexpr int kMfmaProbeChains = 4;      // independent accumulators per wavefront
constexpr int kMfmaProbePerChain = 4;    // products per accumulator per iteration

// One attention work item: query tile [q0, q0 + tq) of request r against key
// tiles [kt_begin, kt_end). part >= 0 marks a split item whose normalised
// partial output goes to partial slot `part`; -1 writes the output directly.
// r < 0 marks an empty item. P, cu and n repeat the request's prefix length,
// first new row and new-token count, so that one load gives all of an item's
// lengths.
struct WorkItem {
    int32_t r, q0, kt_begin, kt_end, part, P, cu, n;
};

// One query tile whose keys were split: partial slots [part_base, part_base + ns).
struct CombineItem {
    int32_t r, q0, part_base, ns;
};

// ---------------------------------------------------------------- plan math
// Used by the host (grid sizes, workspace) and the planner kernel (the list
// itself); both must agree exactly.

__host__ __device__ inline int ceil_div(int a, int b) { return (a + b - 1) / b; }
__host__ __device__ inline int64_t ceil_div64(int64_t a, int64_t b) { return (a + b - 1) / b; }

// new tokens per query tile of block_m rows for a GQA group of g query heads per KV head
__host__ __device__ inline int tokens_per_tile(int group, int block_m) { return block_m / group; }

__host__ __device__ inline int key_tiles(int prefix, int q0, int ntok, int block_n) {
    return ceil_div(prefix + q0 + ntok, block_n);
}

// number of key chunks of a query tile with kt key tiles; chunk <= 0 means never split
__host__ __device__ inline int num_splits(int kt, int chunk) {
    return (chunk <= 0 || kt <= chunk) ? 1 : ceil_div(kt, chunk);
}

// first key tile of chunk s out of ns (balanced; every chunk non-empty when ns <= kt)
__host__ __device__ inline int split_begin(int s, int kt, int ns) {
    return (int)(((int64_t)s * kt) / ns);
}

// Pool pages that receive new tokens over the batch (the append grid), from the
// host lengths: pages P_r / 16 .. (P_r + n_r - 1) / 16 of every request with n_r > 0.
inline int64_t append_pages_host(const int32_t* prefix, const int32_t* n, int batch) {
    int64_t u = 0;
    for (int r = 0; r < batch; ++r)
        if (n[r] > 0) u += ((int64_t)prefix[r] + n[r] + kPage - 1) / kPage - prefix[r] / kPage;
    return u;
}

struct RequestCounts {
    int items;     // work items of this request (per KV head)
    int combines;  // query tiles that were split
    int partials;  // partial slots (per KV head)
};

__host__ __device__ inline RequestCounts request_counts(int prefix, int n, int tq, int chunk, int block_n) {
    RequestCounts c{0, 0, 0};
    for (int q0 = 0; q0 < n; q0 += tq) {
        int ntok = n - q0 < tq ? n - q0 : tq;
        int ns = num_splits(key_tiles(prefix, q0, ntok, block_n), chunk);
        c.items += ns;
        if (ns > 1) {
            c.combines += 1;
            c.partials += ns;
        }
    }
    return c;
}

// ---------------------------------------------------------------- workspace
constexpr size_t kStatusOffset = 0;  // byte offset of the planner's status word in the workspace
// Work queues of the resident attention launch: kQueues ticket counters and one exit
// counter (int32) in the workspace's leading 256-byte block, zeroed by the planner and
// left at zero by every launch that uses them.
constexpr size_t kQueueOffset = 64;
constexpr int kQueues = 8;  // one per XCD

struct WorkspaceLayout {
    size_t items_off, combine_off, scratch_off, part_lse_off, part_o_off, status_off, queue_off, total;
};

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

inline WorkspaceLayout workspace_layout(int batch, int64_t items, int64_t combines,
                                        int64_t partials, int num_kv_heads, int head_dim, int block_m) {
    WorkspaceLayout w{};
    size_t off = kStatusOffset;
    w.status_off = off;
    w.queue_off = off + kQueueOffset;
    off = align_up(off + 256, 256);
    w.items_off = off;
    off = align_up(off + sizeof(WorkItem) * (size_t)(items > 0 ? items : 1), 256);
    w.combine_off = off;
    off = align_up(off + sizeof(CombineItem) * (size_t)(combines > 0 ? combines : 1), 256);
    w.scratch_off = off;  // 3 int32 per request + 1, then the unsorted work list
    off = align_up(off + sizeof(int32_t) * 3 * (size_t)(batch + 1), 256);
    off = align_up(off + sizeof(WorkItem) * (size_t)(items > 0 ? items : 1), 256);
    w.part_lse_off = off;
    off = align_up(off + sizeof(float) * (size_t)partials * num_kv_heads * block_m, 256);
    w.part_o_off = off;
    off = align_up(off + sizeof(float) * (size_t)partials * num_kv_heads * block_m * head_dim, 256);
    w.total = off;
    return w;
}

// ---------------------------------------------------------------- kernel launch arguments
struct AppendArgs {
    const uint16_t* k_new;
    const uint16_t* v_new;
    void* k_pool;        // bf16 elements, or E4M3 codes for 8-bit pools
    void* v_pool;
    const int32_t* prefix_lens;
    const int32_t* cu_new_lens;
    const int32_t* block_tables;
    int32_t batch, total_tokens, num_kv_heads, num_blocks, max_blocks;
    int32_t total_pages;  // pool pages that receive new tokens (host count; the append grid)
    float k_inv, v_inv;  // 8-bit pools: fl32(1 / scale) of each pool
};

struct PlanArgs {
    const int32_t* prefix_lens;
    const int32_t* cu_new_lens;
    int32_t* scratch;         // 3 * (batch + 1) int32
    WorkItem* unsorted;       // [items]
    WorkItem* items;          // [items], in launch order (see group_cost)
    CombineItem* combines;    // [combines]
    int32_t* status;          // status[0] = 0 when the device lengths matched the host's
    int32_t* queues;          // [kQueues + 1] work-queue counters, zeroed here
    int32_t batch, tq, chunk, block_n;
    int32_t expect_items, expect_combines, expect_partials;
    int32_t total_tokens;     // the host's T (= cu_new_lens[batch] on the device)
    int32_t max_blocks;       // row length of the block tables
    // Items of at least group_cost key tiles are sorted by their request's key
    // tiles (so the items of one request stay together), lighter ones by their own
    // cost; kCostBuckets gives the plain cost order.
    int32_t group_cost;
};

struct AttnArgs {
    const uint16_t* q;
    const uint16_t* k_pool;
    const uint16_t* v_pool;
    uint16_t* out;
    float* lse;          // may be null
    float* part_o;       // [partials][Hkv][block_m][D]
    float* part_lse;     // [partials][Hkv][block_m]
    const int32_t* prefix_lens;
    const int32_t* cu_new_lens;
    const int32_t* block_tables;
    const WorkItem* items;
    int32_t* queues;     // resident launch: [kQueues] ticket counters, then the exit counter
    int32_t num_q_heads, num_kv_heads, group, tq;
    int32_t num_blocks, max_blocks;
    float scale_log2;    // softmax scale * log2(e) (times the key scale for 8-bit pools)
    float v_scale;       // value scale of 8-bit pools, 1 for bf16 pools
    // Append fused into the launch: keys at or past a request's prefix length are read
    // from the new tokens' arrays ([T][Hkv][D]) instead of the pool, and each work item
    // writes its own tokens' keys and values into the pools (k_dst / v_dst, the same
    // memory as k_pool / v_pool). Null otherwise.
    const uint16_t* k_new;
    const uint16_t* v_new;
    uint16_t* k_dst;
    uint16_t* v_dst;
};

struct CombineArgs {
    uint16_t* out;
    float* lse;
    const float* part_o;
    const float* part_lse;
    const int32_t* prefix_lens;
    const int32_t* cu_new_lens;
    const CombineItem* combines;
    int32_t num_q_heads, num_kv_heads, group, tq;
    int32_t batch, num_partials, block_m;
};

hipError_t launch_append(const AppendArgs& a, int head_dim, bool fp8, hipStream_t s);
hipError_t launch_plan(const PlanArgs& a, hipStream_t s);
// append (AppendArgs) and plan (PlanArgs) in one launch
hipError_t launch_prepare(const AppendArgs& aa, const PlanArgs& pa, int head_dim, bool fp8, hipStream_t s);
// resident > 0 (wide tiles only): that many resident workgroups take
// the items from the work queues instead of one workgroup per item
hipError_t launch_attention(const AttnArgs& a, int head_dim, int64_t num_items, bool wide, bool fp8,
                            int resident, hipStream_t s);
// the same over 8-bit pools (launch_attention forwards fp8 launches here)
hipError_t launch_attention_fp8(const AttnArgs& a, int head_dim, int64_t num_items, bool wide, int resident,
                                hipStream_t s);
// attention with the KV append fused in (AttnArgs with k_new, v_new, k_dst, v_dst
// set); prefill tiles over bf16 pools
hipError_t launch_attention_append(const AttnArgs& a, int head_dim, int64_t num_items, bool wide,
                                   hipStream_t s);
hipError_t launch_attention_small(const AttnArgs& a, int head_dim, int64_t num_items, bool fp8,
                                  hipStream_t s);
hipError_t launch_read_probe(const void* buf, size_t bytes, uint32_t* sink, hipStream_t s);
hipError_t launch_mfma_probe(int iterations, float* sink, hipStream_t s);
hipError_t launch_combine(const CombineArgs& a, int head_dim, int64_t num_combines, hipStream_t s);

}  // namespace gc
