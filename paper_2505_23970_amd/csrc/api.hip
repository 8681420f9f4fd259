// Host side of the C ABI declared in include/greencache.h: argument checks,
// work-split policy, workspace layout and kernel launches. Every check runs
// before the first HIP call, so invalid calls enqueue nothing.
#include <cmath>
#include <cstdint>
#include <mutex>

#include "gc_internal.h"
#include "greencache.h"

namespace {

using gc::RequestCounts;


struct Shape {
    int64_t total_tokens = 0;
    int group = 1;
    bool small = false;          // small-tile (decode) path
    bool wide = false;           // 8-wavefront prefill tiles
    int block_m = gc::kBlockM;   // query rows per tile
    int block_n = gc::kBlockN;   // keys per tile
    int tq = 1;                  // new tokens per query tile
};

struct Plan {
    int chunk = 0;  // key tiles per chunk, 0 = no split
    int64_t items = 0, combines = 0, partials = 0;
    int group_cost = gc::kCostBuckets;  // work-list order (gc::PlanArgs)
    gc::WorkspaceLayout layout{};
};

gc_status check_common(const gc_geometry* geo, const gc_batch* b, Shape* sh) {
    if (geo == nullptr || b == nullptr) return GC_ERR_NULL_ARG;
    if (b->batch < 0) return GC_ERR_BAD_SHAPE;
    if (geo->num_q_heads <= 0 || geo->num_kv_heads <= 0 || geo->head_dim <= 0 ||
        geo->page_size <= 0 || geo->num_blocks < 0 || geo->max_blocks_per_seq < 0)
        return GC_ERR_BAD_SHAPE;
    if (geo->num_q_heads % geo->num_kv_heads != 0) return GC_ERR_BAD_SHAPE;
    const int group = geo->num_q_heads / geo->num_kv_heads;
    if (group > gc::kBlockM) return GC_ERR_UNSUPPORTED;
    if (geo->num_kv_heads > 65535) return GC_ERR_UNSUPPORTED;  // append grid dimension
    if (geo->head_dim != 64 && geo->head_dim != 128) return GC_ERR_UNSUPPORTED;
    if (geo->page_size != gc::kPage) return GC_ERR_UNSUPPORTED;
    sh->group = group;
    sh->tq = gc::tokens_per_tile(group, sh->block_m);
    sh->total_tokens = 0;
    if (b->batch == 0) return GC_OK;
    if (b->prefix_lens_host == nullptr || b->new_lens_host == nullptr) return GC_ERR_NULL_ARG;
    int64_t total = 0;
    for (int r = 0; r < b->batch; ++r) {
        const int64_t P = b->prefix_lens_host[r], n = b->new_lens_host[r];
        if (P < 0 || n < 0) return GC_ERR_BAD_SHAPE;
        if (P + n > (int64_t)INT32_MAX - gc::kBlockN) return GC_ERR_BAD_SHAPE;
        total += n;
    }
    if (total > (int64_t)INT32_MAX) return GC_ERR_BAD_SHAPE;
    for (int r = 0; r < b->batch; ++r) {
        const int64_t P = b->prefix_lens_host[r], n = b->new_lens_host[r];
        if (n > 0 && (P + n + gc::kPage - 1) / gc::kPage > geo->max_blocks_per_seq)
            return GC_ERR_BLOCK_TABLE;
    }
    sh->total_tokens = total;
    // the append grid: one workgroup per (page receiving new tokens, KV head), plus
    // the planner's in the combined launch
    if (gc::append_pages_host(b->prefix_lens_host, b->new_lens_host, b->batch) * geo->num_kv_heads >=
        (int64_t)INT32_MAX)
        return GC_ERR_UNSUPPORTED;
    if (total > 0) {
        if (geo->num_blocks <= 0) return GC_ERR_BAD_SHAPE;
        if (b->prefix_lens_dev == nullptr || b->cu_new_lens_dev == nullptr ||
            b->block_tables_dev == nullptr)
            return GC_ERR_NULL_ARG;
    }
    return GC_OK;
}

gc_status check_options(const gc_plan_options* o) {
    if (o == nullptr) return GC_OK;
    if (o->tiling != GC_TILES_AUTO && o->tiling != GC_TILES_PREFILL && o->tiling != GC_TILES_SMALL &&
        o->tiling != GC_TILES_WIDE)
        return GC_ERR_BAD_SHAPE;
    for (int i = 0; i < 6; ++i)
        if (o->reserved[i] != 0) return GC_ERR_BAD_SHAPE;
    return GC_OK;
}

// Tiling: small tiles (one wavefront per 16 query rows, keys read straight from
// global memory) when every request's new tokens fit one such tile, which is the
// decode case. Otherwise LDS-staged prefill tiles: wide ones (256 rows, 8
// wavefronts, one workgroup per CU) when they would be at least 85 % full and
// their count is not between one and two per CU (whole units there would leave
// the last round of workgroups mostly idle, and below one per CU the keys are
// split into equal chunks); 128-row tiles otherwise.
int device_cus();

gc_status choose_tiling(const gc_batch* b, const gc_plan_options* o, int num_kv_heads, Shape* sh) {
    const int want = o == nullptr ? GC_TILES_AUTO : o->tiling;
    bool small = false, wide = false;
    if (want == GC_TILES_SMALL) {
        if (sh->group > gc::kDecM) return GC_ERR_UNSUPPORTED;
        small = true;
    } else if (want == GC_TILES_WIDE) {
        wide = true;
    } else if (want == GC_TILES_AUTO) {
        if (sh->group <= gc::kDecM) {
            small = true;
            for (int r = 0; r < b->batch && small; ++r)
                small = (int64_t)b->new_lens_host[r] * sh->group <= gc::kDecM;
        }
        if (!small) {
            const int tq = gc::tokens_per_tile(sh->group, gc::kWideM);
            int64_t units = 0, rows = 0;
            for (int r = 0; r < b->batch; ++r) {
                units += (b->new_lens_host[r] + tq - 1) / tq;
                rows += (int64_t)b->new_lens_host[r] * sh->group;
            }
            const int64_t cus = device_cus();
            const int64_t grid = units * num_kv_heads;
            wide = rows * 100 >= units * gc::kWideM * 85 && !(grid > cus && grid < 2 * cus);
        }
    }
    sh->small = small;
    sh->wide = wide;
    sh->block_m = small ? gc::kDecM : (wide ? gc::kWideM : gc::kBlockM);
    sh->block_n = small ? gc::kDecN : gc::kBlockN;
    sh->tq = gc::tokens_per_tile(sh->group, sh->block_m);
    return GC_OK;
}

// Compute units of the current device (cached per device id).
int device_cus() {
    static std::mutex mu;
    static int cache[64] = {0};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0) return 256;
    if (dev < 64) {
        std::lock_guard<std::mutex> g(mu);
        if (cache[dev] > 0) return cache[dev];
    }
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
        cus = 256;
    if (dev < 64) {
        std::lock_guard<std::mutex> g(mu);
        cache[dev] = cus;
    }
    return cus;
}

// Split policy: keep whole query tiles when there are at least as many work
// items as resident slots (per compute unit: two 128-row workgroups, one wide
// workgroup, or four small-tile wavefronts); otherwise cut the keys into chunks
// (at least 512 keys, 1024 for small tiles, whose wavefronts each stream their
// own K/V) so that the launch fills those slots.
int64_t resident_slots(const Shape& sh) { return (sh.small ? 4LL : (sh.wide ? 1LL : 2LL)) * device_cus(); }

int choose_chunk(const gc_geometry* geo, const gc_batch* b, const Shape& sh,
                 const gc_plan_options* o) {
    if (o != nullptr && o->kv_split_tiles != 0) return o->kv_split_tiles > 0 ? o->kv_split_tiles : 0;
    int64_t units = 0, tiles = 0;
    for (int r = 0; r < b->batch; ++r) {
        const int P = b->prefix_lens_host[r], n = b->new_lens_host[r];
        for (int q0 = 0; q0 < n; q0 += sh.tq) {
            const int ntok = n - q0 < sh.tq ? n - q0 : sh.tq;
            units += 1;
            tiles += gc::key_tiles(P, q0, ntok, sh.block_n);
        }
    }
    units *= geo->num_kv_heads;
    tiles *= geo->num_kv_heads;
    const int64_t target = resident_slots(sh);
    if (units >= target || units == 0) return 0;
    int64_t chunk = (tiles + target - 1) / target;
    const int min_keys = sh.small ? 1024 : 512;
    if (chunk < min_keys / sh.block_n) chunk = min_keys / sh.block_n;
    return chunk > INT32_MAX ? 0 : (int)chunk;
}

// Work-list order. Items run in list order, and a list in strict cost order,
// heaviest first, ends on its lightest items (longest-processing-time order).
// Only the end needs that order, though: before it the items are sorted by the
// length of their request instead, so that a request's query tiles, which read
// nearly the same keys, run side by side and share the K/V tiles in L2. In cost
// order the tiles of a long miss (one of every cost from 1 up) are spread over the
// whole launch and each fetches the same K/V again. The lightest items, two rounds
// of the resident slots, keep the strict order: items of fewer than group_cost
// key tiles; a list no longer than that is not grouped at all.
void choose_order(const gc_geometry* geo, const gc_batch* b, const Shape& sh, Plan* pl) {
    pl->group_cost = gc::kCostBuckets;
    const int64_t tail = (2 * resident_slots(sh) + geo->num_kv_heads - 1) / geo->num_kv_heads;  // items per KV head
    if (pl->items <= tail) return;
    int64_t hist[gc::kCostBuckets] = {};  // items per cost (clamped like the planner's buckets)
    for (int r = 0; r < b->batch; ++r) {
        const int P = b->prefix_lens_host[r], n = b->new_lens_host[r];
        for (int q0 = 0; q0 < n; q0 += sh.tq) {
            const int ntok = n - q0 < sh.tq ? n - q0 : sh.tq;
            const int kt = gc::key_tiles(P, q0, ntok, sh.block_n);
            const int ns = gc::num_splits(kt, pl->chunk);
            const int lo = kt / ns, n_hi = kt - lo * ns;
            hist[lo < gc::kCostBuckets - 1 ? lo : gc::kCostBuckets - 1] += ns - n_hi;
            if (n_hi > 0) hist[lo + 1 < gc::kCostBuckets - 1 ? lo + 1 : gc::kCostBuckets - 1] += n_hi;
        }
    }
    int64_t below = 0;
    int c = 0;
    while (c < gc::kCostBuckets && below < tail) below += hist[c++];
    pl->group_cost = c;  // the items of cost < c make up the tail
}

gc_status make_plan(const gc_geometry* geo, const gc_batch* b, const Shape& sh,
                    const gc_plan_options* o, Plan* pl) {
    pl->chunk = choose_chunk(geo, b, sh, o);
    pl->items = pl->combines = pl->partials = 0;
    for (int r = 0; r < b->batch; ++r) {
        const RequestCounts c = gc::request_counts(b->prefix_lens_host[r], b->new_lens_host[r], sh.tq,
                                                   pl->chunk, sh.block_n);
        pl->items += c.items;
        pl->combines += c.combines;
        pl->partials += c.partials;
    }
    if (pl->items > (int64_t)INT32_MAX / geo->num_kv_heads) return GC_ERR_BAD_SHAPE;
    pl->layout = gc::workspace_layout(b->batch, pl->items, pl->combines, pl->partials,
                                      geo->num_kv_heads, geo->head_dim, sh.block_m);
    choose_order(geo, b, sh, pl);
    return GC_OK;
}

template <typename T>
T* at(void* ws, size_t off) {
    return reinterpret_cast<T*>(static_cast<char*>(ws) + off);
}

gc_status plan_checked(const gc_geometry* geo, const gc_batch* b, const gc_plan_options* o,
                       Shape* sh, Plan* pl) {
    gc_status st = check_common(geo, b, sh);
    if (st != GC_OK) return st;
    st = check_options(o);
    if (st != GC_OK) return st;
    st = choose_tiling(b, o, geo->num_kv_heads, sh);
    if (st != GC_OK) return st;
    if (sh->total_tokens == 0) return GC_OK;
    return make_plan(geo, b, *sh, o, pl);
}

gc::PlanArgs plan_args(const gc_geometry* geo, const gc_batch* b, const Shape& sh, const Plan& pl, void* ws) {
    gc::PlanArgs a{};
    a.prefix_lens = b->prefix_lens_dev;
    a.cu_new_lens = b->cu_new_lens_dev;
    a.scratch = at<int32_t>(ws, pl.layout.scratch_off);
    a.unsorted = reinterpret_cast<gc::WorkItem*>(
        at<char>(ws, pl.layout.scratch_off) +
        gc::align_up(sizeof(int32_t) * 3 * (size_t)(b->batch + 1), 256));
    a.items = at<gc::WorkItem>(ws, pl.layout.items_off);
    a.combines = at<gc::CombineItem>(ws, pl.layout.combine_off);
    a.status = at<int32_t>(ws, pl.layout.status_off);
    a.queues = at<int32_t>(ws, pl.layout.queue_off);
    a.batch = b->batch;
    a.tq = sh.tq;
    a.chunk = pl.chunk;
    a.block_n = sh.block_n;
    a.expect_items = (int32_t)pl.items;
    a.expect_combines = (int32_t)pl.combines;
    a.expect_partials = (int32_t)pl.partials;
    a.total_tokens = (int32_t)sh.total_tokens;
    a.max_blocks = geo->max_blocks_per_seq;
    a.group_cost = pl.group_cost;
    return a;
}

gc_status enqueue_plan(const gc_geometry* geo, const gc_batch* b, const Shape& sh, const Plan& pl,
                       void* ws, hipStream_t stream) {
    return gc::launch_plan(plan_args(geo, b, sh, pl, ws), stream) == hipSuccess ? GC_OK : GC_ERR_HIP;
}

// Wide tiles with at least two rounds of work items per compute unit run as a
// resident launch (one workgroup per CU taking items from per-XCD queues;
// attention_kernels.h): it removes the dispatch gaps between items and lets the XCDs that
// finish first take the last items of the others. A single round has nothing to
// balance. 0: the regular launch.
int resident_workgroups(const gc_geometry* geo, const Shape& sh, const Plan& pl) {
    if (!sh.wide) return 0;
    const int cus = device_cus();
    if (cus % gc::kQueues != 0) return 0;
    return pl.items * geo->num_kv_heads >= 2LL * cus ? cus : 0;
}

// Pools of bf16 elements (fp8 false, scales 1) or of E4M3 codes with one scale each.
struct PoolKind {
    bool fp8 = false;
    float k_scale = 1.f, v_scale = 1.f;
};

gc_status enqueue_run(const gc_geometry* geo, const gc_batch* b, const Shape& sh, const Plan& pl,
                      const void* q, const void* k_pool, const void* v_pool, float scale,
                      void* out, float* lse, void* ws, hipStream_t stream, const PoolKind& pk = PoolKind{},
                      const gc::AppendArgs* fused = nullptr) {
    gc::AttnArgs a{};
    a.q = static_cast<const uint16_t*>(q);
    a.k_pool = static_cast<const uint16_t*>(k_pool);
    a.v_pool = static_cast<const uint16_t*>(v_pool);
    a.out = static_cast<uint16_t*>(out);
    a.lse = lse;
    a.part_o = at<float>(ws, pl.layout.part_o_off);
    a.part_lse = at<float>(ws, pl.layout.part_lse_off);
    a.prefix_lens = b->prefix_lens_dev;
    a.cu_new_lens = b->cu_new_lens_dev;
    a.block_tables = b->block_tables_dev;
    a.items = at<gc::WorkItem>(ws, pl.layout.items_off);
    a.queues = at<int32_t>(ws, pl.layout.queue_off);
    a.num_q_heads = geo->num_q_heads;
    a.num_kv_heads = geo->num_kv_heads;
    a.group = sh.group;
    a.tq = sh.tq;
    a.num_blocks = geo->num_blocks;
    a.max_blocks = geo->max_blocks_per_seq;
    a.scale_log2 = (float)((double)scale * (double)pk.k_scale * 1.4426950408889634074);
    a.v_scale = pk.v_scale;
    hipError_t e;
    if (fused != nullptr) {  // prefill tiles over bf16 pools only
        a.k_new = fused->k_new;
        a.v_new = fused->v_new;
        a.k_dst = static_cast<uint16_t*>(fused->k_pool);
        a.v_dst = static_cast<uint16_t*>(fused->v_pool);
        e = gc::launch_attention_append(a, geo->head_dim, pl.items, sh.wide, stream);
    } else {
        e = sh.small ? gc::launch_attention_small(a, geo->head_dim, pl.items, pk.fp8, stream)
                     : gc::launch_attention(a, geo->head_dim, pl.items, sh.wide, pk.fp8,
                                            resident_workgroups(geo, sh, pl), stream);
    }
    if (e != hipSuccess) return GC_ERR_HIP;
    if (pl.combines > 0) {
        gc::CombineArgs c{};
        c.out = a.out;
        c.lse = lse;
        c.part_o = a.part_o;
        c.part_lse = a.part_lse;
        c.prefix_lens = b->prefix_lens_dev;
        c.cu_new_lens = b->cu_new_lens_dev;
        c.combines = at<gc::CombineItem>(ws, pl.layout.combine_off);
        c.num_q_heads = geo->num_q_heads;
        c.num_kv_heads = geo->num_kv_heads;
        c.group = sh.group;
        c.tq = sh.tq;
        c.batch = b->batch;
        c.num_partials = (int32_t)pl.partials;
        c.block_m = sh.block_m;
        if (gc::launch_combine(c, geo->head_dim, pl.combines, stream) != hipSuccess) return GC_ERR_HIP;
    }
    return GC_OK;
}

gc_status check_run_args(const void* q, const void* k_pool, const void* v_pool, float scale,
                         void* out) {
    if (q == nullptr || k_pool == nullptr || v_pool == nullptr || out == nullptr)
        return GC_ERR_NULL_ARG;
    if (!std::isfinite(scale) || !(scale > 0.f)) return GC_ERR_BAD_SHAPE;
    return GC_OK;
}

gc_status check_pool_scales(float k_scale, float v_scale) {
    if (!std::isfinite(k_scale) || !(k_scale > 0.f) || !std::isfinite(v_scale) || !(v_scale > 0.f))
        return GC_ERR_BAD_SHAPE;
    // the append multiplies by fl32(1 / scale), which must be finite as well
    if (!std::isfinite(1.f / k_scale) || !std::isfinite(1.f / v_scale)) return GC_ERR_BAD_SHAPE;
    return GC_OK;
}

gc_status check_workspace(const Plan& pl, const void* ws, size_t bytes) {
    if (ws == nullptr || bytes < pl.layout.total) return GC_ERR_WORKSPACE;
    return GC_OK;
}

gc::AppendArgs append_args(const gc_geometry* geo, const gc_batch* batch, const Shape& sh,
                           const void* k_new, const void* v_new, void* k_pool, void* v_pool,
                           const PoolKind& pk) {
    gc::AppendArgs a{};
    a.k_new = static_cast<const uint16_t*>(k_new);
    a.v_new = static_cast<const uint16_t*>(v_new);
    a.k_pool = k_pool;
    a.v_pool = v_pool;
    a.prefix_lens = batch->prefix_lens_dev;
    a.cu_new_lens = batch->cu_new_lens_dev;
    a.block_tables = batch->block_tables_dev;
    a.batch = batch->batch;
    a.total_tokens = (int32_t)sh.total_tokens;
    a.num_kv_heads = geo->num_kv_heads;
    a.num_blocks = geo->num_blocks;
    a.max_blocks = geo->max_blocks_per_seq;
    a.total_pages = (int32_t)gc::append_pages_host(batch->prefix_lens_host, batch->new_lens_host, batch->batch);
    a.k_inv = 1.f / pk.k_scale;  // IEEE division: the same fl32(1 / scale) the definition uses
    a.v_inv = 1.f / pk.v_scale;
    return a;
}

gc_status append(const gc_geometry* geo, const gc_batch* batch, const void* k_new, const void* v_new,
                 void* k_pool, void* v_pool, const PoolKind& pk, hipStream_t stream) {
    Shape sh;
    gc_status st = check_common(geo, batch, &sh);
    if (st != GC_OK) return st;
    if (sh.total_tokens == 0) return GC_OK;
    if (k_new == nullptr || v_new == nullptr || k_pool == nullptr || v_pool == nullptr)
        return GC_ERR_NULL_ARG;
    const gc::AppendArgs a = append_args(geo, batch, sh, k_new, v_new, k_pool, v_pool, pk);
    return gc::launch_append(a, geo->head_dim, pk.fp8, stream) == hipSuccess ? GC_OK : GC_ERR_HIP;
}

// Append and plan in one launch (the plan reads only the lengths, so the two are
// independent).
gc_status prepare(const gc_geometry* geo, const gc_batch* batch, const gc_plan_options* opts,
                  const void* k_new, const void* v_new, void* k_pool, void* v_pool, void* workspace,
                  size_t workspace_bytes, hipStream_t stream, const PoolKind& pk) {
    Shape sh;
    Plan pl;
    gc_status st = plan_checked(geo, batch, opts, &sh, &pl);
    if (st != GC_OK || sh.total_tokens == 0) return st;
    if (k_new == nullptr || v_new == nullptr || k_pool == nullptr || v_pool == nullptr)
        return GC_ERR_NULL_ARG;
    if (pk.fp8) {
        st = check_pool_scales(pk.k_scale, pk.v_scale);
        if (st != GC_OK) return st;
    }
    st = check_workspace(pl, workspace, workspace_bytes);
    if (st != GC_OK) return st;
    const gc::AppendArgs aa = append_args(geo, batch, sh, k_new, v_new, k_pool, v_pool, pk);
    return gc::launch_prepare(aa, plan_args(geo, batch, sh, pl, workspace), geo->head_dim, pk.fp8, stream) ==
                   hipSuccess
               ? GC_OK
               : GC_ERR_HIP;
}

gc_status run(const gc_geometry* geo, const gc_batch* batch, const gc_plan_options* opts,
              const void* q, const void* k_pool, const void* v_pool, float scale, void* out,
              float* lse, void* workspace, size_t workspace_bytes, hipStream_t stream,
              bool with_plan, const PoolKind& pk) {
    Shape sh;
    Plan pl;
    gc_status st = plan_checked(geo, batch, opts, &sh, &pl);
    if (st != GC_OK || sh.total_tokens == 0) return st;
    st = check_run_args(q, k_pool, v_pool, scale, out);
    if (st != GC_OK) return st;
    if (pk.fp8) {
        st = check_pool_scales(pk.k_scale, pk.v_scale);
        if (st != GC_OK) return st;
    }
    st = check_workspace(pl, workspace, workspace_bytes);
    if (st != GC_OK) return st;
    if (with_plan) {
        st = enqueue_plan(geo, batch, sh, pl, workspace, stream);
        if (st != GC_OK) return st;
    }
    return enqueue_run(geo, batch, sh, pl, q, k_pool, v_pool, scale, out, lse, workspace, stream, pk);
}

// ---------------------------------------------------------------- no-allocation variant
// Workspace of gc_prefix_prefill_attention_noalloc: one file-scope device array per
// GPU the library runs on (held until the process ends). Host code never passes the
// array's name to a kernel or a copy: in host code it is a host-side stand-in, not
// a device address. The device address comes from hipGetSymbolAddress, taken once
// per device with that device current, and is kept per device.
static __device__ __align__(256) unsigned char scratch[GC_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
struct DeviceScratch {
    std::once_flag once;
    void* ptr = nullptr;
    hipError_t err = hipSuccess;
};
DeviceScratch g_scratch[kMaxDevices];

// Device address of the current device's scratch array (nullptr and a status on failure).
void* scratch_address(gc_status* st) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0) {
        *st = GC_ERR_HIP;
        return nullptr;
    }
    if (dev >= kMaxDevices) {
        *st = GC_ERR_UNSUPPORTED;
        return nullptr;
    }
    DeviceScratch& d = g_scratch[dev];
    std::call_once(d.once, [&d]() { d.err = hipGetSymbolAddress(&d.ptr, HIP_SYMBOL(scratch)); });
    if (d.err != hipSuccess || d.ptr == nullptr) {
        *st = GC_ERR_HIP;
        return nullptr;
    }
    *st = GC_OK;
    return d.ptr;
}

// Append and run from a plan already in the workspace. Prefill tiles: one launch
// (the work items read the new keys from k_new / v_new and write their own tokens'
// K/V into the pools). Small tiles read every key from the pool, so there the append
// is its own launch, before the attention.
gc_status run_with_append(const gc_geometry* geo, const gc_batch* batch, const gc_plan_options* opts,
                          const void* q, const void* k_new, const void* v_new, void* k_pool, void* v_pool,
                          float scale, void* out, float* lse, void* workspace, size_t workspace_bytes,
                          hipStream_t stream) {
    Shape sh;
    Plan pl;
    gc_status st = plan_checked(geo, batch, opts, &sh, &pl);
    if (st != GC_OK || sh.total_tokens == 0) return st;
    st = check_run_args(q, k_pool, v_pool, scale, out);
    if (st != GC_OK) return st;
    if (k_new == nullptr || v_new == nullptr) return GC_ERR_NULL_ARG;
    st = check_workspace(pl, workspace, workspace_bytes);
    if (st != GC_OK) return st;
    // the attention addresses a request's new rows with 32-bit offsets
    const int64_t row_bytes = (int64_t)geo->num_kv_heads * geo->head_dim * 2;
    for (int r = 0; r < batch->batch; ++r)
        if ((int64_t)batch->new_lens_host[r] * row_bytes > INT32_MAX) return GC_ERR_UNSUPPORTED;
    const gc::AppendArgs aa = append_args(geo, batch, sh, k_new, v_new, k_pool, v_pool, PoolKind{});
    if (sh.small) {
        if (gc::launch_append(aa, geo->head_dim, false, stream) != hipSuccess) return GC_ERR_HIP;
        return enqueue_run(geo, batch, sh, pl, q, k_pool, v_pool, scale, out, lse, workspace, stream);
    }
    return enqueue_run(geo, batch, sh, pl, q, k_pool, v_pool, scale, out, lse, workspace, stream, PoolKind{},
                       &aa);
}

}  // namespace

extern "C" {

__attribute__((visibility("default")))
gc_status gc_kv_append(const gc_geometry* geo, const gc_batch* batch, const void* k_new,
                       const void* v_new, void* k_pool, void* v_pool, hipStream_t stream) {
    return append(geo, batch, k_new, v_new, k_pool, v_pool, PoolKind{}, stream);
}

__attribute__((visibility("default")))
gc_status gc_kv_append_fp8(const gc_geometry* geo, const gc_batch* batch, const void* k_new,
                           const void* v_new, float k_scale, float v_scale, void* k_pool,
                           void* v_pool, hipStream_t stream) {
    const gc_status st = check_pool_scales(k_scale, v_scale);
    if (st != GC_OK) return st;
    return append(geo, batch, k_new, v_new, k_pool, v_pool, PoolKind{true, k_scale, v_scale}, stream);
}

__attribute__((visibility("default")))
gc_status gc_prefix_prefill_workspace_size(const gc_geometry* geo, const gc_batch* batch,
                                           const gc_plan_options* opts, size_t* bytes) {
    if (bytes == nullptr) return GC_ERR_NULL_ARG;
    Shape sh;
    Plan pl;
    gc_status st = plan_checked(geo, batch, opts, &sh, &pl);
    if (st != GC_OK) return st;
    *bytes = sh.total_tokens == 0 ? 0 : pl.layout.total;
    return GC_OK;
}

__attribute__((visibility("default")))
gc_status gc_prefix_prefill_plan(const gc_geometry* geo, const gc_batch* batch,
                                 const gc_plan_options* opts, void* workspace,
                                 size_t workspace_bytes, hipStream_t stream) {
    Shape sh;
    Plan pl;
    gc_status st = plan_checked(geo, batch, opts, &sh, &pl);
    if (st != GC_OK || sh.total_tokens == 0) return st;
    st = check_workspace(pl, workspace, workspace_bytes);
    if (st != GC_OK) return st;
    return enqueue_plan(geo, batch, sh, pl, workspace, stream);
}

__attribute__((visibility("default")))
gc_status gc_prefix_prefill_run(const gc_geometry* geo, const gc_batch* batch,
                                const gc_plan_options* opts, const void* q, const void* k_pool,
                                const void* v_pool, float scale, void* out, float* lse,
                                void* workspace, size_t workspace_bytes, hipStream_t stream) {
    return run(geo, batch, opts, q, k_pool, v_pool, scale, out, lse, workspace, workspace_bytes,
               stream, false, PoolKind{});
}

__attribute__((visibility("default")))
gc_status gc_prefix_prefill_attention(const gc_geometry* geo, const gc_batch* batch,
                                      const gc_plan_options* opts, const void* q,
                                      const void* k_pool, const void* v_pool, float scale,
                                      void* out, float* lse, void* workspace,
                                      size_t workspace_bytes, hipStream_t stream) {
    return run(geo, batch, opts, q, k_pool, v_pool, scale, out, lse, workspace, workspace_bytes,
               stream, true, PoolKind{});
}

__attribute__((visibility("default")))
gc_status gc_prefix_prefill_attention_noalloc(const gc_geometry* geo, const gc_batch* batch,
                                              const gc_plan_options* opts, const void* q,
                                              const void* k_pool, const void* v_pool, float scale,
                                              void* out, float* lse, hipStream_t stream) {
    // every host check first (workspace size included), then the device address
    Shape sh;
    Plan pl;
    gc_status st = plan_checked(geo, batch, opts, &sh, &pl);
    if (st != GC_OK || sh.total_tokens == 0) return st;
    st = check_run_args(q, k_pool, v_pool, scale, out);
    if (st != GC_OK) return st;
    if (pl.layout.total > (size_t)GC_NOALLOC_SCRATCH_BYTES) return GC_ERR_WORKSPACE;
    void* ws = scratch_address(&st);
    if (ws == nullptr) return st;
    return run(geo, batch, opts, q, k_pool, v_pool, scale, out, lse, ws, GC_NOALLOC_SCRATCH_BYTES, stream,
               true, PoolKind{});
}

__attribute__((visibility("default")))
gc_status gc_prefix_prefill_run_with_append(const gc_geometry* geo, const gc_batch* batch,
                                            const gc_plan_options* opts, const void* q, const void* k_new,
                                            const void* v_new, void* k_pool, void* v_pool, float scale,
                                            void* out, float* lse, void* workspace, size_t workspace_bytes,
                                            hipStream_t stream) {
    return run_with_append(geo, batch, opts, q, k_new, v_new, k_pool, v_pool, scale, out, lse, workspace,
                           workspace_bytes, stream);
}

__attribute__((visibility("default")))
gc_status gc_prefix_prefill_run_fp8(const gc_geometry* geo, const gc_batch* batch,
                                    const gc_plan_options* opts, const void* q, const void* k_pool,
                                    const void* v_pool, float k_scale, float v_scale, float scale,
                                    void* out, float* lse, void* workspace, size_t workspace_bytes,
                                    hipStream_t stream) {
    return run(geo, batch, opts, q, k_pool, v_pool, scale, out, lse, workspace, workspace_bytes,
               stream, false, PoolKind{true, k_scale, v_scale});
}

__attribute__((visibility("default")))
gc_status gc_prefix_prefill_attention_fp8(const gc_geometry* geo, const gc_batch* batch,
                                          const gc_plan_options* opts, const void* q,
                                          const void* k_pool, const void* v_pool, float k_scale,
                                          float v_scale, float scale, void* out, float* lse,
                                          void* workspace, size_t workspace_bytes,
                                          hipStream_t stream) {
    return run(geo, batch, opts, q, k_pool, v_pool, scale, out, lse, workspace, workspace_bytes,
               stream, true, PoolKind{true, k_scale, v_scale});
}

__attribute__((visibility("default")))
gc_status gc_prefix_prefill_prepare(const gc_geometry* geo, const gc_batch* batch,
                                    const gc_plan_options* opts, const void* k_new, const void* v_new,
                                    void* k_pool, void* v_pool, void* workspace, size_t workspace_bytes,
                                    hipStream_t stream) {
    return prepare(geo, batch, opts, k_new, v_new, k_pool, v_pool, workspace, workspace_bytes, stream,
                   PoolKind{});
}

__attribute__((visibility("default")))
gc_status gc_prefix_prefill_prepare_fp8(const gc_geometry* geo, const gc_batch* batch,
                                        const gc_plan_options* opts, const void* k_new, const void* v_new,
                                        float k_scale, float v_scale, void* k_pool8, void* v_pool8,
                                        void* workspace, size_t workspace_bytes, hipStream_t stream) {
    return prepare(geo, batch, opts, k_new, v_new, k_pool8, v_pool8, workspace, workspace_bytes, stream,
                   PoolKind{true, k_scale, v_scale});
}

__attribute__((visibility("default")))
gc_status gc_prefix_prefill_plan_status(const void* workspace, size_t workspace_bytes, hipStream_t stream) {
    if (workspace == nullptr) return GC_ERR_NULL_ARG;
    if (workspace_bytes < sizeof(int32_t)) return GC_ERR_WORKSPACE;
    static_assert(gc::kStatusOffset == 0, "the status word leads the workspace");
    int32_t word = 0;
    if (hipMemcpyAsync(&word, workspace, sizeof(word), hipMemcpyDeviceToHost, stream) != hipSuccess ||
        hipStreamSynchronize(stream) != hipSuccess)
        return GC_ERR_HIP;
    return word == 0 ? GC_OK : GC_ERR_LENGTHS;
}

__attribute__((visibility("default")))
gc_status gc_read_bandwidth_probe(const void* buf, size_t bytes, void* sink, hipStream_t stream) {
    if (buf == nullptr || sink == nullptr) return GC_ERR_NULL_ARG;
    if (bytes % 16 != 0) return GC_ERR_BAD_SHAPE;
    if (bytes == 0) return GC_OK;
    return gc::launch_read_probe(buf, bytes, static_cast<uint32_t*>(sink), stream) == hipSuccess ? GC_OK
                                                                                               : GC_ERR_HIP;
}

__attribute__((visibility("default")))
gc_status gc_mfma_peak_probe(int32_t iterations, void* sink, hipStream_t stream) {
    static_assert(GC_MFMA_PROBE_SINK_FLOATS == gc::kMfmaProbeBlocks * gc::kProbeThreads, "sink size");
    static_assert(GC_MFMA_PROBE_PRODUCTS_PER_ITERATION ==
                      gc::kMfmaProbeBlocks * (gc::kProbeThreads / 64) * gc::kMfmaProbeChains * gc::kMfmaProbePerChain,
                  "products per iteration");
    if (sink == nullptr) return GC_ERR_NULL_ARG;
    if (iterations < 0) return GC_ERR_BAD_SHAPE;
    if (iterations == 0) return GC_OK;
    return gc::launch_mfma_probe(iterations, static_cast<float*>(sink), stream) == hipSuccess ? GC_OK : GC_ERR_HIP;
}

__attribute__((visibility("default")))
const char* gc_status_string(gc_status s) {
    switch (s) {
        case GC_OK: return "GC_OK: success";
        case GC_ERR_NULL_ARG: return "GC_ERR_NULL_ARG: a required pointer is NULL";
        case GC_ERR_BAD_SHAPE: return "GC_ERR_BAD_SHAPE: invalid size, length or scale";
        case GC_ERR_UNSUPPORTED: return "GC_ERR_UNSUPPORTED: head_dim must be 64 or 128, page_size 16, Hq/Hkv <= 128 (<= 16 for small tiles)";
        case GC_ERR_BLOCK_TABLE: return "GC_ERR_BLOCK_TABLE: block table too short for a request";
        case GC_ERR_WORKSPACE: return "GC_ERR_WORKSPACE: workspace missing or too small";
        case GC_ERR_HIP: return "GC_ERR_HIP: a HIP launch failed";
        case GC_ERR_LENGTHS: return "GC_ERR_LENGTHS: the device length arrays disagree with the host's";
    }
    return "unknown gc_status";
}

}  // extern "C"
