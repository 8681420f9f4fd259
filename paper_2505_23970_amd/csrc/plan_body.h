// Attention work-list builder (device code shared by the plan kernel and the
// fused append-and-plan launch), run on the device from the device copies of the
// batch lengths (no host-to-device copy, so a plan can be enqueued freely and
// captured in a graph).
//
// One workgroup:
//   1. per-request query-tile counts and their exclusive scan (cum[], in LDS
//      with the batch lengths for batches of up to kPlanLdsBatch requests, else
//      in the workspace), so that every thread can take query tiles of any
//      request by a global tile index;
//   2. a histogram of item costs (key tiles per item) in LDS, scanned so that
//      the heaviest items come first (above the host's cost threshold, the
//      items of one request side by side: bucket_of);
//   3. every item is written straight to its sorted position (an LDS cursor per
//      cost bucket, advanced once per distinct chunk size of a tile); split query
//      tiles take their partial slots and merge entry from two LDS counters.
// The hardware dispatcher starts workgroups in index order (the resident launch
// hands out its tickets in the same order): the items of the
// longest requests start first, each request's items together, and the launch
// ends on its lightest items in cost order (longest-processing-time scheduling
// where it matters, at the end). Order inside a bucket and slot numbers may
// differ between runs; results do not depend on them (every item writes its own
// outputs, merges run in chunk order).
// The device lengths are checked before anything is derived from them: cu[0]
// must be 0, cu non-decreasing with cu[B] equal to the host's T, every prefix
// length non-negative, every request's keys within the block-table row, and the
// item, merge and partial counts equal to the host's. Otherwise (the caller
// passed host and device arrays that disagree) every item is emitted empty and
// status[0] is set to 1: the attention kernels then write nothing, and nothing
// is accessed out of bounds. gc_prefix_prefill_plan_status reads the word.
#pragma once
#include "gc_internal.h"

namespace gc {
namespace {


// exclusive scan of one value per thread; *total receives the sum (a scan inside
// each wavefront, then one exchange of the wavefront totals through LDS)
__device__ int block_exclusive_scan(int v, int* s_tmp, int* total) {
    constexpr int kWavesPlan = kPlanThreads / 64;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    int x = v;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const int y = __shfl_up(x, d);
        if (lane >= d) x += y;
    }
    if (lane == 63) s_tmp[wave] = x;
    __syncthreads();
    int base = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < kWavesPlan; ++w) {
        const int t = s_tmp[w];
        base += w < wave ? t : 0;
        tot += t;
    }
    __syncthreads();  // s_tmp is reused by the next scan
    *total = tot;
    return base + x - v;
}

// Counting-sort bucket of an item of `cost` key tiles from a request of
// `req_tiles` key tiles in all. Items of at least group_cost key tiles are sorted
// by req_tiles, longest request first, so that all of a request's items run side
// by side: its query tiles read nearly the same keys and share them in L2, where
// in cost order the tiles of one request (a long miss has tiles of every cost
// from 1 up) are spread over the launch and fetch the same K/V again each time.
// Lighter items, the last rounds of the launch, follow in cost order, heaviest
// first, so that the launch still ends on its lightest items. req_tiles >= cost,
// so every grouped item precedes every lighter one.
__device__ __forceinline__ int bucket_of(const PlanArgs& a, int cost, int req_tiles) {
    const int c = min(cost, kCostBuckets - 1);
    return kCostBuckets - 1 - (c >= a.group_cost ? min(req_tiles, kCostBuckets - 1) : c);
}

struct Tile {
    int r, q0, kt, ns;
    int req_tiles;  // key tiles of the whole request
};

// Batch lengths as the planner reads them: LDS copies for batches of up to
// kPlanLdsBatch requests (the searches below then cost no memory round trips),
// else the global arrays.
struct Lens {
    const int* cum;     // [batch + 1] exclusive scan of query tiles per request
    const int* cu;      // [batch + 1] exclusive scan of new tokens
    const int* prefix;  // [batch]
};

// query tile number g (over the whole batch) -> request, first token, key tiles, splits
__device__ __forceinline__ Tile tile_at(const PlanArgs& a, const Lens& l, int g) {
    int lo = 0, hi = a.batch;  // largest r with cum[r] <= g
    while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (l.cum[mid] <= g) lo = mid;
        else hi = mid;
    }
    Tile t;
    t.r = lo;
    t.q0 = (g - l.cum[lo]) * a.tq;
    const int n = l.cu[lo + 1] - l.cu[lo];
    const int ntok = min(a.tq, n - t.q0);
    t.kt = key_tiles(l.prefix[lo], t.q0, ntok, a.block_n);
    t.ns = num_splits(t.kt, a.chunk);
    t.req_tiles = key_tiles(l.prefix[lo], 0, n, a.block_n);
    return t;
}

// LDS of the planner's workgroup (the caller provides it, so that a launch that
// also runs the append can overlay the two).
struct PlanLds {
    int tmp[kPlanThreads];
    int hist[kCostBuckets];
    int part, comb, bad, badlen;
    int cum[kPlanLdsBatch + 1], cu[kPlanLdsBatch + 1], pre[kPlanLdsBatch];
};

// The planner's workgroup (kPlanThreads threads).
__device__ __forceinline__ void plan_body(const PlanArgs& a, PlanLds& sm) {
    int* const s_tmp = sm.tmp;
    int* const s_hist = sm.hist;
    int& s_part = sm.part;
    int& s_comb = sm.comb;
    int& s_bad = sm.bad;
    int& s_badlen = sm.badlen;
    int* const s_cum = sm.cum;
    int* const s_cu = sm.cu;
    int* const s_pre = sm.pre;
    const int tid = threadIdx.x;
    if (tid <= kQueues) a.queues[tid] = 0;  // the resident attention launch starts from empty tickets
    const bool small = a.batch <= kPlanLdsBatch;
    int* cum = small ? s_cum : a.scratch;  // [batch + 1]
    if (tid == 0) s_badlen = 0;
    if (small) {
        for (int r = tid; r <= a.batch; r += kPlanThreads) {
            s_cu[r] = a.cu_new_lens[r];
            if (r < a.batch) s_pre[r] = a.prefix_lens[r];
        }
    }
    __syncthreads();
    const Lens lens{cum, small ? s_cu : a.cu_new_lens, small ? s_pre : a.prefix_lens};

    // 0. the device lengths must describe the batch the host checked
    const int per = ceil_div(a.batch, kPlanThreads);
    const int r0 = min(a.batch, tid * per), r1 = min(a.batch, r0 + per);
    {
        bool bad = tid == 0 && (lens.cu[0] != 0 || lens.cu[a.batch] != a.total_tokens);
        for (int r = r0; r < r1; ++r) {
            const int64_t P = lens.prefix[r], c0 = lens.cu[r], n = (int64_t)lens.cu[r + 1] - c0;
            bad |= P < 0 || n < 0 || P + n > (int64_t)INT32_MAX - kBlockN ||
                   (n > 0 && ceil_div64(P + n, kPage) > a.max_blocks);
        }
        if (bad) s_badlen = 1;
    }
    __syncthreads();
    if (s_badlen) {
        for (int i = tid; i < a.expect_combines; i += kPlanThreads) a.combines[i] = CombineItem{0, 0, 0, 0};
        for (int i = tid; i < a.expect_items; i += kPlanThreads) a.items[i] = WorkItem{-1, 0, 0, 0, -1, 0, 0, 0};
        if (tid == 0) a.status[0] = 1;
        return;
    }

    // 1. query tiles per request, scanned
    int mine = 0;
    for (int r = r0; r < r1; ++r)
        mine += ceil_div(lens.cu[r + 1] - lens.cu[r], a.tq);
    int total_tiles;
    int off = block_exclusive_scan(mine, s_tmp, &total_tiles);
    for (int r = r0; r < r1; ++r) {
        cum[r] = off;
        off += ceil_div(lens.cu[r + 1] - lens.cu[r], a.tq);
    }
    if (tid == 0) cum[a.batch] = total_tiles;
    for (int b = tid; b < kCostBuckets; b += kPlanThreads) s_hist[b] = 0;
    if (tid == 0) {
        s_part = 0;
        s_comb = 0;
        s_bad = 0;
    }
    __threadfence_block();
    __syncthreads();

    // 2. cost histogram. The ns chunks of a tile have kt / ns key tiles (rounded
    // down) or one more, so two additions per tile cover all of its chunks.
    for (int g = tid; g < total_tiles; g += kPlanThreads) {
        const Tile t = tile_at(a, lens, g);
        const int lo = t.kt / t.ns, n_hi = t.kt - lo * t.ns, n_lo = t.ns - n_hi;
        if (n_lo > 0) atomicAdd(&s_hist[bucket_of(a, lo, t.req_tiles)], n_lo);
        if (n_hi > 0) atomicAdd(&s_hist[bucket_of(a, lo + 1, t.req_tiles)], n_hi);
    }
    __syncthreads();
    constexpr int kPer = kCostBuckets / kPlanThreads;
    int local = 0;
    for (int k = 0; k < kPer; ++k) local += s_hist[tid * kPer + k];
    int total_items;
    int base = block_exclusive_scan(local, s_tmp, &total_items);
    for (int k = 0; k < kPer; ++k) {
        const int c = s_hist[tid * kPer + k];
        s_hist[tid * kPer + k] = base;
        base += c;
    }
    // merge entries start empty; the split tiles below fill theirs
    for (int i = tid; i < a.expect_combines; i += kPlanThreads) a.combines[i] = CombineItem{0, 0, 0, 0};
    __syncthreads();
    if (total_items != a.expect_items) {
        for (int i = tid; i < a.expect_items; i += kPlanThreads)
            a.items[i] = WorkItem{-1, 0, 0, 0, -1, 0, 0, 0};
        if (tid == 0) a.status[0] = 1;
        return;
    }

    // 3. items at their sorted positions
    for (int g = tid; g < total_tiles; g += kPlanThreads) {
        const Tile t = tile_at(a, lens, g);
        int part0 = -1;
        if (t.ns > 1) {
            part0 = atomicAdd(&s_part, t.ns);
            const int ci = atomicAdd(&s_comb, 1);
            if (part0 + t.ns > a.expect_partials || ci >= a.expect_combines) {
                s_bad = 1;  // cannot happen when the item totals matched; never write out of range
                part0 = -2;
            } else {
                a.combines[ci] = CombineItem{t.r, t.q0, part0, t.ns};
            }
        }
        // reserve the tile's positions in both cost buckets at once, then hand them out
        const int lo = t.kt / t.ns, n_hi = t.kt - lo * t.ns, n_lo = t.ns - n_hi;
        int pos_lo = n_lo > 0 ? atomicAdd(&s_hist[bucket_of(a, lo, t.req_tiles)], n_lo) : 0;
        int pos_hi = n_hi > 0 ? atomicAdd(&s_hist[bucket_of(a, lo + 1, t.req_tiles)], n_hi) : 0;
        for (int s = 0; s < t.ns; ++s) {
            const int b0 = split_begin(s, t.kt, t.ns), b1 = split_begin(s + 1, t.kt, t.ns);
            const int pos = b1 - b0 == lo ? pos_lo++ : pos_hi++;
            a.items[pos] = part0 == -2 ? WorkItem{-1, 0, 0, 0, -1, 0, 0, 0}
                                       : WorkItem{t.r, t.q0, b0, b1, part0 < 0 ? -1 : part0 + s, lens.prefix[t.r],
                                                  lens.cu[t.r], lens.cu[t.r + 1] - lens.cu[t.r]};
        }
    }
    __syncthreads();
    if (tid == 0) a.status[0] = s_bad;
}

}  // namespace
}  // namespace gc
