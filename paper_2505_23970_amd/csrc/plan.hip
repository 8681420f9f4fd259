// Attention work-list builder, run on the device from the device copies of the
// batch lengths (no host-to-device copy, so a plan can be enqueued freely and
// captured in a graph).
//
// One workgroup:
//   1. each thread counts the work items, split query tiles and partial slots
//      of a contiguous range of requests, then an exclusive scan over threads
//      gives every request its output offsets;
//   2. items are emitted request-major (query tile, then key chunk), each split
//      tile also emitting a merge entry with its partial slots;
//   3. a counting sort by cost (key tiles) orders the list heaviest first, so
//      the hardware dispatcher, which starts workgroups in index order, runs
//      the longest items first (longest-processing-time scheduling).
// If the device lengths do not reproduce the host's totals (the caller passed
// different host and device arrays), every item is emitted empty and status[0]
// is set to 1: the attention kernel then writes nothing, but never strays out
// of bounds.
#include "gc_internal.h"

namespace gc {
namespace {

// exclusive scan of one value per thread; returns the thread's offset, *total the sum
__device__ int block_exclusive_scan(int v, int* s_tmp, int* total) {
    const int tid = threadIdx.x;
    s_tmp[tid] = v;
    __syncthreads();
    for (int d = 1; d < kPlanThreads; d <<= 1) {
        const int add = tid >= d ? s_tmp[tid - d] : 0;
        __syncthreads();
        s_tmp[tid] += add;
        __syncthreads();
    }
    const int incl = s_tmp[tid];
    *total = s_tmp[kPlanThreads - 1];
    __syncthreads();
    return incl - v;
}

__global__ __launch_bounds__(kPlanThreads) void plan_kernel(const PlanArgs a) {
    __shared__ int s_tmp[kPlanThreads];
    __shared__ int s_hist[kCostBuckets];
    const int tid = threadIdx.x;
    const int per = ceil_div(a.batch, kPlanThreads);
    const int r0 = min(a.batch, tid * per), r1 = min(a.batch, r0 + per);

    int ni = 0, nc = 0, np = 0;
    for (int r = r0; r < r1; ++r) {
        const int n = a.cu_new_lens[r + 1] - a.cu_new_lens[r];
        const RequestCounts c = request_counts(a.prefix_lens[r], n, a.tq, a.chunk);
        ni += c.items;
        nc += c.combines;
        np += c.partials;
    }
    int ti, tc, tp;
    int oi = block_exclusive_scan(ni, s_tmp, &ti);
    int oc = block_exclusive_scan(nc, s_tmp, &tc);
    int op = block_exclusive_scan(np, s_tmp, &tp);

    if (ti != a.expect_items || tc != a.expect_combines || tp != a.expect_partials) {
        for (int i = tid; i < a.expect_items; i += kPlanThreads)
            a.items[i] = WorkItem{-1, 0, 0, 0, -1, 0, 0, 0};
        for (int i = tid; i < a.expect_combines; i += kPlanThreads)
            a.combines[i] = CombineItem{0, 0, 0, 0};
        if (tid == 0) a.status[0] = 1;
        return;
    }

    for (int r = r0; r < r1; ++r) {
        const int P = a.prefix_lens[r];
        const int n = a.cu_new_lens[r + 1] - a.cu_new_lens[r];
        for (int q0 = 0; q0 < n; q0 += a.tq) {
            const int ntok = min(a.tq, n - q0);
            const int kt = key_tiles(P, q0, ntok);
            const int ns = num_splits(kt, a.chunk);
            if (ns == 1) {
                a.unsorted[oi++] = WorkItem{r, q0, 0, kt, -1, 0, 0, 0};
            } else {
                a.combines[oc++] = CombineItem{r, q0, op, ns};
                for (int s = 0; s < ns; ++s)
                    a.unsorted[oi++] = WorkItem{r, q0, split_begin(s, kt, ns), split_begin(s + 1, kt, ns), op + s, 0, 0, 0};
                op += ns;
            }
        }
    }

    // counting sort, heaviest first: bucket kCostBuckets-1-cost
    for (int b = tid; b < kCostBuckets; b += kPlanThreads) s_hist[b] = 0;
    __threadfence_block();
    __syncthreads();
    for (int i = tid; i < ti; i += kPlanThreads) {
        const WorkItem w = a.unsorted[i];
        const int cost = min(w.kt_end - w.kt_begin, kCostBuckets - 1);
        atomicAdd(&s_hist[kCostBuckets - 1 - cost], 1);
    }
    __syncthreads();
    constexpr int kPer = kCostBuckets / kPlanThreads;
    int local = 0;
    for (int k = 0; k < kPer; ++k) local += s_hist[tid * kPer + k];
    int dummy;
    int base = block_exclusive_scan(local, s_tmp, &dummy);
    for (int k = 0; k < kPer; ++k) {
        const int c = s_hist[tid * kPer + k];
        s_hist[tid * kPer + k] = base;
        base += c;
    }
    __syncthreads();
    for (int i = tid; i < ti; i += kPlanThreads) {
        const WorkItem w = a.unsorted[i];
        const int cost = min(w.kt_end - w.kt_begin, kCostBuckets - 1);
        const int pos = atomicAdd(&s_hist[kCostBuckets - 1 - cost], 1);
        a.items[pos] = w;
    }
    if (tid == 0) a.status[0] = 0;
}

}  // namespace

hipError_t launch_plan(const PlanArgs& a, hipStream_t s) {
    plan_kernel<<<1, kPlanThreads, 0, s>>>(a);
    return hipGetLastError();
}

}  // namespace gc
