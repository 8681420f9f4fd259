// Append and plan in one launch: workgroup 0 builds the attention work list while
// the others save the new tokens' K/V into the pool. The two jobs are
// independent (the plan reads only the batch lengths), so one launch overlaps
// them and saves a kernel boundary per step. The two roles overlay one LDS
// allocation (the planner's, ~15 KiB), which leaves room for eight append
// workgroups per compute unit.
#include "append_body.h"
#include "plan_body.h"

namespace gc {
namespace {

static_assert(kAppendThreads == kPlanThreads, "one block size for both jobs");

template <int D>
union PrepareLds {
    PlanLds plan;
    AppendLds<D> append;
};

template <int D, bool FP8>
__global__ __launch_bounds__(kAppendThreads) void prepare_kernel(const AppendArgs aa, const PlanArgs pa) {
    __shared__ PrepareLds<D> lds;
    if (blockIdx.x == 0) {
        plan_body(pa, lds.plan);
    } else {
        const unsigned b = blockIdx.x - 1;
        append_body<D, FP8>(aa, lds.append, (int)(b % (unsigned)aa.total_pages), (int)(b / (unsigned)aa.total_pages));
    }
}

}  // namespace

hipError_t launch_prepare(const AppendArgs& aa, const PlanArgs& pa, int head_dim, bool fp8, hipStream_t s) {
    const dim3 grid((unsigned)(1 + (int64_t)aa.total_pages * aa.num_kv_heads));
    if (fp8) {
        if (head_dim == 128)
            prepare_kernel<128, true><<<grid, kAppendThreads, 0, s>>>(aa, pa);
        else
            prepare_kernel<64, true><<<grid, kAppendThreads, 0, s>>>(aa, pa);
    } else {
        if (head_dim == 128)
            prepare_kernel<128, false><<<grid, kAppendThreads, 0, s>>>(aa, pa);
        else
            prepare_kernel<64, false><<<grid, kAppendThreads, 0, s>>>(aa, pa);
    }
    return hipGetLastError();
}

}  // namespace gc
