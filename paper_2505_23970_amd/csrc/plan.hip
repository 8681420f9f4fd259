// Attention work-list kernel: one workgroup builds the plan on the device (the
// device code is in plan_body.h).
#include "plan_body.h"

namespace gc {
namespace {

__global__ __launch_bounds__(kPlanThreads) void plan_kernel(const PlanArgs a) {
    __shared__ PlanLds lds;
    plan_body(a, lds);
}

}  // namespace

hipError_t launch_plan(const PlanArgs& a, hipStream_t s) {
    plan_kernel<<<1, kPlanThreads, 0, s>>>(a);
    return hipGetLastError();
}

}  // namespace gc
