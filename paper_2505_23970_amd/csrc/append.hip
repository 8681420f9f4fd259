// KV append kernel: one workgroup per pool page that receives new tokens and KV
// head (the device code is in append_body.h).
#include "append_body.h"

namespace gc {
namespace {

template <int D, bool FP8>
__global__ __launch_bounds__(kAppendThreads) void append_kernel(const AppendArgs a) {
    __shared__ AppendLds<D> lds;
    append_body<D, FP8>(a, lds, (int)blockIdx.x, (int)blockIdx.y);
}

}  // namespace

hipError_t launch_append(const AppendArgs& a, int head_dim, bool fp8, hipStream_t s) {
    if (a.total_pages <= 0) return hipSuccess;
    const dim3 grid((unsigned)a.total_pages, (unsigned)a.num_kv_heads);
    if (fp8) {
        if (head_dim == 128)
            append_kernel<128, true><<<grid, kAppendThreads, 0, s>>>(a);
        else
            append_kernel<64, true><<<grid, kAppendThreads, 0, s>>>(a);
    } else {
        if (head_dim == 128)
            append_kernel<128, false><<<grid, kAppendThreads, 0, s>>>(a);
        else
            append_kernel<64, false><<<grid, kAppendThreads, 0, s>>>(a);
    }
    return hipGetLastError();
}

}  // namespace gc
