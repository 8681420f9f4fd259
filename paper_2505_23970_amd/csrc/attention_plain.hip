// Launchers of the attention kernels over 8-bit pools, of the attention kernels
// with the KV append fused in, and of the split merge (the kernels are in
// attention_kernels.h), built with the compiler's default scheduling.
#include "attention_kernels.h"

namespace gc {

hipError_t launch_attention_fp8(const AttnArgs& a, int head_dim, int64_t num_items, bool wide, int resident,
                                hipStream_t s) {
    const dim3 grid((unsigned)(num_items * a.num_kv_heads));
    if (resident > 0 && wide) {
        const int total = (int)(num_items * a.num_kv_heads);
        const dim3 rg((unsigned)resident), rb(kWideWaves * 64);
        if (head_dim == 128)
            hipLaunchKernelGGL((attention_resident_kernel<128, true>), rg, rb, 0, s, a, total);
        else
            hipLaunchKernelGGL((attention_resident_kernel<64, true>), rg, rb, 0, s, a, total);
        return hipGetLastError();
    }
    if (wide) {
        if (head_dim == 128)
            attention_kernel<128, kWideWaves, true><<<grid, kWideWaves * 64, 0, s>>>(a);
        else
            attention_kernel<64, kWideWaves, true><<<grid, kWideWaves * 64, 0, s>>>(a);
    } else {
        if (head_dim == 128)
            attention_kernel<128, kWaves, true><<<grid, kWaves * 64, 0, s>>>(a);
        else
            attention_kernel<64, kWaves, true><<<grid, kWaves * 64, 0, s>>>(a);
    }
    return hipGetLastError();
}

hipError_t launch_attention_append(const AttnArgs& a, int head_dim, int64_t num_items, bool wide,
                                   hipStream_t s) {
    const dim3 grid((unsigned)(num_items * a.num_kv_heads));
    if (wide) {
        if (head_dim == 128)
            attention_append_kernel<128, kWideWaves><<<grid, kWideWaves * 64, 0, s>>>(a);
        else
            attention_append_kernel<64, kWideWaves><<<grid, kWideWaves * 64, 0, s>>>(a);
    } else {
        if (head_dim == 128)
            attention_append_kernel<128, kWaves><<<grid, kWaves * 64, 0, s>>>(a);
        else
            attention_append_kernel<64, kWaves><<<grid, kWaves * 64, 0, s>>>(a);
    }
    return hipGetLastError();
}

hipError_t launch_combine(const CombineArgs& a, int head_dim, int64_t num_combines, hipStream_t s) {
    const int groups = ceil_div(a.block_m, kCombineThreads / (head_dim / 4));
    const dim3 grid((unsigned)(num_combines * a.num_kv_heads * groups));
    if (head_dim == 128)
        combine_kernel<128><<<grid, kCombineThreads, 0, s>>>(a);
    else
        combine_kernel<64><<<grid, kCombineThreads, 0, s>>>(a);
    return hipGetLastError();
}

}  // namespace gc
