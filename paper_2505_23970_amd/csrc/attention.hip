// Launchers of the attention kernels over bf16 pools (the kernels are in
// attention_kernels.h). This file is compiled with the scheduler's
// register-pressure trackers enabled (the flags in build.py): measured on the
// bf16 kernels, 0.4-0.9 % faster on the compute-bound workloads and neutral on
// the others. The 8-bit-pool, fused-append and merge kernels are launched from
// attention_plain.hip, built without that option (the 8-bit 128-row kernel was
// 2 % slower with it).
#include "attention_kernels.h"

namespace gc {

hipError_t launch_attention(const AttnArgs& a, int head_dim, int64_t num_items, bool wide, bool fp8,
                            int resident, hipStream_t s) {
    if (fp8) return launch_attention_fp8(a, head_dim, num_items, wide, resident, s);
    const dim3 grid((unsigned)(num_items * a.num_kv_heads));
    if (resident > 0 && wide) {
        const int total = (int)(num_items * a.num_kv_heads);
        const dim3 rg((unsigned)resident), rb(kWideWaves * 64);
        if (head_dim == 128)
            hipLaunchKernelGGL((attention_resident_kernel<128, false>), rg, rb, 0, s, a, total);
        else
            hipLaunchKernelGGL((attention_resident_kernel<64, false>), rg, rb, 0, s, a, total);
        return hipGetLastError();
    }
    if (wide) {
        if (head_dim == 128)
            attention_kernel<128, kWideWaves, false><<<grid, kWideWaves * 64, 0, s>>>(a);
        else
            attention_kernel<64, kWideWaves, false><<<grid, kWideWaves * 64, 0, s>>>(a);
    } else {
        if (head_dim == 128)
            attention_kernel<128, kWaves, false><<<grid, kWaves * 64, 0, s>>>(a);
        else
            attention_kernel<64, kWaves, false><<<grid, kWaves * 64, 0, s>>>(a);
    }
    return hipGetLastError();
}

}  // namespace gc
