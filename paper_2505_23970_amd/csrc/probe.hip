// Calibration probes, not part of the attention path.
// Streaming-read probe: the sustained HBM read rate that the memory-bound
// attention cases are reported against (the nominal 8 TB/s of MI355X is not
// reachable by a read-only stream).
// Matrix-core probe: the sustained bf16 MFMA rate (a register-only loop of
// independent v_mfma_f32_32x32x16_bf16 products on every SIMD), which the
// compute-bound attention cases are also reported against.
#include "gc_internal.h"

namespace gc {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(kProbeThreads) void read_probe_kernel(const u32x4* __restrict__ p, size_t n16,
                                                                  uint32_t* __restrict__ sink) {
    u32x4 acc = {0u, 0u, 0u, 0u};
    const size_t stride = (size_t)gridDim.x * kProbeThreads;
    for (size_t i = (size_t)blockIdx.x * kProbeThreads + threadIdx.x; i < n16; i += stride) acc ^= p[i];
    sink[(size_t)blockIdx.x * kProbeThreads + threadIdx.x] = acc[0] ^ acc[1] ^ acc[2] ^ acc[3];
}

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

// kMfmaProbeChains independent accumulators per wavefront, each advanced by
// kMfmaProbePerChain products per iteration; every operand element is 1, so each
// product adds 16 to every accumulator element and a thread's sum of its
// accumulators is exactly kMfmaProbeChains * 16 * 16 * kMfmaProbePerChain * iterations.
__global__ __launch_bounds__(kProbeThreads) void mfma_probe_kernel(int iterations, float* __restrict__ sink) {
    bf16x8 one;
#pragma unroll
    for (int i = 0; i < 8; ++i) one[i] = (__bf16)1.0f;
    f32x16 acc[kMfmaProbeChains];
#pragma unroll
    for (int c = 0; c < kMfmaProbeChains; ++c) acc[c] = f32x16{};
    for (int it = 0; it < iterations; ++it) {
#pragma unroll
        for (int j = 0; j < kMfmaProbePerChain; ++j)
#pragma unroll
            for (int c = 0; c < kMfmaProbeChains; ++c)
                acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(one, one, acc[c], 0, 0, 0);
    }
    float t = 0.f;
#pragma unroll
    for (int c = 0; c < kMfmaProbeChains; ++c)
#pragma unroll
        for (int e = 0; e < 16; ++e) t += acc[c][e];
    sink[(size_t)blockIdx.x * kProbeThreads + threadIdx.x] = t;
}

}  // namespace

hipError_t launch_mfma_probe(int iterations, float* sink, hipStream_t s) {
    mfma_probe_kernel<<<kMfmaProbeBlocks, kProbeThreads, 0, s>>>(iterations, sink);
    return hipGetLastError();
}

hipError_t launch_read_probe(const void* buf, size_t bytes, uint32_t* sink, hipStream_t s) {
    read_probe_kernel<<<kProbeBlocks, kProbeThreads, 0, s>>>(static_cast<const u32x4*>(buf), bytes / 16, sink);
    return hipGetLastError();
}

}  // namespace gc
