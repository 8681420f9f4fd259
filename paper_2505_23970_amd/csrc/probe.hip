// Streaming-read probe: the sustained HBM read rate that the memory-bound
// attention cases are reported against (the nominal 8 TB/s of MI355X is not
// reachable by a read-only stream).
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

}  // namespace

hipError_t launch_read_probe(const void* buf, size_t bytes, uint32_t* sink, hipStream_t s) {
    read_probe_kernel<<<kProbeBlocks, kProbeThreads, 0, s>>>(static_cast<const u32x4*>(buf), bytes / 16, sink);
    return hipGetLastError();
}

}  // namespace gc
