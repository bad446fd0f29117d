// Measurement helper (not a step of the method): a streaming read of device
// memory, timed by the benchmark to report the achievable read bandwidth of the
// device beside its nominal HBM peak.  Workgroup w reads the contiguous share
// [w * n / W, (w + 1) * n / W) of the n 16-byte packets with non-temporal loads,
// four packets per thread in flight, and folds them with XOR; the result is
// written only when it equals a fixed value, so the loads cannot be dropped and
// nothing else is written.
#include "e2s_device.h"
#include "e2s_kernels.h"

namespace e2s {
namespace {

constexpr int kProbeThreads = 256;
constexpr int kProbeUnroll = 4;
constexpr uint32_t kProbeMagic = 0x9E3779B9u;

__global__ __launch_bounds__(kProbeThreads) void read_probe_kernel(const u32x4* __restrict__ p,
                                                                   int64_t n,
                                                                   uint32_t* __restrict__ sink) {
    const int64_t first = n * blockIdx.x / gridDim.x;
    const int64_t end = n * (blockIdx.x + 1) / gridDim.x;
    uint32_t acc = 0;
    for (int64_t i = first + threadIdx.x; i < end; i += kProbeThreads * kProbeUnroll) {
        u32x4 v[kProbeUnroll];
#pragma unroll
        for (int u = 0; u < kProbeUnroll; ++u) {
            const int64_t j = i + u * kProbeThreads;
            const u32x4 zero = {0u, 0u, 0u, 0u};
            v[u] = j < end ? __builtin_nontemporal_load(p + j) : zero;
        }
#pragma unroll
        for (int u = 0; u < kProbeUnroll; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
    }
    if (acc == kProbeMagic) sink[0] = acc;
}

}  // namespace

hipError_t launch_read_probe(const void* buf, size_t bytes, int workgroups, uint32_t* sink,
                             hipStream_t stream) {
    hipLaunchKernelGGL(read_probe_kernel, dim3(static_cast<unsigned>(workgroups)),
                       dim3(kProbeThreads), 0, stream, static_cast<const u32x4*>(buf),
                       static_cast<int64_t>(bytes / 16), sink);
    return hipGetLastError();
}

}  // namespace e2s
