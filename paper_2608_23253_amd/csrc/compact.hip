// Token compaction (the model side of a pruning operation, Algorithm 1's V_keep):
// dst[b, r, j, :] = src[b, r, keep_idx[b, j], :].
//
// A streaming gather: every token vector is C * elem_bytes contiguous bytes, moved
// as 16-byte packets.  Thread g of the grid takes packets g, g + stride, ... of the
// flattened (image, row, kept token, packet) space, four at a time (all four loads
// issued before the first store), so a wave reads and writes whole runs of
// consecutive packets of one or more token vectors; the loads and stores carry
// the non-temporal hint (each byte is moved once).
#include "e2s_device.h"
#include "e2s_kernels.h"

namespace e2s {
namespace {

constexpr int kThreads = 256;
constexpr int kUnroll = 4;

struct CompactArgs {
    int64_t B, R, K, V;            // V: 16-byte packets per token vector
    int64_t N;
    int64_t ss[3], ds[3];          // strides in bytes
};

__device__ __forceinline__ bool packet_address(const CompactArgs& a, const int32_t* keep,
                                               int64_t i, int64_t& so, int64_t& dof) {
    const int64_t item = i / a.V, p = i - item * a.V;
    const int64_t b = item / (a.R * a.K), rk = item - b * a.R * a.K;
    const int64_t r = rk / a.K, j = rk - r * a.K;
    const int32_t n = keep[b * a.K + j];
    so = b * a.ss[0] + r * a.ss[1] + static_cast<int64_t>(n) * a.ss[2] + 16 * p;
    dof = b * a.ds[0] + r * a.ds[1] + j * a.ds[2] + 16 * p;
    return n >= 0 && n < a.N;
}

__global__ __launch_bounds__(kThreads) void compact_kernel(const int32_t* __restrict__ keep,
                                                           const char* __restrict__ src,
                                                           char* __restrict__ dst,
                                                           CompactArgs a, int64_t total) {
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kThreads;
    for (int64_t i0 = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x; i0 < total;
         i0 += kUnroll * stride) {
        u32x4 v[kUnroll];
        int64_t dof[kUnroll];
        bool ok[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const int64_t i = i0 + u * stride;
            int64_t so = 0;
            ok[u] = i < total && packet_address(a, keep, i, so, dof[u]);
            v[u] = ok[u] ? __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(src + so))
                         : u32x4{0u, 0u, 0u, 0u};
        }
#pragma unroll
        for (int u = 0; u < kUnroll; ++u)
            if (ok[u]) __builtin_nontemporal_store(v[u], reinterpret_cast<u32x4*>(dst + dof[u]));
    }
}

}  // namespace

hipError_t launch_compact(const e2s_compact_shape& s, const int32_t* keep, const void* src,
                          void* dst, hipStream_t st) {
    CompactArgs a;
    a.B = s.batch;
    a.R = s.rows;
    a.K = s.keep;
    a.N = s.num_tokens;
    a.V = static_cast<int64_t>(s.channels) * s.elem_bytes / 16;
    for (int i = 0; i < 3; ++i) {
        a.ss[i] = s.src_stride[i] * s.elem_bytes;
        a.ds[i] = s.dst_stride[i] * s.elem_bytes;
    }
    const int64_t total = a.B * a.R * a.K * a.V;
    if (total == 0) return hipSuccess;
    // enough workgroups to fill the device several times over, each thread moving
    // a few groups of kUnroll packets
    const int64_t want = (total + kThreads * kUnroll - 1) / (kThreads * kUnroll);
    const unsigned blocks = static_cast<unsigned>(want < 65536 ? want : 65536);
    hipLaunchKernelGGL(compact_kernel, dim3(blocks), dim3(kThreads), 0, st, keep,
                       static_cast<const char*>(src), static_cast<char*>(dst), a, total);
    return hipGetLastError();
}

}  // namespace e2s
