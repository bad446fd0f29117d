// Evidence stages (Sec. 4.1 Eq. 10-11, Sec. 4.2 Eq. 12-19).
//
// One thread per (image, visual token); consecutive threads take consecutive
// tokens, so every read of a [.., H, N] or [.., L, N] row is a coalesced
// 256-byte wave access.  The running fused mass of a token lives in registers
// across the L layers.  The staged kernels and the fused kernel call the same
// device functions (e2s_device.h), compiled without floating-point contraction,
// so e2s_fuse_evidence returns the same bits as the three staged calls.
#include "e2s_device.h"
#include "e2s_kernels.h"

namespace e2s {
namespace {

constexpr int kThreads = 256;

// sum_h e_h and sum_h |e_h - ebar| over the H heads of one (image, layer, token).
__device__ __forceinline__ void head_sums(const float* __restrict__ e, int64_t stride, int H,
                                          float& s1, float& ebar, float& s2) {
    s1 = 0.f;
    for (int h = 0; h < H; ++h) s1 += e[h * stride];
    ebar = s1 / static_cast<float>(H);
    s2 = 0.f;
    for (int h = 0; h < H; ++h) s2 += fabsf(e[h * stride] - ebar);
}

__global__ __launch_bounds__(kThreads) void head_reliability_kernel(
    const float* __restrict__ e, float* __restrict__ rho, float* __restrict__ pbar_c,
    int64_t BL, int H, int N) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x;
    if (i >= BL * N) return;
    const int64_t bl = i / N, n = i - bl * N;
    const float two_over_h = 2.0f / static_cast<float>(H);
    float s1, ebar, s2;
    head_sums(e + bl * H * N + n, N, H, s1, ebar, s2);
    rho[i] = reliability_from_sums(s1, s2, two_over_h);
    pbar_c[i] = ebar;
}

__global__ __launch_bounds__(kThreads) void head_masses_kernel(
    const float* __restrict__ rho, const float* __restrict__ pbar_c, float* __restrict__ mass,
    int64_t count) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x;
    if (i >= count) return;
    float mI, mU, mT;
    masses_from_reliability(rho[i], pbar_c[i], mI, mU, mT);
    mass[3 * i + 0] = mI;
    mass[3 * i + 1] = mU;
    mass[3 * i + 2] = mT;
}

__global__ __launch_bounds__(kThreads) void ds_combine_kernel(
    const float* __restrict__ mass, float* __restrict__ fused, float* __restrict__ conflict,
    float* __restrict__ prio_c, int B, int L, int N) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x;
    if (i >= static_cast<int64_t>(B) * N) return;
    const int64_t b = i / N, n = i - b * N;
    const float* m0 = mass + 3 * ((b * L) * N + n);
    float aI = m0[0], aU = m0[1], aT = m0[2];
    float k = 0.f;
    if (conflict) conflict[(b * L) * N + n] = 0.f;
    for (int l = 1; l < L; ++l) {
        const float* ml = mass + 3 * ((b * L + l) * N + n);
        k = ds_step(aI, aU, aT, ml[0], ml[1], ml[2]);
        if (conflict) conflict[(b * L + l) * N + n] = k;
    }
    if (fused) {
        fused[3 * i + 0] = aI;
        fused[3 * i + 1] = aU;
        fused[3 * i + 2] = aT;
    }
    prio_c[i] = priority_complement(aU, k);
}

__global__ __launch_bounds__(kThreads) void fuse_evidence_kernel(
    const float* __restrict__ e, float* __restrict__ fused, float* __restrict__ conflict,
    float* __restrict__ prio_c, int B, int L, int H, int N) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x;
    if (i >= static_cast<int64_t>(B) * N) return;
    const int64_t b = i / N, n = i - b * N;
    const float two_over_h = 2.0f / static_cast<float>(H);
    float aI = 0.f, aU = 0.f, aT = 1.f, k = 0.f;
    for (int l = 0; l < L; ++l) {
        float s1, ebar, s2;
        head_sums(e + ((b * L + l) * H) * N + n, N, H, s1, ebar, s2);
        const float rho = reliability_from_sums(s1, s2, two_over_h);
        float mI, mU, mT;
        masses_from_reliability(rho, ebar, mI, mU, mT);
        if (l == 0) {
            aI = mI;
            aU = mU;
            aT = mT;
            k = 0.f;
        } else {
            k = ds_step(aI, aU, aT, mI, mU, mT);
        }
        if (conflict) conflict[(b * L + l) * N + n] = k;
    }
    if (fused) {
        fused[3 * i + 0] = aI;
        fused[3 * i + 1] = aU;
        fused[3 * i + 2] = aT;
    }
    prio_c[i] = priority_complement(aU, k);
}

inline unsigned blocks_for(int64_t n) { return static_cast<unsigned>((n + kThreads - 1) / kThreads); }

}  // namespace

hipError_t launch_head_reliability(const Dims& d, const float* support_c, float* rho,
                                   float* pbar_c, hipStream_t st) {
    const int64_t BL = d.B * d.L;
    hipLaunchKernelGGL(head_reliability_kernel, dim3(blocks_for(BL * d.N)), dim3(kThreads), 0, st,
                       support_c, rho, pbar_c, BL, static_cast<int>(d.H), static_cast<int>(d.N));
    return hipGetLastError();
}

hipError_t launch_head_masses(const Dims& d, const float* rho, const float* pbar_c, float* mass,
                              hipStream_t st) {
    const int64_t count = d.B * d.L * d.N;
    hipLaunchKernelGGL(head_masses_kernel, dim3(blocks_for(count)), dim3(kThreads), 0, st, rho,
                       pbar_c, mass, count);
    return hipGetLastError();
}

hipError_t launch_ds_combine(const Dims& d, const float* mass, float* fused, float* conflict,
                             float* prio_c, hipStream_t st) {
    hipLaunchKernelGGL(ds_combine_kernel, dim3(blocks_for(d.B * d.N)), dim3(kThreads), 0, st, mass,
                       fused, conflict, prio_c, static_cast<int>(d.B), static_cast<int>(d.L),
                       static_cast<int>(d.N));
    return hipGetLastError();
}

hipError_t launch_fuse_evidence(const Dims& d, const float* support_c, float* fused,
                                float* conflict, float* prio_c, hipStream_t st) {
    hipLaunchKernelGGL(fuse_evidence_kernel, dim3(blocks_for(d.B * d.N)), dim3(kThreads), 0, st,
                       support_c, fused, conflict, prio_c, static_cast<int>(d.B),
                       static_cast<int>(d.L), static_cast<int>(d.H), static_cast<int>(d.N));
    return hipGetLastError();
}

}  // namespace e2s
