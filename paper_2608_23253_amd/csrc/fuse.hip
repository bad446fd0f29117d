// Evidence stages (Sec. 4.1 Eq. 10-11, Sec. 4.2 Eq. 12-19).
//
// Reliability needs two reductions over the H heads of every (image, layer, token)
// (sum e_h, then sum |e_h - ebar|).  A workgroup owns 64 consecutive tokens of one
// image and splits the heads over 4 groups of 64 threads: thread (g, t) reads heads
// g, g+4, g+8, ... of token t, so every wave load is a coalesced 256-byte row of
// [.., H, N].  The four partial sums meet in LDS and are combined in a fixed order,
// so every thread of the token holds the same sums.  The running fused mass of a
// token stays in registers across the L layers, and the next layer's supports are
// loaded while the current layer is reduced.
//
// The staged reliability kernel runs the same reduction code and the staged
// masses / Dempster kernels the same per-token arithmetic (e2s_device.h); the
// library is compiled without floating-point contraction, so e2s_fuse_evidence
// returns the same bits as the three staged calls.
#include "e2s_device.h"
#include "e2s_kernels.h"

namespace e2s {
namespace {

constexpr int kTok = 64;                 // tokens per workgroup
constexpr int kHG = 4;                   // head groups per token
constexpr int kThreads = kTok * kHG;
static_assert(kMaxHeads == kHG * 32, "head limit = 4 groups x 32 heads in registers");

template <int HPT>
__device__ __forceinline__ void load_heads(float (&v)[HPT], const float* __restrict__ e_bl,
                                           int64_t N, int n, bool ok, int hg, int H) {
#pragma unroll
    for (int i = 0; i < HPT; ++i) {
        const int h = hg + kHG * i;
        v[i] = (ok && h < H) ? e_bl[h * N + n] : 0.f;
    }
}

// Eq. 10 for one (image, layer) and the token of thread (hg, t).  red points to
// two [kHG][kTok] buffers used alternately, which lets consecutive layers share
// them with two barriers per layer.
template <int HPT>
__device__ __forceinline__ void reliability_group(const float (&v)[HPT], int H, int hg, int t,
                                                  float* red, float& rho, float& ebar) {
    float p = 0.f;
#pragma unroll
    for (int i = 0; i < HPT; ++i)
        if (hg + kHG * i < H) p += v[i];
    red[hg * kTok + t] = p;
    __syncthreads();
    const float s1 = ((red[t] + red[kTok + t]) + red[2 * kTok + t]) + red[3 * kTok + t];
    ebar = s1 / static_cast<float>(H);
    float p2 = 0.f;
#pragma unroll
    for (int i = 0; i < HPT; ++i)
        if (hg + kHG * i < H) p2 += fabsf(v[i] - ebar);
    float* red2 = red + kHG * kTok;
    red2[hg * kTok + t] = p2;
    __syncthreads();
    const float s2 = ((red2[t] + red2[kTok + t]) + red2[2 * kTok + t]) + red2[3 * kTok + t];
    rho = reliability_from_sums(s1, s2, 2.0f / static_cast<float>(H));
}

template <int HPT>
__global__ __launch_bounds__(kThreads) void head_reliability_kernel(
    const float* __restrict__ e, float* __restrict__ rho, float* __restrict__ pbar_c,
    BatchGeom bg, int tiles) {
    __shared__ float red[2 * kHG * kTok];
    const int64_t bl = blockIdx.x / tiles;        // b*L + l
    const int tile = blockIdx.x - static_cast<int>(bl) * tiles;
    const int64_t b = bl / bg.L;
    const int l = static_cast<int>(bl - b * bg.L);
    const ImageGeom ig = image_geom(bg, b);
    const int H = bg.H, N = ig.N;
    if (tile * kTok >= N) return;                 // past a smaller image's tokens (whole block)
    const int t = threadIdx.x % kTok, hg = threadIdx.x / kTok;
    const int n = tile * kTok + t;
    const bool ok = n < N;
    float v[HPT];
    load_heads(v, e + bg.L * H * ig.tok + static_cast<int64_t>(l) * H * N, N, n, ok, hg, H);
    float r, eb;
    reliability_group(v, H, hg, t, red, r, eb);
    if (hg == 0 && ok) {
        const int64_t o = bg.L * ig.tok + static_cast<int64_t>(l) * N + n;
        rho[o] = r;
        pbar_c[o] = eb;
    }
}

__global__ __launch_bounds__(256) void head_masses_kernel(
    const float* __restrict__ rho, const float* __restrict__ pbar_c, float* __restrict__ mass,
    int64_t count) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    if (i >= count) return;
    float mI, mU, mT;
    masses_from_reliability(rho[i], pbar_c[i], mI, mU, mT);
    mass[3 * i + 0] = mI;
    mass[3 * i + 1] = mU;
    mass[3 * i + 2] = mT;
}

__global__ __launch_bounds__(256) void ds_combine_kernel(
    const float* __restrict__ mass, float* __restrict__ fused, float* __restrict__ conflict,
    float* __restrict__ prio_c, int B, int L, int N) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
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

template <int HPT>
__global__ __launch_bounds__(kThreads) void fuse_evidence_kernel(
    const float* __restrict__ e, float* __restrict__ fused, float* __restrict__ conflict,
    float* __restrict__ prio_c, int L, int H, int N, int tiles) {
    __shared__ float red[2 * kHG * kTok];
    const int64_t b = blockIdx.x / tiles;
    const int tile = blockIdx.x - static_cast<int>(b) * tiles;
    const int t = threadIdx.x % kTok, hg = threadIdx.x / kTok;
    const int n = tile * kTok + t;
    const bool ok = n < N;
    const int64_t layer_stride = static_cast<int64_t>(H) * N;
    const float* eb = e + b * L * layer_stride;
    float cur[HPT], nxt[HPT];
    load_heads(cur, eb, N, n, ok, hg, H);
    float aI = 0.f, aU = 0.f, aT = 1.f, k = 0.f;
    for (int l = 0; l < L; ++l) {
        if (l + 1 < L) load_heads(nxt, eb + (l + 1) * layer_stride, N, n, ok, hg, H);
        float rho, ebar;
        reliability_group(cur, H, hg, t, red, rho, ebar);
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
        if (conflict && hg == 0 && ok) conflict[(b * L + l) * N + n] = k;
        if (l + 1 < L) {
#pragma unroll
            for (int i = 0; i < HPT; ++i) cur[i] = nxt[i];
        }
    }
    if (hg == 0 && ok) {
        const int64_t i = b * N + n;
        if (fused) {
            fused[3 * i + 0] = aI;
            fused[3 * i + 1] = aU;
            fused[3 * i + 2] = aT;
        }
        prio_c[i] = priority_complement(aU, k);
    }
}

inline unsigned blocks_for(int64_t n, int per) { return static_cast<unsigned>((n + per - 1) / per); }

template <template <int> class Launch, typename... Args>
hipError_t by_heads(int H, Args... args) {
    const int hpt = (H + kHG - 1) / kHG;
    if (hpt <= 1) return Launch<1>::run(args...);
    if (hpt <= 2) return Launch<2>::run(args...);
    if (hpt <= 4) return Launch<4>::run(args...);
    if (hpt <= 8) return Launch<8>::run(args...);
    if (hpt <= 16) return Launch<16>::run(args...);
    return Launch<32>::run(args...);
}

template <int HPT> struct RelLaunch {
    static hipError_t run(const Dims& d, const float* e, float* rho, float* pbar, hipStream_t st) {
        const int tiles = static_cast<int>((d.N + kTok - 1) / kTok);
        hipLaunchKernelGGL(head_reliability_kernel<HPT>, dim3(static_cast<unsigned>(d.B * d.L * tiles)),
                           dim3(kThreads), 0, st, e, rho, pbar, batch_geom(d), tiles);
        return hipGetLastError();
    }
};

template <int HPT> struct FuseLaunch {
    static hipError_t run(const Dims& d, const float* e, float* fused, float* conflict,
                          float* prio, hipStream_t st) {
        const int tiles = static_cast<int>((d.N + kTok - 1) / kTok);
        hipLaunchKernelGGL(fuse_evidence_kernel<HPT>, dim3(static_cast<unsigned>(d.B * tiles)),
                           dim3(kThreads), 0, st, e, fused, conflict, prio, static_cast<int>(d.L),
                           static_cast<int>(d.H), static_cast<int>(d.N), tiles);
        return hipGetLastError();
    }
};

}  // namespace

hipError_t launch_head_reliability(const Dims& d, const float* support_c, float* rho,
                                   float* pbar_c, hipStream_t st) {
    return by_heads<RelLaunch>(static_cast<int>(d.H), d, support_c, rho, pbar_c, st);
}

hipError_t launch_head_masses(const Dims& d, const float* rho, const float* pbar_c, float* mass,
                              hipStream_t st) {
    const int64_t count = d.B * d.L * d.N;
    hipLaunchKernelGGL(head_masses_kernel, dim3(blocks_for(count, 256)), dim3(256), 0, st, rho,
                       pbar_c, mass, count);
    return hipGetLastError();
}

hipError_t launch_ds_combine(const Dims& d, const float* mass, float* fused, float* conflict,
                             float* prio_c, hipStream_t st) {
    hipLaunchKernelGGL(ds_combine_kernel, dim3(blocks_for(d.B * d.N, 256)), dim3(256), 0, st, mass,
                       fused, conflict, prio_c, static_cast<int>(d.B), static_cast<int>(d.L),
                       static_cast<int>(d.N));
    return hipGetLastError();
}

hipError_t launch_fuse_evidence(const Dims& d, const float* support_c, float* fused,
                                float* conflict, float* prio_c, hipStream_t st) {
    return by_heads<FuseLaunch>(static_cast<int>(d.H), d, support_c, fused, conflict, prio_c, st);
}

}  // namespace e2s
