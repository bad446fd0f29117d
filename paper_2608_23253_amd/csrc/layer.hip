// Score and head reliability of one whole source layer per workgroup
// (Sec. 3.1 Eq. 1; Sec. 4.1 Eq. 8-10), mean-of-logits reading, one query head per
// key head.  Used by e2s_prune when a layer's supports fit in LDS.
//
// The per-head score kernel writes every support e [B, L, H, N] to HBM for the
// reliability stage to read back; interleaved with the key stream those small
// writes cost more read bandwidth than the bytes they carry.  Here one workgroup
// of up to 16 waves owns an (image, layer), keeps the H x N supports in LDS and
// writes only rho and ebar [B, L, N] (1/H of the support bytes):
//
//   1. query means: wave w computes qbar of heads w, w + 16, ... into LDS;
//   2. logits: the layer's key rows are cut into units of 2 batches (64 rows for
//      bf16, d = 128) in head-major order; a wave takes its first unit statically
//      (its loads overlap step 1) and every further unit from an LDS counter,
//      claiming the next unit and requesting its rows before it finishes the
//      current one.  Waves of a workgroup are served unevenly by the memory
//      system; taking work in small units keeps all of them streaming until the
//      layer is done instead of leaving the fastest idle;
//   3. the wave that completes the last unit of a head (an LDS counter per head)
//      runs that head's softmax and supports at once, while the other waves keep
//      streaming;
//   4. after one barrier, Eq. 10 per token, four threads per token (one per head
//      group).
//
// Every value is computed as by the per-head kernel (same functions, same lane
// mapping per row and per head, the evidence kernels' reliability order), so
// e2s_prune returns the same bits through either path.
#include <algorithm>

#include "e2s_device.h"
#include "e2s_kernels.h"
#include "score_common.h"

namespace e2s {
namespace {

constexpr int kMaxWaves = 16;
constexpr size_t kLdsLimit = 150 * 1024;
constexpr int kMaxLayerHeads = 128;

// quad_perm broadcasts of lanes 0..3 of each quad
constexpr int kQuadLane0 = 0x00, kQuadLane1 = 0x55, kQuadLane2 = 0xAA, kQuadLane3 = 0xFF;

// ((p0 + p1) + p2) + p3 of the four lanes of a quad, in every lane of the quad.
__device__ __forceinline__ float quad_sum_in_order(float p) {
    return ((dpp<kQuadLane0>(p) + dpp<kQuadLane1>(p)) + dpp<kQuadLane2>(p)) + dpp<kQuadLane3>(p);
}

__device__ __forceinline__ int wave_uniform(int v) { return __builtin_amdgcn_readfirstlane(v); }

template <typename T, int D>
__global__ __launch_bounds__(kMaxWaves * kWave) void layer_evidence_kernel(
    const T* __restrict__ q, const T* __restrict__ k, float* __restrict__ rho_out,
    float* __restrict__ pbar_out, BatchGeom bg, float scale) {
    using G = WaveRows<T, D>;
    constexpr int CR = 2 * G::BATCH;      // key rows per unit
    const int64_t b = blockIdx.x / bg.L;  // workgroup (b, l)
    const int l = static_cast<int>(blockIdx.x - b * bg.L);
    const ImageGeom ig = image_geom(bg, b);
    const int H = bg.H, NT = ig.NT, N = ig.N;
    const float qscale = mean_query_scale(scale, NT);
    extern __shared__ float smem[];
    float* buf = smem;                    // [H][N] logits, then supports
    float* qbar = smem + H * N;           // [H][D]
    __shared__ int s_next;                // next unit to hand out
    __shared__ int s_done[kMaxLayerHeads];   // finished units per head

    const int tid = threadIdx.x, nthreads = blockDim.x;
    const int wave = tid / kWave, lane = tid % kWave, nwaves = nthreads / kWave;
    const int wrow = lane / G::LPR, wl = lane % G::LPR;
    const int nch = (N + CR - 1) / CR, units = H * nch;
    const int64_t qld = query_ld(bg), kld = key_ld(bg);
    // key rows of head h, offset by this lane's 8 elements (one key head per head)
    auto key_head = [&](int h) { return key_rows(k, bg, ig, b, l, h) + wl * 8; };
    float* rho_l = rho_out + bg.L * ig.tok + static_cast<int64_t>(l) * N;
    float* pbar_l = pbar_out + bg.L * ig.tok + static_cast<int64_t>(l) * N;

    if (tid == 0) s_next = nwaves;
    for (int h = tid; h < H; h += nthreads) s_done[h] = 0;

    // Key requests are unconditional (unit ids clamped, rows clamped to N - 1 by
    // load_key_batch; surplus rows are never used), so every path through the loop
    // has the same loads in flight and the compiler's wait before a batch's first
    // use leaves the later batch's loads pending.
    int u = wave;                         // first unit; its rows load during step 1
    Packet<T> ka[G::KU], kb[G::KU];
    {
        const int uc = min(u, units - 1), h = uc / nch;
        load_key_batch<T, D>(ka, key_head(h), (uc - h * nch) * CR, wrow, N, kld);
    }

    // ---- 1. query means ---------------------------------------------------------
    for (int h = wave; h < H; h += nwaves) {
        float qb[8];
        wave_query_mean<T, D>(query_rows(q, bg, ig, b, l, h) + wl * 8, NT, wrow, qscale, qb, qld);
        if (wrow == 0) {
#pragma unroll
            for (int m = 0; m < 8; ++m) qbar[h * D + wl * 8 + m] = qb[m];
        }
    }
    __syncthreads();

    // ---- 2, 3. logits in units; each head's softmax by its last unit's wave ----
    while (u < units) {
        int un = 0;
        if (lane == 0) un = atomicAdd(&s_next, 1);
        un = wave_uniform(un);
        const int h = u / nch, base = (u - h * nch) * CR;
        const T* kh = key_head(h);
        float* a = buf + h * N;
        float qb[8];
#pragma unroll
        for (int m = 0; m < 8; ++m) qb[m] = qbar[h * D + wl * 8 + m];
        const bool second = base + G::BATCH < N;
        load_key_batch<T, D>(kb, kh, base + G::BATCH, wrow, N, kld);
        key_batch_logits<T, D>(ka, qb, a, base, wrow, wl, N);
        {
            const int uc = min(un, units - 1), hn = uc / nch;
            load_key_batch<T, D>(ka, key_head(hn), (uc - hn * nch) * CR, wrow, N, kld);
        }
        if (second) key_batch_logits<T, D>(kb, qb, a, base + G::BATCH, wrow, wl, N);

        // publish this unit's logits; the wave completing the head finishes it
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
        int done = 0;
        if (lane == 0) done = atomicAdd(&s_done[h], 1);
        done = wave_uniform(done);
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
        if (done == nch - 1)
            wave_softmax(a, N, lane,
                         [&](int n, float dc, bool near) { a[n] = support_from_centred(dc, near); });
        u = un;
    }
    __syncthreads();

    // ---- 4. reliability per token (Eq. 10) --------------------------------------
    // thread 4n + g sums heads g, g + 4, ...; quads are whole because 4 | nthreads
    const float two_over_h = 2.0f / static_cast<float>(H);
    for (int i = tid; i < 4 * N; i += nthreads) {
        const int n = i >> 2, g = i & 3;
        float p = 0.f;
        for (int hh = g; hh < H; hh += 4) p += buf[hh * N + n];
        const float s1 = quad_sum_in_order(p);
        const float ebar = s1 / static_cast<float>(H);
        float d = 0.f;
        for (int hh = g; hh < H; hh += 4) d += fabsf(buf[hh * N + n] - ebar);
        const float s2 = quad_sum_in_order(d);
        if (g == 0) {
            rho_l[n] = reliability_from_sums(s1, s2, two_over_h);
            pbar_l[n] = ebar;
        }
    }
}

size_t layer_lds(const Dims& d) {
    return (static_cast<size_t>(d.H) * d.N + static_cast<size_t>(d.H) * d.D) * sizeof(float);
}

template <typename T, int D>
hipError_t launch_layer(const Dims& d, float scale, const void* q, const void* k, float* rho,
                        float* pbar, hipStream_t st) {
    const size_t lds = layer_lds(d);
    auto kern = layer_evidence_kernel<T, D>;
    if (lds > 64 * 1024) {
        hipError_t err = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                             hipFuncAttributeMaxDynamicSharedMemorySize,
                                             static_cast<int>(lds));
        if (err != hipSuccess) return err;
    }
    const int waves = static_cast<int>(std::min<int64_t>(d.H, kMaxWaves));
    hipLaunchKernelGGL(kern, dim3(static_cast<unsigned>(d.B * d.L)), dim3(waves * kWave), lds, st,
                       static_cast<const T*>(q), static_cast<const T*>(k), rho, pbar,
                       batch_geom(d), scale);
    return hipGetLastError();
}

}  // namespace

bool layer_evidence_fits(const Dims& d) {
    return d.group == 1 && d.H <= kMaxLayerHeads && layer_lds(d) <= kLdsLimit;
}

hipError_t launch_layer_evidence(const Dims& d, int dtype, float scale, const void* q,
                                 const void* k, float* rho, float* pbar_c, hipStream_t stream) {
    if (dtype == E2S_DTYPE_BF16) {
        if (d.D == 128) return launch_layer<uint16_t, 128>(d, scale, q, k, rho, pbar_c, stream);
        return launch_layer<uint16_t, 64>(d, scale, q, k, rho, pbar_c, stream);
    }
    if (dtype == E2S_DTYPE_F16) {
        if (d.D == 128) return launch_layer<_Float16, 128>(d, scale, q, k, rho, pbar_c, stream);
        return launch_layer<_Float16, 64>(d, scale, q, k, rho, pbar_c, stream);
    }
    if (d.D == 128) return launch_layer<float, 128>(d, scale, q, k, rho, pbar_c, stream);
    return launch_layer<float, 64>(d, scale, q, k, rho, pbar_c, stream);
}

}  // namespace e2s
