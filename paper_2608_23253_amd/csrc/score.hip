// Score stage: text->visual attention per head, normalized over the visual tokens
// and mapped to a centred support e = p - 1/2 (Sec. 3.1 Eq. 1; Sec. 4.1 Eq. 8-9).
//
// Mean-of-logits reading.  Eq. 1 averages Q_t.K_n / sqrt(d) over the text queries;
// by linearity that equals (mean_t Q_t).K_n / sqrt(d), so the stage is a stream of
// the key tensor against one query vector per head: an HBM-bound matrix-vector
// product.
//
// One query head per key head (multi-head attention): one wave owns one (image,
// layer, head) unit and runs all steps below on its own, without workgroup
// barriers (wave_head: the query mean in registers, the key rows streamed with
// the next batch in flight, the softmax reduced across the wave).
//
// Grouped-query attention: one workgroup owns one (image, layer, key head) unit
// (and a chunk of at most 8 of the query heads that share that key head), so every
// key row is read from HBM exactly once:
//
//   A  qbar_h = (scale / N_T) * sum_t Q[h, t, :]             (fp32, LDS); the first
//      key rows are already being loaded while this runs, and all heads of the
//      workgroup are reduced before a single barrier
//   B  a[h, n] = qbar_h . K[n, :]                             (fp32, LDS)
//      16 lanes (d = 128) or 8 lanes (d = 64) share one key row; each lane loads
//      16 contiguous bytes, so a wave-wide load covers 1 KB of contiguous keys;
//      the partial dot products are summed with DPP row operations.
//   C  per head (one wave per head, or the whole workgroup when it owns a single
//      head): m = max_n a, S = sum_n exp(a_n - m),
//      E = sum_n expm1(a_n - m) = S - N, and L = log(S / N)
//   D  u_n = N r_n - 1 = expm1(a_n - m - L),  e_n = u_n / (2 (2 + u_n)) = p_n - 1/2,
//      r_n = exp(a_n - m - L) / N.
//
// The supports are written with non-temporal stores: the key stream reads at
// ~7 TB/s on its own, and cached write-backs interleaved with it cost more
// read bandwidth than the bytes they carry.
//
// Steps C-D carry the softmax in log-sum-exp-centred form.  Near uniform attention
// (a_n - m = O(1e-3), the regime of Gaussian keys at the 1/sqrt(d) scale) the
// naive N r - 1 loses ~10 bits to cancellation; expm1 of the centred logit keeps
// full relative precision.  L itself is taken from whichever sum is exact in the
// current regime: log1p(E / N) when S > N/2 (E, a sum of small non-positive
// terms, has no cancellation), log(S / N) when attention is peaked (S is then a
// sum dominated by a few O(1) positive terms).
#include "e2s_device.h"
#include "e2s_kernels.h"
#include "score_common.h"

#include <algorithm>
#include <cmath>

namespace e2s {
namespace {

constexpr int kThreads = kGroupThreads;     // one 4-wave reduction group
constexpr int kWaves = kGroupWaves;
constexpr int kMaxChunk = 8;                  // query heads per workgroup
constexpr int kLdsBudget = 96 * 1024;         // bytes of dynamic LDS per workgroup
constexpr int kUnroll = 8;                    // key rows in flight per lane

template <typename T, int D, int RC>
__global__ __launch_bounds__(kThreads) void score_mean_logit_kernel(
    const T* __restrict__ q, const T* __restrict__ k, float* __restrict__ e_out,
    float* __restrict__ r_out, int H, int Hkv, int NT, int N, int group, int chunk,
    int nchunks, float qscale) {
    constexpr int LPR = D / 8;            // lanes per row (8 elements per lane)
    constexpr int RPW = kWave / LPR;      // rows per wave-wide load
    constexpr int STEP = kWaves * RPW;    // rows per block-wide load

    extern __shared__ float smem[];
    float* qbar = smem;                   // [RC][D]
    float* part = qbar + RC * D;          // [RC][kWaves][D]
    float* logits = part + RC * kWaves * D;   // [rc][N]

    const int unit = blockIdx.x / nchunks;        // (b*L + l)*Hkv + g
    const int ci = blockIdx.x - unit * nchunks;
    const int g = unit % Hkv;
    const int64_t bl = unit / Hkv;                // b*L + l
    const int hq0 = g * group + ci * chunk;       // first query head of this chunk
    const int rc = min(chunk, group - ci * chunk);
    const int tid = threadIdx.x;
    const int wave = tid / kWave, lane = tid % kWave;
    const int wrow = lane / LPR, wl = lane % LPR;
    const T* kg = k + static_cast<int64_t>(unit) * N * D + wl * 8;

    // Key rows past N are clamped to row N-1 (loads stay in bounds and branch-free);
    // their products are discarded.
    auto load_keys = [&](Packet<T> (&pk)[kUnroll], int base) {
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const int n = min(base + wrow + u * STEP, N - 1);
            load_packet(pk[u], kg + static_cast<int64_t>(n) * D);
        }
    };

    // The first key rows do not depend on the query mean: start loading them now
    // so that their latency overlaps phase A.
    Packet<T> pk[kUnroll];
    load_keys(pk, wave * RPW);

    // ---- A: mean query per head (one barrier for all heads) -----------------
    // Wave w sums rows w*RPW + wrow + i*STEP of every head, lane wl holding 8
    // consecutive dims; the RPW row groups of a wave meet by shuffles, the waves
    // in LDS.
    {
        for (int j = 0; j < rc; ++j) {
            float acc[8];
            query_partial<T, D>(q + ((bl * H + hq0 + j) * NT) * D + wl * 8, NT, wave, wrow, acc);
            if (wrow == 0) {
#pragma unroll
                for (int m = 0; m < 8; ++m) part[(j * kWaves + wave) * D + wl * 8 + m] = acc[m];
            }
        }
        __syncthreads();
        for (int i = tid; i < rc * D; i += kThreads) {
            const int j = i / D, dd = i - j * D;
            qbar[i] = query_mean(part + j * kWaves * D + dd, D, qscale);
        }
        __syncthreads();
    }

    // ---- B: logits a[h, n] --------------------------------------------------
    float qb[RC][8];
#pragma unroll
    for (int j = 0; j < RC; ++j)
#pragma unroll
        for (int m = 0; m < 8; ++m) qb[j][m] = (j < rc) ? qbar[j * D + wl * 8 + m] : 0.f;

    for (int base = wave * RPW; base < N; base += STEP * kUnroll) {
        if (base != wave * RPW) load_keys(pk, base);
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const int n = base + wrow + u * STEP;
            float x[8];
            unpack(pk[u], x);
#pragma unroll
            for (int j = 0; j < RC; ++j) {
                if (j < rc) {
                    const float s = row_logit<LPR>(qb[j], x);
                    if (wl == 0 && n < N) logits[j * N + n] = s;
                }
            }
        }
    }
    __syncthreads();

    // ---- C, D: centred softmax and support -----------------------------------
    const float fN = static_cast<float>(N);
    if (rc == 1) {
        // a single head: the whole workgroup shares it
        __shared__ float red[16];
        float* a = logits;
        bool near;
        const float lse = softmax_centre(a, N, tid, red, true, near);
        const int64_t row = (bl * H + hq0) * static_cast<int64_t>(N);
        float* eo = e_out + row;
        float* ro = r_out ? r_out + row : nullptr;
        for (int n = tid; n < N; n += kThreads) {
            const float dc = a[n] - lse;
            __builtin_nontemporal_store(support_from_centred(dc, near), eo + n);
            if (ro) ro[n] = expf(dc) / fN;
        }
        return;
    }
    // several heads: one wave per head
    for (int j = wave; j < rc; j += kWaves) {
        float* a = logits + j * N;
        float m = -INFINITY;
        for (int n = lane; n < N; n += kWave) m = fmaxf(m, a[n]);
        m = wave_max(m);
        float E = 0.f, S = 0.f;
        for (int n = lane; n < N; n += kWave) {
            const float d = a[n] - m;
            a[n] = d;
            E += expm1f(d);
            S += expf(d);
        }
        E = wave_sum(E);
        S = wave_sum(S);
        const float lse = log_mean_exp(E, S, fN);
        const int64_t row = (bl * H + hq0 + j) * static_cast<int64_t>(N);
        float* eo = e_out + row;
        float* ro = r_out ? r_out + row : nullptr;
        for (int n = lane; n < N; n += kWave) {
            const float dc = a[n] - lse;
            __builtin_nontemporal_store(support_from_centred(dc, false), eo + n);
            if (ro) ro[n] = expf(dc) / fN;
        }
    }
}

template <typename T, int D, int RC>
hipError_t launch_ml(const Dims& d, float qscale, const void* q, const void* k, float* e,
                     float* r, int chunk, int nchunks, hipStream_t st) {
    const size_t lds = (static_cast<size_t>(RC) * D * (1 + kWaves) +
                        static_cast<size_t>(chunk) * d.N) * sizeof(float);
    auto kern = score_mean_logit_kernel<T, D, RC>;
    if (lds > 64 * 1024) {
        hipError_t err = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                             hipFuncAttributeMaxDynamicSharedMemorySize,
                                             static_cast<int>(lds));
        if (err != hipSuccess) return err;
    }
    const int64_t blocks = d.B * d.L * d.Hkv * nchunks;
    hipLaunchKernelGGL(kern, dim3(static_cast<unsigned>(blocks)), dim3(kThreads), lds, st,
                       static_cast<const T*>(q), static_cast<const T*>(k), e, r,
                       static_cast<int>(d.H), static_cast<int>(d.Hkv), static_cast<int>(d.NT),
                       static_cast<int>(d.N), static_cast<int>(d.group), chunk, nchunks, qscale);
    return hipGetLastError();
}

// One query head per key head: one wave per (image, layer, head) unit, no
// workgroup barrier (wave_head); the workgroup only packs up to 4 independent
// waves together.
template <typename T, int D>
__global__ __launch_bounds__(kThreads) void score_wave_kernel(
    const T* __restrict__ q, const T* __restrict__ k, float* __restrict__ e_out,
    float* __restrict__ r_out, int64_t units, int NT, int N, float qscale) {
    extern __shared__ float smem[];
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int64_t unit = static_cast<int64_t>(blockIdx.x) * (blockDim.x / kWave) + wave;
    if (unit >= units) return;
    float* a = smem + wave * N;
    float* eo = e_out + unit * N;
    float* ro = r_out ? r_out + unit * N : nullptr;
    const float fN = static_cast<float>(N);
    wave_head<T, D>(q + unit * NT * D, k + unit * N * D, NT, N, qscale, a, lane,
                    [&](int n, float dc, bool near) {
                        __builtin_nontemporal_store(support_from_centred(dc, near), eo + n);
                        if (ro) ro[n] = expf(dc) / fN;
                    });
}

template <typename T, int D>
hipError_t launch_wave(const Dims& d, float qscale, const void* q, const void* k, float* e,
                       float* r, hipStream_t st) {
    const int64_t per_wave = d.N * static_cast<int64_t>(sizeof(float));
    const int wpg = static_cast<int>(std::clamp<int64_t>(kLdsBudget / per_wave, 1, kWaves));
    const int64_t units = d.B * d.L * d.H;
    const int64_t blocks = (units + wpg - 1) / wpg;
    const size_t lds = static_cast<size_t>(wpg * per_wave);
    auto kern = score_wave_kernel<T, D>;
    if (lds > 64 * 1024) {
        hipError_t err = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                             hipFuncAttributeMaxDynamicSharedMemorySize,
                                             static_cast<int>(lds));
        if (err != hipSuccess) return err;
    }
    hipLaunchKernelGGL(kern, dim3(static_cast<unsigned>(blocks)), dim3(wpg * kWave), lds, st,
                       static_cast<const T*>(q), static_cast<const T*>(k), e, r, units,
                       static_cast<int>(d.NT), static_cast<int>(d.N), qscale);
    return hipGetLastError();
}

template <typename T, int D>
hipError_t dispatch_rc(const Dims& d, float qscale, const void* q, const void* k, float* e,
                       float* r, hipStream_t st) {
    if (d.group == 1) return launch_wave<T, D>(d, qscale, q, k, e, r, st);
    const int64_t fixed = static_cast<int64_t>(kMaxChunk) * D * (1 + kWaves) * 4;
    int64_t fit = (kLdsBudget - fixed) / (d.N * 4);
    if (fit < 1) fit = 1;
    int chunk = static_cast<int>(std::min<int64_t>({d.group, kMaxChunk, fit}));
    const int nchunks = static_cast<int>((d.group + chunk - 1) / chunk);
    chunk = static_cast<int>((d.group + nchunks - 1) / nchunks);  // balance the chunks
    if (chunk <= 1) return launch_ml<T, D, 1>(d, qscale, q, k, e, r, chunk, nchunks, st);
    if (chunk <= 2) return launch_ml<T, D, 2>(d, qscale, q, k, e, r, chunk, nchunks, st);
    if (chunk <= 4) return launch_ml<T, D, 4>(d, qscale, q, k, e, r, chunk, nchunks, st);
    return launch_ml<T, D, 8>(d, qscale, q, k, e, r, chunk, nchunks, st);
}

}  // namespace

hipError_t launch_score_mean_logit(const Dims& d, int dtype, float scale, const void* q,
                                   const void* k, float* support_c, float* r_opt,
                                   hipStream_t stream) {
    const float qscale = static_cast<float>(static_cast<double>(scale) / static_cast<double>(d.NT));
    if (dtype == E2S_DTYPE_BF16) {
        if (d.D == 128)
            return dispatch_rc<uint16_t, 128>(d, qscale, q, k, support_c, r_opt, stream);
        return dispatch_rc<uint16_t, 64>(d, qscale, q, k, support_c, r_opt, stream);
    }
    if (d.D == 128) return dispatch_rc<float, 128>(d, qscale, q, k, support_c, r_opt, stream);
    return dispatch_rc<float, 64>(d, qscale, q, k, support_c, r_opt, stream);
}

}  // namespace e2s
