// Score stage: text->visual attention per head, normalized over the visual tokens
// and mapped to a centred support e = p - 1/2 (Sec. 3.1 Eq. 1; Sec. 4.1 Eq. 8-9).
//
// Mean-of-logits reading.  Eq. 1 averages Q_t.K_n / sqrt(d) over the text queries;
// by linearity that equals (mean_t Q_t).K_n / sqrt(d), so the stage is a stream of
// the key tensor against one query vector per head: an HBM-bound matrix-vector
// product.
//
// Per head, in every kernel (score_common.h):
//   qbar_h = (scale / N_T) * sum_t Q[h, t, :]                       (fp32)
//   a[h, n] = qbar_h . K[n, :]: 16 lanes (d = 128) or 8 lanes (d = 64) share one
//      key row, each loading 16 contiguous bytes, so a wave-wide load covers 1 KB
//      of contiguous keys; the partial dot products are summed with DPP row ops
//   m = max_n a, S = sum_n exp(a_n - m), E = sum_n expm1(a_n - m) = S - N,
//      L = log(S / N)
//   u_n = N r_n - 1 = expm1(a_n - m - L),  e_n = u_n / (2 (2 + u_n)) = p_n - 1/2,
//      r_n = exp(a_n - m - L) / N.
//
// One query head per key head (multi-head attention): one wave owns one (image,
// layer, head) unit and runs all steps on its own, without workgroup barriers
// (wave_head).  Grouped-query attention: one workgroup owns one (image, layer,
// key head) unit and a chunk of the query heads sharing it, so every key row is
// read from HBM once per chunk; with bf16 keys the logits of the chunk's heads are
// one matrix-core product per 16 keys (score_group_mfma_kernel), with fp32 keys a
// dot product per head (score_group_kernel).
//
// The supports are written with non-temporal stores: the key stream reads at
// ~7 TB/s on its own, and cached write-backs interleaved with it cost more
// read bandwidth than the bytes they carry.
//
// The softmax is carried in log-sum-exp-centred form.  Near uniform attention
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
#include <type_traits>

namespace e2s {
namespace {

constexpr int kThreads = 256;                 // one-head-per-key-head kernel: 4 waves
constexpr int kWaves = kThreads / kWave;
constexpr int kGroupKernelThreads = 512;      // grouped-query kernel: 8 waves
constexpr int kMaxChunk = 8;                  // query heads per grouped-query workgroup
constexpr int kLdsBudget = 96 * 1024;         // bytes of dynamic LDS per workgroup

// Grouped-query attention: one workgroup of 8 waves owns one (image, layer, key
// head) unit and a chunk of at most HC of the query heads sharing that key head,
// so every key row is read from HBM once per chunk:
//   1. wave j computes the query mean of head j of the chunk (wave_query_mean)
//      into LDS; all waves already request their first key rows;
//   2. the waves split the key rows in batches; each row gives the logits of every
//      head of the chunk (row_logit), written to LDS;
//   3. wave j runs head j's softmax and supports (wave_softmax).
// Per head the arithmetic is that of the one-head-per-key-head kernels.
template <typename T, int D, int HC, bool GLOBAL>
__global__ __launch_bounds__(kGroupKernelThreads) void score_group_kernel(
    const T* __restrict__ q, const T* __restrict__ k, float* __restrict__ e_out,
    float* __restrict__ r_out, BatchGeom bg, int group, int hchunk, int nchunks, float scale) {
    using G = WaveRows<T, D>;
    constexpr int KU = G::KU / 2;         // rows per lane per batch (registers: HC q-means)
    constexpr int BATCH = KU * G::RPW;
    constexpr int NW = kGroupKernelThreads / kWave;
    const int64_t unit = blockIdx.x / nchunks;    // (b*L + l)*Hkv + g
    const int ci = static_cast<int>(blockIdx.x - unit * nchunks);
    const int64_t b = unit / (bg.L * bg.Hkv);
    const int lkv = static_cast<int>(unit - b * bg.L * bg.Hkv);   // l*Hkv + g
    const int l = lkv / bg.Hkv, g = lkv - l * bg.Hkv;
    const ImageGeom ig = image_geom(bg, b);
    const int H = bg.H, NT = ig.NT, N = ig.N;
    const float qscale = mean_query_scale(scale, NT);
    extern __shared__ float smem[];
    const int h0 = g * group + ci * hchunk;
    const int nh = min(hchunk, group - ci * hchunk);
    const int64_t erow = bg.L * bg.H * ig.tok + static_cast<int64_t>(l) * H * N;
    float* qbar = smem;                   // [hchunk][D]
    // [hchunk][N] logits: LDS, or (GLOBAL) the chunk's output rows, overwritten
    float* a = GLOBAL ? e_out + erow + static_cast<int64_t>(h0) * N : smem + hchunk * D;

    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int wrow = lane / G::LPR, wl = lane % G::LPR;
    const T* kg = key_rows(k, bg, ig, b, l, g) + wl * 8;
    const int64_t qld = query_ld(bg), kld = key_ld(bg);

    Packet<T> ka[KU], kb[KU];
    load_key_batch<T, D>(ka, kg, wave * BATCH, wrow, N, kld);
    for (int j = wave; j < nh; j += NW) {
        float qb[8];
        wave_query_mean<T, D>(query_rows(q, bg, ig, b, l, h0 + j) + wl * 8, NT, wrow, qscale, qb,
                              qld);
        if (wrow == 0) {
#pragma unroll
            for (int m = 0; m < 8; ++m) qbar[j * D + wl * 8 + m] = qb[m];
        }
    }
    __syncthreads();

    float qb[HC][8];
#pragma unroll
    for (int j = 0; j < HC; ++j)
#pragma unroll
        for (int m = 0; m < 8; ++m) qb[j][m] = j < nh ? qbar[j * D + wl * 8 + m] : 0.f;
    auto consume = [&](const Packet<T> (&p)[KU], int base) {
#pragma unroll
        for (int u = 0; u < KU; ++u) {
            float x[8];
            unpack(p[u], x);
            const int n = base + wrow + u * G::RPW;
#pragma unroll
            for (int j = 0; j < HC; ++j) {
                if (j < nh) {
                    const float sj = row_logit<G::LPR>(qb[j], x);
                    if (wl == 0 && n < N) a[static_cast<int64_t>(j) * N + n] = sj;
                }
            }
        }
    };
    constexpr int STRIDE = NW * BATCH;
    for (int base = wave * BATCH; base < N; base += 2 * STRIDE) {
        if (base + STRIDE < N) load_key_batch<T, D>(kb, kg, base + STRIDE, wrow, N, kld);
        consume(ka, base);
        if (base + STRIDE >= N) break;
        if (base + 2 * STRIDE < N) load_key_batch<T, D>(ka, kg, base + 2 * STRIDE, wrow, N, kld);
        consume(kb, base + STRIDE);
    }
    __syncthreads();

    for (int j = wave; j < nh; j += NW) {
        const int64_t row = erow + static_cast<int64_t>(h0 + j) * N;
        wave_softmax_store(a + static_cast<int64_t>(j) * N, N, lane, e_out + row,
                           r_out ? r_out + row : nullptr);
    }
}

// Grouped-query attention with bf16 keys: the logits of every head of a chunk
// against a 16-row key tile form a (16 x d) . (d x heads) product, which runs on
// the matrix cores (v_mfma_f32_16x16x32_bf16: 16 keys x 16 query heads per tile).
// The fp32 query means are split exactly into three bf16 terms
// (hi + mid + lo = qbar: each term takes the next 8 significant bits, 24 in all),
// kept in LDS, and the three products are accumulated in fp32, so a logit carries
// the same information as the fp32 dot product of the vector kernels; only the
// rounding of the sums differs.  Steps 1 and 3 are those of score_group_kernel.
//
// The stage streams Q and K with no reuse, and a launch has few workgroups (one
// per (image, layer, key head)), so what bounds it is the bytes each wave keeps
// in flight: up to kQueryRows query rows per lane in step 1 (with the first
// kTilesEarly key tiles already requested), then kTilesInFlight key tiles, a
// tile's registers being refilled with the tile kTilesInFlight positions ahead as
// soon as its products are issued.
constexpr int kMfmaMaxChunk = 16;             // query heads per MFMA tile (B columns)
constexpr int kTilesInFlight = 4;
constexpr int kTilesEarly = 2;
constexpr int kQueryRows = 8;

// MFMA operand layout (k = 32 per step): lane (lr, lg) = (lane % 16, lane / 16)
// supplies row lr and elements 8 lg .. 8 lg + 7 of the step, i.e. head dims
// 32 s + 8 lg .. + 7 of step s in both operands, so one wave-wide key load reads 64
// contiguous bytes of each of 16 rows.
// Two workgroups per CU (at most 128 VGPRs): a launch has about two per CU.
template <int D, bool GLOBAL>
__global__ __launch_bounds__(kGroupKernelThreads, 2) void score_group_mfma_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k, float* __restrict__ e_out,
    float* __restrict__ r_out, BatchGeom bg, int group, int hchunk, int nchunks, float scale) {
    const int64_t unit = blockIdx.x / nchunks;    // (b*L + l)*Hkv + g
    const int ci = static_cast<int>(blockIdx.x - unit * nchunks);
    const int64_t b = unit / (bg.L * bg.Hkv);
    const int lkv = static_cast<int>(unit - b * bg.L * bg.Hkv);   // l*Hkv + g
    const int l = lkv / bg.Hkv, g = lkv - l * bg.Hkv;
    const ImageGeom ig = image_geom(bg, b);
    const int H = bg.H, NT = ig.NT, N = ig.N;
    const float qscale = mean_query_scale(scale, NT);
    constexpr int NS = D / 32;            // MFMA steps per tile
    constexpr int P = kTilesInFlight;
    constexpr int NW = kGroupKernelThreads / kWave;
    constexpr int BS = D + 8;             // padded row of the split query means
    extern __shared__ __align__(16) float smem_mfma[];
    uint16_t* bsplit = reinterpret_cast<uint16_t*>(smem_mfma);   // [3][16][BS] bf16 bits
    float* qbar = smem_mfma + 3 * 16 * BS / 2;                    // [hchunk][D]
    const int h0 = g * group + ci * hchunk;
    const int nh = min(hchunk, group - ci * hchunk);
    const int64_t erow = bg.L * bg.H * ig.tok + static_cast<int64_t>(l) * H * N;
    // [hchunk][N] logits: LDS (rows 16-byte aligned if 4 | N), or (GLOBAL) the
    // chunk's output rows, overwritten in place
    float* a = GLOBAL ? e_out + erow + static_cast<int64_t>(h0) * N : qbar + hchunk * D;
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int lr = lane % 16, lg = lane / 16;
    const uint16_t* kg = key_rows(k, bg, ig, b, l, g) + 8 * lg;
    const int64_t qld = query_ld(bg), kld = key_ld(bg);
    const int tiles = (N + 15) / 16;
    const int cnt = wave < tiles ? (tiles - wave + NW - 1) / NW : 0;   // this wave's tiles

    bf16x8 kt[P][NS];
    auto load_tile = [&](bf16x8 (&f)[NS], int i) {
        const int row = min((wave + i * NW) * 16 + lr, N - 1);
        const uint16_t* src = kg + static_cast<int64_t>(row) * kld;
#pragma unroll
        for (int s = 0; s < NS; ++s)
            f[s] = __builtin_nontemporal_load(reinterpret_cast<const bf16x8*>(src + 32 * s));
    };
#pragma unroll
    for (int p = 0; p < kTilesEarly; ++p)
        if (p < cnt) load_tile(kt[p], p);

    // ---- 1. query means, split into bf16 terms ------------------------------------
    {
        using G = WaveRows<uint16_t, D>;
        const int wrow = lane / G::LPR, wl = lane % G::LPR;
        for (int j = wave; j < nh; j += NW) {
            float qb[8];
            wave_query_mean<uint16_t, D, kQueryRows>(
                query_rows(q, bg, ig, b, l, h0 + j) + wl * 8, NT, wrow, qscale, qb, qld);
            if (wrow == 0) {
#pragma unroll
                for (int m = 0; m < 8; ++m) qbar[j * D + wl * 8 + m] = qb[m];
            }
        }
    }
    __syncthreads();
    for (int idx = threadIdx.x; idx < 16 * D; idx += kGroupKernelThreads) {
        const int hh = idx / D, dd = idx - hh * D;
        uint16_t hi, mid, lo;
        split_bf16x3(hh < nh ? qbar[hh * D + dd] : 0.f, hi, mid, lo);
        bsplit[hh * BS + dd] = hi;
        bsplit[(16 + hh) * BS + dd] = mid;
        bsplit[(32 + hh) * BS + dd] = lo;
    }
#pragma unroll
    for (int p = kTilesEarly; p < P; ++p)
        if (p < cnt) load_tile(kt[p], p);
    __syncthreads();

    // ---- 2. logits of every head of the chunk, 16 keys per tile ----------------
    const uint16_t* bq = bsplit + lr * BS + 8 * lg;
    const bool vec_store = !GLOBAL && (N & 3) == 0;
    for (int i0 = 0; i0 < cnt; i0 += P) {
#pragma unroll
        for (int p = 0; p < P; ++p) {
            const int i = i0 + p;
            if (i < cnt) {
                const f32x4 z = split_tile_logits<NS>(kt[p], bq, bq + 16 * BS, bq + 32 * BS);
                if (i + P < cnt) load_tile(kt[p], i + P);
                // lane (lr, lg): keys 4 lg + r of the tile against head lr
                const int key0 = (wave + i * NW) * 16 + 4 * lg;
                if (lr < nh) {
                    float* dst = a + static_cast<int64_t>(lr) * N + key0;
                    if (vec_store && key0 + 3 < N) {
                        *reinterpret_cast<f32x4*>(dst) = z;
                    } else {
#pragma unroll
                        for (int r = 0; r < 4; ++r)
                            if (key0 + r < N) dst[r] = z[r];
                    }
                }
            }
        }
    }
    __syncthreads();

    // ---- 3. softmax and supports per head ----------------------------------------
    for (int j = wave; j < nh; j += NW) {
        const int64_t row = erow + static_cast<int64_t>(h0 + j) * N;
        wave_softmax_store(a + static_cast<int64_t>(j) * N, N, lane, e_out + row,
                           r_out ? r_out + row : nullptr);
    }
}

template <int D, bool GLOBAL>
hipError_t launch_group_mfma(const Dims& d, float scale, const void* q, const void* k, float* e,
                             float* r, int hchunk, hipStream_t st) {
    const int nchunks = static_cast<int>((d.group + hchunk - 1) / hchunk);
    const size_t lds = 3 * 16 * (D + 8) * sizeof(uint16_t) +
                       static_cast<size_t>(hchunk) * (D + (GLOBAL ? 0 : d.N)) * sizeof(float);
    auto kern = score_group_mfma_kernel<D, GLOBAL>;
    if (lds > 64 * 1024) {
        hipError_t err = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                             hipFuncAttributeMaxDynamicSharedMemorySize,
                                             static_cast<int>(lds));
        if (err != hipSuccess) return err;
    }
    const int64_t blocks = d.B * d.L * d.Hkv * nchunks;
    hipLaunchKernelGGL(kern, dim3(static_cast<unsigned>(blocks)), dim3(kGroupKernelThreads), lds,
                       st, static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k), e, r,
                       batch_geom(d), static_cast<int>(d.group), hchunk, nchunks, scale);
    return hipGetLastError();
}

template <typename T, int D, int HC, bool GLOBAL>
hipError_t launch_group(const Dims& d, float scale, const void* q, const void* k, float* e,
                        float* r, int hchunk, hipStream_t st) {
    const int nchunks = static_cast<int>((d.group + hchunk - 1) / hchunk);
    const size_t lds = static_cast<size_t>(hchunk) * (D + (GLOBAL ? 0 : d.N)) * sizeof(float);
    auto kern = score_group_kernel<T, D, HC, GLOBAL>;
    if (lds > 64 * 1024) {
        hipError_t err = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                             hipFuncAttributeMaxDynamicSharedMemorySize,
                                             static_cast<int>(lds));
        if (err != hipSuccess) return err;
    }
    const int64_t blocks = d.B * d.L * d.Hkv * nchunks;
    hipLaunchKernelGGL(kern, dim3(static_cast<unsigned>(blocks)), dim3(kGroupKernelThreads), lds,
                       st, static_cast<const T*>(q), static_cast<const T*>(k), e, r,
                       batch_geom(d), static_cast<int>(d.group), hchunk, nchunks, scale);
    return hipGetLastError();
}

// One query head per key head: one wave per (image, layer, head) unit, no
// workgroup barrier (wave_head); the workgroup only packs up to 4 independent
// waves together.
template <typename T, int D, bool GLOBAL>
__global__ __launch_bounds__(kThreads) void score_wave_kernel(
    const T* __restrict__ q, const T* __restrict__ k, float* __restrict__ e_out,
    float* __restrict__ r_out, BatchGeom bg, int64_t units, int nmax, float scale) {
    extern __shared__ float smem[];
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int64_t unit = static_cast<int64_t>(blockIdx.x) * (blockDim.x / kWave) + wave;
    if (unit >= units) return;
    const int64_t b = unit / (bg.L * bg.H);               // unit = (b*L + l)*H + h
    const int lh = static_cast<int>(unit - b * bg.L * bg.H);
    const ImageGeom ig = image_geom(bg, b);
    const int NT = ig.NT, N = ig.N;
    const int64_t row = bg.L * bg.H * ig.tok + static_cast<int64_t>(lh) * N;
    // logits in LDS, or (GLOBAL) in the head's output row, overwritten in place
    float* a = GLOBAL ? e_out + row : smem + wave * nmax;
    const int l = lh / bg.H, h = lh - l * bg.H;              // one query head per key head
    wave_head<T, D, GLOBAL>(query_rows(q, bg, ig, b, l, h), key_rows(k, bg, ig, b, l, h), NT, N,
                            mean_query_scale(scale, NT), a, lane, e_out + row,
                            r_out ? r_out + row : nullptr, query_ld(bg), key_ld(bg));
}

template <typename T, int D>
hipError_t launch_wave(const Dims& d, float scale, const void* q, const void* k, float* e,
                       float* r, hipStream_t st) {
    // a head's logits in LDS when one fits the budget, else in its output row
    const int64_t per_wave = d.N * static_cast<int64_t>(sizeof(float));
    const bool global = per_wave > kLdsBudget;
    const int wpg = global ? kWaves
                           : static_cast<int>(std::clamp<int64_t>(kLdsBudget / per_wave, 1, kWaves));
    const int64_t units = d.B * d.L * d.H;
    const int64_t blocks = (units + wpg - 1) / wpg;
    const size_t lds = global ? 0 : static_cast<size_t>(wpg * per_wave);
    auto kern = global ? score_wave_kernel<T, D, true> : score_wave_kernel<T, D, false>;
    if (lds > 64 * 1024) {
        hipError_t err = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                             hipFuncAttributeMaxDynamicSharedMemorySize,
                                             static_cast<int>(lds));
        if (err != hipSuccess) return err;
    }
    hipLaunchKernelGGL(kern, dim3(static_cast<unsigned>(blocks)), dim3(wpg * kWave), lds, st,
                       static_cast<const T*>(q), static_cast<const T*>(k), e, r, batch_geom(d),
                       units, static_cast<int>(d.N), scale);
    return hipGetLastError();
}

template <typename T, int D>
hipError_t dispatch(const Dims& d, float scale, const void* q, const void* k, float* e, float* r,
                    hipStream_t st) {
    if (d.group == 1) return launch_wave<T, D>(d, scale, q, k, e, r, st);
    // query heads per workgroup: all of the group, at most one MFMA tile's columns
    // (bf16) or kMaxChunk (fp32), and as many as fit the LDS budget with their
    // logits; chunks balanced.  When not even one head's logits fit, they go to
    // the output rows instead and the chunk is bounded by the first two limits.
    constexpr bool mfma = std::is_same<T, uint16_t>::value;
    const int64_t fit = kLdsBudget / ((D + d.N) * 4);
    const bool global = fit < 1;
    int hchunk = static_cast<int>(std::min<int64_t>(
        {d.group, mfma ? kMfmaMaxChunk : kMaxChunk, global ? d.group : fit}));
    const int nchunks = static_cast<int>((d.group + hchunk - 1) / hchunk);
    hchunk = static_cast<int>((d.group + nchunks - 1) / nchunks);
    if constexpr (mfma) {
        if (global) return launch_group_mfma<D, true>(d, scale, q, k, e, r, hchunk, st);
        return launch_group_mfma<D, false>(d, scale, q, k, e, r, hchunk, st);
    } else {
        auto run = [&](auto tag) {
            constexpr bool G = decltype(tag)::value;
            if (hchunk <= 2) return launch_group<T, D, 2, G>(d, scale, q, k, e, r, hchunk, st);
            if (hchunk <= 4) return launch_group<T, D, 4, G>(d, scale, q, k, e, r, hchunk, st);
            return launch_group<T, D, 8, G>(d, scale, q, k, e, r, hchunk, st);
        };
        return global ? run(std::true_type{}) : run(std::false_type{});
    }
}

}  // namespace

hipError_t launch_score_mean_logit(const Dims& d, int dtype, float scale, const void* q,
                                   const void* k, float* support_c, float* r_opt,
                                   hipStream_t stream) {
    if (dtype == E2S_DTYPE_BF16) {
        if (d.D == 128)
            return dispatch<uint16_t, 128>(d, scale, q, k, support_c, r_opt, stream);
        return dispatch<uint16_t, 64>(d, scale, q, k, support_c, r_opt, stream);
    }
    if (dtype == E2S_DTYPE_F16) {
        if (d.D == 128)
            return dispatch<_Float16, 128>(d, scale, q, k, support_c, r_opt, stream);
        return dispatch<_Float16, 64>(d, scale, q, k, support_c, r_opt, stream);
    }
    if (d.D == 128) return dispatch<float, 128>(d, scale, q, k, support_c, r_opt, stream);
    return dispatch<float, 64>(d, scale, q, k, support_c, r_opt, stream);
}

}  // namespace e2s
