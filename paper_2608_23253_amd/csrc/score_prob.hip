// Score stage, mean-of-probabilities reading: for every text query t a softmax
// over the visual tokens of the scaled logits z[t, n] = Q_t.K_n * scale, then the
// mean over the queries, r_n = mean_t P[t, n]; support as in Eq. 9 (Sec. 4.1).
//
// Unlike the mean-of-logits reading this is a genuine dense contraction
// (N_T x N_V logits per head), computed on the matrix cores with
// v_mfma_f32_16x16x32_bf16 (bf16 storage) or v_mfma_f32_16x16x4_f32 (fp32
// storage), fp32 accumulation.  One workgroup owns one (image, layer, query head).
// Its text queries (chunks of up to 128 rows) are staged in LDS as the B operand;
// key tiles of 16 rows are loaded from HBM straight into A-operand registers, so a
// 16x16 result tile holds 16 keys (4 per lane) x 16 queries (one per lane).  Two
// passes over the keys:
//
//   pass 1  online row statistics of the lane's query: m_t = max_n z,
//           S_t = sum exp(z - m_t), E_t = sum expm1(z - m_t); merged across the
//           lanes and waves that saw other keys, then the centring constant
//           L_t = log(S_t / N)                               (as in the other reading)
//   pass 2  per key: sum over queries of  N P[t,n] - 1 = expm1(z - m_t - L_t),
//           accumulated in-lane over all query blocks, then summed across the 16
//           query lanes of a DPP row
//
// so u_n = N r_n - 1 = (1/N_T) sum_t expm1(z[t,n] - m_t - L_t) is accumulated in
// centred form; e_n = u_n / (2 (2 + u_n)), r_n = (1 + u_n) / N.
//
// expm1 of the small centred logits uses a degree-5 Taylor series on |x| <= 1/8;
// the library's expm1f / expf take over for a batch of 16 logits only when some
// lane of the wave has one outside that range (peaked attention).
// The query-block loops are not unrolled (the per-lane statistics live in LDS),
// which keeps the kernel's code within the instruction cache.
//
// Query heads that share a key head (grouped-query attention) run in workgroups
// with consecutive logical ids; the ids are remapped so that those workgroups land
// on the same XCD (blocks are dispatched round-robin over the 8 XCDs) and re-read
// the shared keys from that XCD's L2.
#include <type_traits>

#include "e2s_device.h"
#include "e2s_kernels.h"

namespace e2s {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4v __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;

__device__ __forceinline__ int xcd_remap(int bid, int nblocks) {
    const int q = nblocks / 8, r = nblocks % 8;
    const int x = bid % 8, i = bid / 8;
    return x * q + min(x, r) + i;
}

// expm1 on [-1/8, 1/8]: Taylor series to degree 5 (truncation below 6e-9, i.e.
// under one float32 ulp of the result, there).
constexpr float kSeriesRange = 0.125f;
__device__ __forceinline__ float expm1_series(float x) {
    float p = 1.0f / 120.0f;
    p = fmaf(p, x, 1.0f / 24.0f);
    p = fmaf(p, x, 1.0f / 6.0f);
    p = fmaf(p, x, 0.5f);
    p = fmaf(p, x, 1.0f);
    return p * x;
}

template <typename T, int D> struct ProbCfg;
template <int D> struct ProbCfg<uint16_t, D> {
    static constexpr int QC = 128;           // query rows per LDS chunk
    static constexpr int TG = 4;             // key tiles per wave iteration
    static constexpr int QS = D + 8;         // padded LDS row (elements)
    static constexpr int NA = D / 32;        // A registers (bf16x8) per key tile
    using AFrag = bf16x8;
};
template <int D> struct ProbCfg<float, D> {
    static constexpr int QC = 64;
    static constexpr int TG = 2;
    static constexpr int QS = D + 4;
    static constexpr int NA = D / 4;
    using AFrag = float;
};

// A operand (keys) of one 16-key tile for all k steps.
//   bf16: lane (lr, lg) holds key lr, elements 32 s + 8 lg .. +7 of step s.
//   fp32: lane holds key lr, element d(s, lg) = 16 (s/4) + 4 lg + s%4 of step s.
// The B operand (queries, from LDS) uses the same element mapping.
template <int NS>
__device__ __forceinline__ void load_keys(bf16x8 (&a)[NS], const uint16_t* row, bool valid) {
#pragma unroll
    for (int s = 0; s < NS; ++s)
        a[s] = valid ? __builtin_nontemporal_load(reinterpret_cast<const bf16x8*>(row + 32 * s))
                     : bf16x8{};
}
template <int NS>
__device__ __forceinline__ void load_keys(float (&a)[NS], const float* row, bool valid) {
#pragma unroll
    for (int t = 0; t < NS / 4; ++t) {
        const f32x4v v = valid
            ? __builtin_nontemporal_load(reinterpret_cast<const f32x4v*>(row + 16 * t))
            : f32x4v{0.f, 0.f, 0.f, 0.f};
        a[4 * t + 0] = v.x;
        a[4 * t + 1] = v.y;
        a[4 * t + 2] = v.z;
        a[4 * t + 3] = v.w;
    }
}

// Query operand (B) of one 16-query block, all k steps, read from LDS once and
// reused for every key tile.  Same element mapping as the keys.
template <int D>
__device__ __forceinline__ void load_queries(bf16x8 (&b)[D / 32], const uint16_t* qs, int qrow,
                                             int lr, int lg) {
    const uint16_t* brow = qs + (qrow + lr) * (D + 8) + 8 * lg;
#pragma unroll
    for (int s = 0; s < D / 32; ++s) b[s] = *reinterpret_cast<const bf16x8*>(brow + 32 * s);
}
template <int D>
__device__ __forceinline__ void load_queries(float (&b)[D / 4], const float* qs, int qrow, int lr,
                                             int lg) {
    const float* brow = qs + (qrow + lr) * (D + 4) + 4 * lg;
#pragma unroll
    for (int t = 0; t < D / 16; ++t) {
        const f32x4v v = *reinterpret_cast<const f32x4v*>(brow + 16 * t);
        b[4 * t + 0] = v.x;
        b[4 * t + 1] = v.y;
        b[4 * t + 2] = v.z;
        b[4 * t + 3] = v.w;
    }
}

// 16 keys x 16 queries: lane (lr, lg) gets the logits of keys 4 lg + r (r = 0..3)
// against query lr of the block.
template <int NA>
__device__ __forceinline__ f32x4v tile_mma(const bf16x8 (&a)[NA], const bf16x8 (&b)[NA]) {
    f32x4v acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < NA; ++s) acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[s], b[s], acc, 0, 0, 0);
    return acc;
}
template <int NA>
__device__ __forceinline__ f32x4v tile_mma(const float (&a)[NA], const float (&b)[NA]) {
    f32x4v acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < NA; ++s) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a[s], b[s], acc, 0, 0, 0);
    return acc;
}

template <typename T, int D>
__global__ __launch_bounds__(kThreads) void score_mean_prob_kernel(
    const T* __restrict__ q, const T* __restrict__ k, float* __restrict__ e_out,
    float* __restrict__ r_out, int H, int NT, int N, int group, int Hkv, float scale,
    int nblocks, int qcap) {
    using C = ProbCfg<T, D>;
    constexpr int TG = C::TG, QS = C::QS, NA = C::NA;
    using AFrag = typename C::AFrag;

    extern __shared__ __align__(16) unsigned char smem[];
    // qcap = min(QC, N_T rounded up to 16) query rows per chunk
    const int qbcap = qcap / 16;
    T* qs = reinterpret_cast<T*>(smem);                          // [qcap][QS]
    float* st_m = reinterpret_cast<float*>(qs + qcap * QS);      // [qcap] m + L per query
    float* wpart = st_m + qcap;                                  // [kWaves][qcap][4]
    float* lstat = wpart + kWaves * qcap * 4;                    // [3][qbcap][kThreads]
    float* colsum = lstat + 3 * qbcap * kThreads;                // [N]

    const int bid = xcd_remap(blockIdx.x, nblocks);              // (b*L + l)*H + h
    const int h = bid % H;
    const int64_t bl = bid / H;
    const int g = h / group;
    const T* qh = q + (bl * H + h) * static_cast<int64_t>(NT) * D;
    const T* kg = k + (bl * Hkv + g) * static_cast<int64_t>(N) * D;
    const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
    const int lr = lane % 16, lg = lane / 16;
    const int ntiles = (N + 15) / 16;
    const int ngroups = (ntiles + TG - 1) / TG;
    const float fN = static_cast<float>(N);
    const int koff = std::is_same<T, float>::value ? 4 * lg : 8 * lg;
    // this lane's online statistics (max, sum expm1, sum exp) of query block qb
    float* lm = lstat + tid;
    float* lE = lstat + qbcap * kThreads + tid;
    float* lS = lstat + 2 * qbcap * kThreads + tid;

    for (int n = tid; n < N; n += kThreads) colsum[n] = 0.f;

    for (int t0 = 0; t0 < NT; t0 += qcap) {
        const int rows = min(qcap, NT - t0);
        const int QB = (rows + 15) / 16;
        __syncthreads();
        // ---- stage this chunk of queries (rows past NT are zero) ----
        constexpr int EPV = 16 / sizeof(T);                       // elements per 16 bytes
        for (int idx = tid; idx < QB * 16 * (D / EPV); idx += kThreads) {
            const int row = idx / (D / EPV), c = idx % (D / EPV);
            f32x4v v = {0.f, 0.f, 0.f, 0.f};
            if (row < rows)
                v = *reinterpret_cast<const f32x4v*>(qh + static_cast<int64_t>(t0 + row) * D +
                                                     c * EPV);
            *reinterpret_cast<f32x4v*>(qs + row * QS + c * EPV) = v;
        }
        for (int qb = 0; qb < QB; ++qb) {
            lm[qb * kThreads] = -INFINITY;
            lE[qb * kThreads] = 0.f;
            lS[qb * kThreads] = 0.f;
        }
        __syncthreads();

        // ---- pass 1: online statistics of this lane's query in each block ----
        float cnt = 0.f;                                          // valid keys seen by this lane
        for (int gi = wave; gi < ngroups; gi += kWaves) {
            AFrag a[TG][NA];
            bool kval[TG][4];
#pragma unroll
            for (int tt = 0; tt < TG; ++tt) {
                const int tile = gi * TG + tt;
                const int key = tile * 16 + lr;
                load_keys<NA>(a[tt], kg + static_cast<int64_t>(min(key, N - 1)) * D + koff,
                              key < N);
#pragma unroll
                for (int r = 0; r < 4; ++r) kval[tt][r] = tile * 16 + 4 * lg + r < N;
            }
            const bool full = (gi + 1) * TG * 16 <= N;            // no key past N
            float cntg = 0.f;                                     // valid keys of this lane here
#pragma unroll
            for (int tt = 0; tt < TG; ++tt)
#pragma unroll
                for (int r = 0; r < 4; ++r) cntg += kval[tt][r] ? 1.f : 0.f;
            for (int qb = 0; qb < QB; ++qb) {
                AFrag bq[NA];
                load_queries<D>(bq, qs, qb * 16, lr, lg);
                float z[TG * 4];
#pragma unroll
                for (int tt = 0; tt < TG; ++tt) {
                    const f32x4v zt = tile_mma<NA>(a[tt], bq);
#pragma unroll
                    for (int r = 0; r < 4; ++r) z[tt * 4 + r] = zt[r];
                }
                float zmax = -INFINITY, zmin = INFINITY;
#pragma unroll
                for (int i = 0; i < TG * 4; ++i) {
                    const bool ok = full || kval[i / 4][i % 4];
                    zmax = fmaxf(zmax, ok ? z[i] : -INFINITY);
                    zmin = fminf(zmin, ok ? z[i] : INFINITY);
                }
                float m = lm[qb * kThreads], E = lE[qb * kThreads], S = lS[qb * kThreads];
                const float mx = fmaxf(m, zmax * scale);          // scale > 0
                if (__any(mx > m)) {
                    // rescale the sums to the new maximum (exact no-op where unchanged)
                    const float dm = (mx > m) ? m - mx : 0.f;
                    const float sc = expf(dm);
                    const float em = (cnt > 0.f) ? expm1f(dm) : 0.f;
                    E = fmaf(cnt, em, E * sc);
                    S = S * sc;
                    m = mx;
                }
                // every x = z * scale - mx lies in [zmin * scale - mx, 0]
                const bool near = cntg == 0.f || fmaf(zmin, scale, -mx) >= -kSeriesRange;
                if (__all(near)) {
                    float el = 0.f;
#pragma unroll
                    for (int i = 0; i < TG * 4; ++i) {
                        const float t = expm1_series(fmaf(z[i], scale, -mx));
                        el += (full || kval[i / 4][i % 4]) ? t : 0.f;
                    }
                    E += el;
                    S += cntg + el;
                } else {
#pragma unroll
                    for (int i = 0; i < TG * 4; ++i) {
                        if (full || kval[i / 4][i % 4]) {
                            const float x = fmaf(z[i], scale, -mx);
                            const float t = expm1f(x);
                            E += t;
                            S += (x < -0.5f) ? expf(x) : 1.0f + t;
                        }
                    }
                }
                lm[qb * kThreads] = m;
                lE[qb * kThreads] = E;
                lS[qb * kThreads] = S;
            }
            cnt += cntg;
        }

        // ---- merge statistics: the 4 lane groups of a wave, then the waves ----
        for (int qb = 0; qb < QB; ++qb) {
            const float m = lm[qb * kThreads];
            float M = fmaxf(m, __shfl_xor(m, 16));
            M = fmaxf(M, __shfl_xor(M, 32));
            float e = 0.f, s = 0.f;
            if (cnt > 0.f) {
                const float dm = m - M;
                e = fmaf(cnt, expm1f(dm), lE[qb * kThreads] * expf(dm));
                s = lS[qb * kThreads] * expf(dm);
            }
            float c = cnt;
            e += __shfl_xor(e, 16);
            s += __shfl_xor(s, 16);
            c += __shfl_xor(c, 16);
            e += __shfl_xor(e, 32);
            s += __shfl_xor(s, 32);
            c += __shfl_xor(c, 32);
            if (lg == 0) {
                float* wp = wpart + (wave * qcap + qb * 16 + lr) * 4;
                wp[0] = (c > 0.f) ? M : -INFINITY;
                wp[1] = e;
                wp[2] = s;
                wp[3] = c;
            }
        }
        __syncthreads();
        if (tid < QB * 16) {
            float M = -INFINITY;
            for (int w = 0; w < kWaves; ++w) M = fmaxf(M, wpart[(w * qcap + tid) * 4]);
            float e = 0.f, s = 0.f;
            for (int w = 0; w < kWaves; ++w) {
                const float* p = wpart + (w * qcap + tid) * 4;
                if (p[0] == -INFINITY) continue;     // this wave saw no key
                const float dm = p[0] - M;
                e += fmaf(p[3], expm1f(dm), p[1] * expf(dm));
                s += p[2] * expf(dm);
            }
            // one shift per query: z * scale - (m + L) is the centred logit
            st_m[tid] = (tid < rows) ? M + log_mean_exp(e, s, fN) : 0.f;
        }
        __syncthreads();

        // ---- pass 2: per key, sum over queries of expm1(z - m - L) ----------
        for (int gi = wave; gi < ngroups; gi += kWaves) {
            AFrag a[TG][NA];
#pragma unroll
            for (int tt = 0; tt < TG; ++tt) {
                const int key = (gi * TG + tt) * 16 + lr;
                load_keys<NA>(a[tt], kg + static_cast<int64_t>(min(key, N - 1)) * D + koff,
                              key < N);
            }
            float col[TG * 4];
#pragma unroll
            for (int i = 0; i < TG * 4; ++i) col[i] = 0.f;
            for (int qb = 0; qb < QB; ++qb) {
                AFrag bq[NA];
                load_queries<D>(bq, qs, qb * 16, lr, lg);
                const float shift = st_m[qb * 16 + lr];
                const bool qval = qb * 16 + lr < rows;
                float x[TG * 4];
                float xmin = INFINITY, xmax = -INFINITY;
#pragma unroll
                for (int tt = 0; tt < TG; ++tt) {
                    const f32x4v z = tile_mma<NA>(a[tt], bq);
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        x[tt * 4 + r] = fmaf(z[r], scale, -shift);
                        xmin = fminf(xmin, x[tt * 4 + r]);
                        xmax = fmaxf(xmax, x[tt * 4 + r]);
                    }
                }
                if (__all(fmaxf(-xmin, xmax) <= kSeriesRange)) {
#pragma unroll
                    for (int i = 0; i < TG * 4; ++i) col[i] += qval ? expm1_series(x[i]) : 0.f;
                } else {
#pragma unroll
                    for (int i = 0; i < TG * 4; ++i) col[i] += qval ? expm1f(x[i]) : 0.f;
                }
            }
#pragma unroll
            for (int i = 0; i < TG * 4; ++i) {
                const float sum = group_sum<16>(col[i]);
                const int key = (gi * TG + i / 4) * 16 + 4 * lg + i % 4;
                if (lr == 0 && key < N) colsum[key] += sum;
            }
        }
    }
    __syncthreads();

    const int64_t row = (bl * H + h) * static_cast<int64_t>(N);
    const float inv_nt = 1.0f / static_cast<float>(NT);
    for (int n = tid; n < N; n += kThreads) {
        const float u = colsum[n] * inv_nt;
        __builtin_nontemporal_store(u / (2.0f * (2.0f + u)), e_out + row + n);
        if (r_out) r_out[row + n] = (1.0f + u) / fN;
    }
}

template <typename T, int D>
hipError_t launch_mp(const Dims& d, float scale, const void* q, const void* k, float* e,
                     float* r, hipStream_t st) {
    using C = ProbCfg<T, D>;
    const int qcap = static_cast<int>(std::min<int64_t>(C::QC, (d.NT + 15) / 16 * 16));
    const size_t lds = static_cast<size_t>(qcap) * C::QS * sizeof(T) +
                       (qcap + kWaves * qcap * 4 + 3 * (qcap / 16) * kThreads) * sizeof(float) +
                       static_cast<size_t>(d.N) * sizeof(float);
    auto kern = score_mean_prob_kernel<T, D>;
    if (lds > 64 * 1024) {
        hipError_t err = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                             hipFuncAttributeMaxDynamicSharedMemorySize,
                                             static_cast<int>(lds));
        if (err != hipSuccess) return err;
    }
    const int64_t blocks = d.B * d.L * d.H;
    hipLaunchKernelGGL(kern, dim3(static_cast<unsigned>(blocks)), dim3(kThreads), lds, st,
                       static_cast<const T*>(q), static_cast<const T*>(k), e, r,
                       static_cast<int>(d.H), static_cast<int>(d.NT), static_cast<int>(d.N),
                       static_cast<int>(d.group), static_cast<int>(d.Hkv), scale,
                       static_cast<int>(blocks), qcap);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_score_mean_prob(const Dims& d, int dtype, float scale, const void* q,
                                  const void* k, float* support_c, float* r_opt,
                                  hipStream_t stream) {
    if (dtype == E2S_DTYPE_BF16) {
        if (d.D == 128) return launch_mp<uint16_t, 128>(d, scale, q, k, support_c, r_opt, stream);
        return launch_mp<uint16_t, 64>(d, scale, q, k, support_c, r_opt, stream);
    }
    if (d.D == 128) return launch_mp<float, 128>(d, scale, q, k, support_c, r_opt, stream);
    return launch_mp<float, 64>(d, scale, q, k, support_c, r_opt, stream);
}

}  // namespace e2s
