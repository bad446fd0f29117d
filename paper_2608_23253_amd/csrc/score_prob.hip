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
//   pass 1  row statistics of the lane's query: with a reference c_t (the mean
//           scaled logit of keys 0..15), E_t = sum_n expm1(z s - c_t), then
//           L_t = log(S_t / N) with S_t = N + E_t, so that z s - c_t - L_t is the
//           centred logit
//   pass 2  per key: sum over queries of  N P[t,n] - 1 = expm1(z s - c_t - L_t),
//           accumulated in-lane over all query blocks, then summed across the 16
//           query lanes of a DPP row
//
// so u_n = N r_n - 1 = (1/N_T) sum_t expm1(z[t,n] s - c_t - L_t) is accumulated in
// centred form; e_n = u_n / (2 (2 + u_n)), r_n = (1 + u_n) / N.
//
// Near uniform attention (every |z s - c_t| <= 1/8, the regime of Gaussian keys
// at the 1/sqrt(d) scale) expm1 is a short Taylor series: degree 5 in pass 1
// (|x| <= 1/8) and degree 6 in pass 2 (|x - L_t| <= 1/4, since L_t lies between
// the smallest and largest x), each truncated below one float32 ulp.  That costs
// about seven vector operations per logit and pass: the products run on the
// matrix cores and the kernel is bound by this elementwise work.  When some
// logit of a query chunk lies further out (peaked attention), the chunk's
// statistics are recomputed online with the running maximum as reference
// (m_t = max_n z s, rescaled as it grows; S_t and E_t relative to it) and pass 2
// uses the library's expm1f wherever a batch of 16 logits leaves the series'
// range.
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
// expm1(x) = x * series_p5(x) on |x| <= 1/8 (degree 5) and x * series_p6(x) on
// |x| <= 1/4 (degree 6: truncation x^7 / 5040, below 6e-8 relative there); the
// callers fold the last product into their running sums.
__device__ __forceinline__ float series_p5(float x) {
    float p = fmaf(1.0f / 120.0f, x, 1.0f / 24.0f);
    p = fmaf(p, x, 1.0f / 6.0f);
    p = fmaf(p, x, 0.5f);
    return fmaf(p, x, 1.0f);
}
__device__ __forceinline__ float series_p6(float x) {
    float p = fmaf(1.0f / 720.0f, x, 1.0f / 120.0f);
    p = fmaf(p, x, 1.0f / 24.0f);
    p = fmaf(p, x, 1.0f / 6.0f);
    p = fmaf(p, x, 0.5f);
    return fmaf(p, x, 1.0f);
}

template <typename T, int D> struct ProbCfg;
template <int D> struct ProbCfg<uint16_t, D> {
    static constexpr int QC = 128;           // query rows per LDS chunk
    static constexpr int QS = D + 8;         // padded LDS row (elements)
    static constexpr int NA = D / 32;        // A registers (bf16x8) per key tile
    using AFrag = bf16x8;
};
template <int D> struct ProbCfg<float, D> {
    static constexpr int QC = 64;
    static constexpr int QS = D + 4;
    static constexpr int NA = D / 4;
    using AFrag = float;
};

// A operand (keys) of one 16-key tile for all k steps.
//   bf16: lane (lr, lg) holds key lr, elements 32 s + 8 lg .. +7 of step s.
//   fp32: lane holds key lr, element d(s, lg) = 16 (s/4) + 4 lg + s%4 of step s.
// The B operand (queries, from LDS) uses the same element mapping.
// Loads are unconditional (callers clamp the row into range and discard the
// results of keys past N), so no branch separates a load from its use and the
// next group's loads stay in flight while the current group is used.  They are
// ordinary cached loads: pass 2 (and the other query heads of a key head) read
// the same keys again, from L2 where they are still there (non-temporal loads
// measured 4-20 % slower).
template <int NS>
__device__ __forceinline__ void load_keys(bf16x8 (&a)[NS], const uint16_t* row) {
#pragma unroll
    for (int s = 0; s < NS; ++s) a[s] = *reinterpret_cast<const bf16x8*>(row + 32 * s);
}
template <int NS>
__device__ __forceinline__ void load_keys(float (&a)[NS], const float* row) {
#pragma unroll
    for (int t = 0; t < NS / 4; ++t) {
        const f32x4v v = *reinterpret_cast<const f32x4v*>(row + 16 * t);
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
// expm1(s y) = s y P(y) with P the series of the scaled argument: coefficients
// s^k / (k+1)! for k = 1 .. DEG-1 (DEG = 5 or 6), so the scale is applied once per
// sum instead of once per logit.
template <int DEG>
struct ScaledSeries {
    float c[DEG - 1];
    __device__ explicit ScaledSeries(float s) {
        float pk = 1.0f, f = 1.0f;
#pragma unroll
        for (int kk = 1; kk < DEG; ++kk) {
            pk *= s;
            f *= static_cast<float>(kk + 1);
            c[kk - 1] = pk / f;
        }
    }
    __device__ __forceinline__ float operator()(float y) const {
        float p = c[DEG - 2];
#pragma unroll
        for (int kk = DEG - 3; kk >= 0; --kk) p = fmaf(p, y, c[kk]);
        return fmaf(p, y, 1.0f);
    }
};

// TG key tiles per group, two groups in flight per wave: 4 tiles (2 workgroups per
// CU by registers) when a chunk has 8 query blocks, else 2 (3 per CU).
template <typename T, int D, int TG>
__global__ __launch_bounds__(kThreads, TG >= 4 ? 2 : 3) void score_mean_prob_kernel(
    const T* __restrict__ q, const T* __restrict__ k, float* __restrict__ e_out,
    float* __restrict__ r_out, BatchGeom bg, int group, float scale, int nblocks, int qcap) {
    using C = ProbCfg<T, D>;
    constexpr int QS = C::QS, NA = C::NA;
    using AFrag = typename C::AFrag;

    extern __shared__ __align__(16) unsigned char smem[];
    // qcap = min(QC, N_T rounded up to 16) query rows per chunk
    const int qbcap = qcap / 16;
    T* qs = reinterpret_cast<T*>(smem);                          // [qcap][QS]
    float* st_m = reinterpret_cast<float*>(qs + qcap * QS);      // [qcap] shift of each query
    float* st_c = st_m + qcap;                                   // [qcap] reference c_t
    float* wpart = st_c + qcap;                                  // [kWaves][qcap][4]
    float* lstat = wpart + kWaves * qcap * 4;                    // [3][qbcap][kThreads]
    float* colsum = lstat + 3 * qbcap * kThreads;                // [N]
    __shared__ int s_far;                                        // some |z s - c_t| > 1/8

    const int64_t bid = xcd_remap(blockIdx.x, nblocks);          // (b*L + l)*H + h
    const int64_t b = bid / (bg.L * bg.H);
    const int lh = static_cast<int>(bid - b * bg.L * bg.H);
    const int l = lh / bg.H, h = lh - l * bg.H;
    const int g = h / group;
    const ImageGeom ig = image_geom(bg, b);
    const int NT = ig.NT, N = ig.N;
    const T* qh = q + ig.q_off + static_cast<int64_t>(lh) * NT * D;
    const T* kg = k + ig.k_off + static_cast<int64_t>(l * bg.Hkv + g) * N * D;
    const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
    const int lr = lane % 16, lg = lane / 16;
    // Key tiles of 16 rows go to the waves round-robin (wave w: tiles w, w + 4,
    // w + 8, ...), and a wave takes its own tiles TG at a time, in ascending order.
    // The tile a lane sees, and the order in which its sums run, do not depend on
    // TG, so the results do not either.
    const int ntiles = (N + 15) / 16;
    const int ntw = wave < ntiles ? (ntiles - wave + kWaves - 1) / kWaves : 0;  // this wave's
    const int ngw = (ntw + TG - 1) / TG;                                       // groups
    auto tile_of = [&](int j, int tt) { return wave + kWaves * (j * TG + tt); };
    const float fN = static_cast<float>(N);
    const int koff = std::is_same<T, float>::value ? 4 * lg : 8 * lg;
    // this lane's statistics of query block qb: series sum E, or online (max,
    // sum expm1, sum exp)
    float* lm = lstat + tid;
    float* lE = lstat + qbcap * kThreads + tid;
    float* lS = lstat + 2 * qbcap * kThreads + tid;

    // keys of this wave's group j (TG tiles of 16 rows) into A-operand registers;
    // rows past N repeat row N - 1
    auto load_group = [&](AFrag (&a)[TG][NA], int j) {
#pragma unroll
        for (int tt = 0; tt < TG; ++tt) {
            const int key = tile_of(j, tt) * 16 + lr;
            load_keys<NA>(a[tt], kg + static_cast<int64_t>(min(key, N - 1)) * D + koff);
        }
    };
    // no key of group j lies past N
    auto group_full = [&](int j) { return (tile_of(j, TG - 1) + 1) * 16 <= N; };

    // body(a, j) for every group j of this wave, the next group's keys requested
    // before the current one is used.  The requests are unconditional (past the
    // last group they repeat it), so every path has the same loads in flight and
    // the wait before a group's first use leaves the next group's loads pending.
    auto stream_groups = [&](auto&& body) {
        AFrag a0[TG][NA], a1[TG][NA];
        const int last = max(ngw - 1, 0);
        load_group(a0, 0);
        for (int j = 0; j < ngw; j += 2) {
            load_group(a1, min(j + 1, last));
            body(a0, j);
            if (j + 1 >= ngw) break;
            load_group(a0, min(j + 2, last));
            body(a1, j + 1);
        }
    };

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
        for (int qb = 0; qb < QB; ++qb) lE[qb * kThreads] = 0.f;
        if (tid == 0) s_far = 0;
        __syncthreads();

        // ---- reference of each query: mean logit Q_t.K_n of keys 0..15 ----------
        // (pairwise, so that equal logits give exactly their value; the logit of
        // key 0 when N < 16; zero query rows past N_T get 0); c_t = s times it
        {
            AFrag a0[NA];
            load_keys<NA>(a0, kg + static_cast<int64_t>(min(lr, N - 1)) * D + koff);
            for (int qb = wave; qb < QB; qb += kWaves) {
                AFrag bq[NA];
                load_queries<D>(bq, qs, qb * 16, lr, lg);
                const f32x4v z = tile_mma<NA>(a0, bq);
                float sum = (z[0] + z[1]) + (z[2] + z[3]);
                sum += __shfl_xor(sum, 16);
                sum += __shfl_xor(sum, 32);
                const float z0 = __shfl(z[0], lr);              // key 0, from lane (lr, 0)
                if (lg == 0) st_c[qb * 16 + lr] = (N >= 16) ? sum * (1.0f / 16.0f) : z0;
            }
        }
        __syncthreads();

        // ---- pass 1: E_t = sum_n expm1(s y) with y = z - c_t / s, by the degree-5
        // series; groups of keys double-buffered
        const ScaledSeries<5> p5(scale);
        const ScaledSeries<6> p6(scale);
        float amax = 0.f;                                         // largest |y| seen
        stream_groups([&](const AFrag (&a)[TG][NA], int j) {
            const bool full = group_full(j);
            for (int qb = 0; qb < QB; ++qb) {
                AFrag bq[NA];
                load_queries<D>(bq, qs, qb * 16, lr, lg);
                const float cz = st_c[qb * 16 + lr];
                float y[TG * 4];
#pragma unroll
                for (int tt = 0; tt < TG; ++tt) {
                    const f32x4v zt = tile_mma<NA>(a[tt], bq);
#pragma unroll
                    for (int r = 0; r < 4; ++r) y[tt * 4 + r] = zt[r] - cz;
                }
                if (!full) {
#pragma unroll
                    for (int i = 0; i < TG * 4; ++i)
                        y[i] = (tile_of(j, i / 4) * 16 + 4 * lg + i % 4 < N) ? y[i] : 0.f;
                }
                float E = lE[qb * kThreads];
#pragma unroll
                for (int i = 0; i < TG * 4; ++i) {
                    amax = fmaxf(amax, fabsf(y[i]));
                    E = fmaf(p5(y[i]), y[i], E);
                }
                lE[qb * kThreads] = E;
            }
        });
        // |s y| <= 1/8 everywhere keeps the series within its range
        if (!(wave_max(amax) * scale <= kSeriesRange) && lane == 0) atomicOr(&s_far, 1);
        __syncthreads();
        const bool far = s_far != 0;

        if (!far) {
            // ---- merge the series sums: the 4 lane groups, then the waves ----
            for (int qb = 0; qb < QB; ++qb) {
                float e = lE[qb * kThreads];
                e += __shfl_xor(e, 16);
                e += __shfl_xor(e, 32);
                if (lg == 0) wpart[(wave * qcap + qb * 16 + lr) * 4] = e;
            }
            __syncthreads();
            if (tid < QB * 16) {
                float e = 0.f;
                for (int w = 0; w < kWaves; ++w) e += wpart[(w * qcap + tid) * 4];
                // E = s e; S = N + E >= N exp(-1/8) > N / 2, so L = log1p(E / N)
                // (as log_mean_exp); the shift of pass 2 in logit units: c_t / s + L / s
                st_m[tid] = (tid < rows) ? st_c[tid] + log1pf((scale * e) / fN) / scale : 0.f;
            }
        } else {
            // ---- pass 1 again, online: running maximum as the reference ----------
            for (int qb = 0; qb < QB; ++qb) {
                lm[qb * kThreads] = -INFINITY;
                lE[qb * kThreads] = 0.f;
                lS[qb * kThreads] = 0.f;
            }
            float cnt = 0.f;                                      // valid keys seen by this lane
            for (int j = 0; j < ngw; ++j) {
                AFrag a[TG][NA];
                load_group(a, j);
                bool kval[TG][4];
#pragma unroll
                for (int tt = 0; tt < TG; ++tt)
#pragma unroll
                    for (int r = 0; r < 4; ++r) kval[tt][r] = tile_of(j, tt) * 16 + 4 * lg + r < N;
                const bool full = group_full(j);
                float cntg = 0.f;                                 // valid keys of this lane here
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
                    const float mx = fmaxf(m, zmax * scale);      // scale > 0
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
        }
        __syncthreads();

        // ---- pass 2: per key, sum over queries of expm1(z s - c_t - L_t) ---------
        // (zero query rows past N_T have z = 0 and shift 0: they add expm1(0) = 0)
        auto add_columns = [&](const float (&col)[TG * 4], int j, float unit) {
#pragma unroll
            for (int i = 0; i < TG * 4; ++i) {
                const float sum = group_sum<16>(col[i]);
                const int key = tile_of(j, i / 4) * 16 + 4 * lg + i % 4;
                if (lr == 0 && key < N) colsum[key] += unit * sum;
            }
        };
        if (!far) {
            // y = z - shift; |s y| <= 1/4: the degree-6 series; the column sums are
            // in units of s
            stream_groups([&](const AFrag (&a)[TG][NA], int j) {
                float col[TG * 4];
#pragma unroll
                for (int i = 0; i < TG * 4; ++i) col[i] = 0.f;
                for (int qb = 0; qb < QB; ++qb) {
                    AFrag bq[NA];
                    load_queries<D>(bq, qs, qb * 16, lr, lg);
                    const float sz = st_m[qb * 16 + lr];
#pragma unroll
                    for (int tt = 0; tt < TG; ++tt) {
                        const f32x4v zt = tile_mma<NA>(a[tt], bq);
#pragma unroll
                        for (int r = 0; r < 4; ++r) {
                            const float y = zt[r] - sz;
                            col[tt * 4 + r] = fmaf(p6(y), y, col[tt * 4 + r]);
                        }
                    }
                }
                add_columns(col, j, scale);
            });
        } else {
            for (int j = 0; j < ngw; ++j) {
                AFrag a[TG][NA];
                load_group(a, j);
                float col[TG * 4];
#pragma unroll
                for (int i = 0; i < TG * 4; ++i) col[i] = 0.f;
                for (int qb = 0; qb < QB; ++qb) {
                    AFrag bq[NA];
                    load_queries<D>(bq, qs, qb * 16, lr, lg);
                    const float shift = st_m[qb * 16 + lr];
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
                        for (int i = 0; i < TG * 4; ++i) col[i] += expm1_series(x[i]);
                    } else {
#pragma unroll
                        for (int i = 0; i < TG * 4; ++i) col[i] += expm1f(x[i]);
                    }
                }
                add_columns(col, j, 1.0f);
            }
        }
    }
    __syncthreads();

    const int64_t row = bg.L * bg.H * ig.tok + static_cast<int64_t>(lh) * N;
    const float inv_nt = 1.0f / static_cast<float>(NT);
    for (int n = tid; n < N; n += kThreads) {
        const float u = colsum[n] * inv_nt;
        __builtin_nontemporal_store(u / (2.0f * (2.0f + u)), e_out + row + n);
        if (r_out) r_out[row + n] = (1.0f + u) / fN;
    }
}

template <typename T, int D, int TG>
hipError_t launch_mp(const Dims& d, float scale, const void* q, const void* k, float* e,
                     float* r, int qcap, hipStream_t st) {
    using C = ProbCfg<T, D>;
    const size_t lds = static_cast<size_t>(qcap) * C::QS * sizeof(T) +
                       (2 * qcap + kWaves * qcap * 4 + 3 * (qcap / 16) * kThreads) * sizeof(float) +
                       static_cast<size_t>(d.N) * sizeof(float);
    auto kern = score_mean_prob_kernel<T, D, TG>;
    if (lds > 64 * 1024) {
        hipError_t err = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                             hipFuncAttributeMaxDynamicSharedMemorySize,
                                             static_cast<int>(lds));
        if (err != hipSuccess) return err;
    }
    const int64_t blocks = d.B * d.L * d.H;
    hipLaunchKernelGGL(kern, dim3(static_cast<unsigned>(blocks)), dim3(kThreads), lds, st,
                       static_cast<const T*>(q), static_cast<const T*>(k), e, r,
                       batch_geom(d), static_cast<int>(d.group), scale,
                       static_cast<int>(blocks), qcap);
    return hipGetLastError();
}

template <typename T, int D>
hipError_t dispatch_mp(const Dims& d, float scale, const void* q, const void* k, float* e,
                       float* r, hipStream_t st) {
    using C = ProbCfg<T, D>;
    // qcap = min(QC, N_T rounded up to 16) query rows per chunk
    const int qcap = static_cast<int>(std::min<int64_t>(C::QC, (d.NT + 15) / 16 * 16));
    if constexpr (std::is_same<T, float>::value) {
        return launch_mp<T, D, 1>(d, scale, q, k, e, r, qcap, st);
    } else {
        // measured: 4 tiles per group pays when a chunk has 8 query blocks
        if (qcap >= 128) return launch_mp<T, D, 4>(d, scale, q, k, e, r, qcap, st);
        return launch_mp<T, D, 2>(d, scale, q, k, e, r, qcap, st);
    }
}

}  // namespace

hipError_t launch_score_mean_prob(const Dims& d, int dtype, float scale, const void* q,
                                  const void* k, float* support_c, float* r_opt,
                                  hipStream_t stream) {
    if (dtype == E2S_DTYPE_BF16) {
        if (d.D == 128) return dispatch_mp<uint16_t, 128>(d, scale, q, k, support_c, r_opt, stream);
        return dispatch_mp<uint16_t, 64>(d, scale, q, k, support_c, r_opt, stream);
    }
    if (d.D == 128) return dispatch_mp<float, 128>(d, scale, q, k, support_c, r_opt, stream);
    return dispatch_mp<float, 64>(d, scale, q, k, support_c, r_opt, stream);
}

}  // namespace e2s
