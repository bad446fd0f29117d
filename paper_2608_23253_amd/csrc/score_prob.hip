// Score stage, mean-of-probabilities reading: for every text query t a softmax
// over the visual tokens of the scaled logits z[t, n] = Q_t.K_n * scale, then the
// mean over the queries, r_n = mean_t P[t, n]; support as in Eq. 9 (Sec. 4.1).
//
// Unlike the mean-of-logits reading this is a genuine dense contraction
// (N_T x N_V logits per head), computed on the matrix cores with
// v_mfma_f32_16x16x32_bf16 (bf16 storage) or v_mfma_f32_16x16x4_f32 (fp32 storage),
// fp32 accumulation.  One workgroup owns one (image, layer, query head); its text
// queries (in chunks of up to 128 rows) are staged in LDS, and the key tiles of 16
// rows are loaded straight into MFMA operand registers.  Two passes over the keys:
//
//   pass 1  online row statistics per query: m_t = max_n z, S_t = sum exp(z - m_t)
//           and E_t = sum expm1(z - m_t), merged across lanes and waves, then the
//           centring constant L_t = log(S_t / N)            (as in the other reading)
//   pass 2  per key column: sum over queries of  N P[t,n] - 1 = expm1(z - m_t - L_t)
//
// so u_n = N r_n - 1 = (1/N_T) sum_t expm1(z[t,n] - m_t - L_t) is accumulated in
// centred form, e_n = u_n / (2 (2 + u_n)), r_n = (1 + u_n) / N.
//
// Query heads that share a key head (grouped-query attention) run in workgroups
// with consecutive logical ids; the ids are remapped so that those workgroups land
// on the same XCD (blocks are dispatched round-robin over the 8 XCDs) and the
// second pass re-reads the keys from that XCD's L2.
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

// Per-type tiling: bf16 keeps 4 key tiles in flight, fp32 (wider operands) 2.
template <typename T, int D> struct ProbCfg;
template <int D> struct ProbCfg<uint16_t, D> {
    static constexpr int QC = 128;           // query rows per LDS chunk
    static constexpr int TG = 4;             // key tiles per statistics update
    static constexpr int QS = D + 8;         // padded LDS row (elements)
};
template <int D> struct ProbCfg<float, D> {
    static constexpr int QC = 64;
    static constexpr int TG = 2;
    static constexpr int QS = D + 4;
};

// B operand (keys) of one 16-key tile for all k steps.
//   bf16: lane (lr, lg) holds key lr, elements 32 s + 8 lg .. +7 of step s.
//   fp32: lane holds key lr, element d(s, lg) = 16 (s/4) + 4 lg + s%4 of step s.
// The A operand (queries) uses the same element mapping, so every product pairs
// Q[t, d] with K[n, d].
template <int NS>
__device__ __forceinline__ void load_b(bf16x8 (&b)[NS], const uint16_t* row, bool valid) {
#pragma unroll
    for (int s = 0; s < NS; ++s) {
        if (valid) {
            b[s] = __builtin_nontemporal_load(reinterpret_cast<const bf16x8*>(row + 32 * s));
        } else {
            b[s] = bf16x8{};
        }
    }
}
template <int NS>
__device__ __forceinline__ void load_b_f32(float (&b)[NS], const float* row, bool valid) {
#pragma unroll
    for (int t = 0; t < NS / 4; ++t) {
        f32x4v v = valid ? __builtin_nontemporal_load(reinterpret_cast<const f32x4v*>(row + 16 * t))
                         : f32x4v{0.f, 0.f, 0.f, 0.f};
        b[4 * t + 0] = v.x;
        b[4 * t + 1] = v.y;
        b[4 * t + 2] = v.z;
        b[4 * t + 3] = v.w;
    }
}

// One 16x16 logit tile (16 queries of block qb x 16 keys) into acc.
template <int D>
__device__ __forceinline__ f32x4v tile_mma(const uint16_t* qs, int qrow, int lg,
                                           const bf16x8 (&b)[D / 32]) {
    constexpr int QS = D + 8;
    f32x4v acc = {0.f, 0.f, 0.f, 0.f};
    const uint16_t* arow = qs + qrow * QS + 8 * lg;
#pragma unroll
    for (int s = 0; s < D / 32; ++s) {
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(arow + 32 * s);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b[s], acc, 0, 0, 0);
    }
    return acc;
}
template <int D>
__device__ __forceinline__ f32x4v tile_mma(const float* qs, int qrow, int lg,
                                           const float (&b)[D / 4]) {
    constexpr int QS = D + 4;
    f32x4v acc = {0.f, 0.f, 0.f, 0.f};
    const float* arow = qs + qrow * QS + 4 * lg;
#pragma unroll
    for (int t = 0; t < D / 16; ++t) {
        const f32x4v a = *reinterpret_cast<const f32x4v*>(arow + 16 * t);
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.x, b[4 * t + 0], acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.y, b[4 * t + 1], acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.z, b[4 * t + 2], acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.w, b[4 * t + 3], acc, 0, 0, 0);
    }
    return acc;
}

template <typename T, int D>
__global__ __launch_bounds__(kThreads) void score_mean_prob_kernel(
    const T* __restrict__ q, const T* __restrict__ k, float* __restrict__ e_out,
    float* __restrict__ r_out, int H, int NT, int N, int group, int Hkv, float scale,
    int nblocks) {
    using C = ProbCfg<T, D>;
    constexpr int QC = C::QC, TG = C::TG, QS = C::QS, QBM = QC / 16;
    constexpr int NB = std::is_same<T, float>::value ? D / 4 : D / 32;  // B regs per tile
    using BFrag = typename std::conditional<std::is_same<T, float>::value, float, bf16x8>::type;

    extern __shared__ __align__(16) unsigned char smem[];
    T* qs = reinterpret_cast<T*>(smem);                          // [QC][QS]
    float* st_m = reinterpret_cast<float*>(qs + QC * QS);        // [QC] row max
    float* st_l = st_m + QC;                                     // [QC] log(S/N)
    float* wpart = st_l + QC;                                    // [kWaves][QC][4]
    float* colsum = wpart + kWaves * QC * 4;                     // [N]

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

    for (int n = tid; n < N; n += kThreads) colsum[n] = 0.f;

    for (int t0 = 0; t0 < NT; t0 += QC) {
        const int rows = min(QC, NT - t0);
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
        __syncthreads();

        // ---- pass 1: online statistics of each query row --------------------
        float m[QBM][4], E[QBM][4], S[QBM][4];
#pragma unroll
        for (int i = 0; i < QBM; ++i)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                m[i][r] = -INFINITY;
                E[i][r] = 0.f;
                S[i][r] = 0.f;
            }
        float cnt = 0.f;                                          // valid keys seen by this lane
        for (int gi = wave; gi < ngroups; gi += kWaves) {
            BFrag b[TG][NB];
            bool valid[TG];
#pragma unroll
            for (int tt = 0; tt < TG; ++tt) {
                const int key = (gi * TG + tt) * 16 + lr;
                valid[tt] = key < N;
                if constexpr (std::is_same<T, float>::value)
                    load_b_f32<NB>(b[tt], kg + static_cast<int64_t>(key) * D + 4 * lg, valid[tt]);
                else
                    load_b<NB>(b[tt], kg + static_cast<int64_t>(key) * D + 8 * lg, valid[tt]);
            }
#pragma unroll
            for (int qb = 0; qb < QBM; ++qb) {
                if (qb < QB) {
                    f32x4v z[TG];
#pragma unroll
                    for (int tt = 0; tt < TG; ++tt) z[tt] = tile_mma<D>(qs, qb * 16 + lr, lg, b[tt]);
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        float v[TG];
                        float mx = m[qb][r];
#pragma unroll
                        for (int tt = 0; tt < TG; ++tt) {
                            v[tt] = valid[tt] ? z[tt][r] * scale : -INFINITY;
                            mx = fmaxf(mx, v[tt]);
                        }
                        if (__any(mx > m[qb][r])) {
                            // rescale the sums to the new maximum (exact no-op where unchanged)
                            const float dm = (mx > m[qb][r]) ? m[qb][r] - mx : 0.f;
                            const float sc = expf(dm);
                            const float em = (cnt > 0.f) ? expm1f(dm) : 0.f;
                            E[qb][r] = fmaf(cnt, em, E[qb][r] * sc);
                            S[qb][r] = S[qb][r] * sc;
                            m[qb][r] = mx;
                        }
#pragma unroll
                        for (int tt = 0; tt < TG; ++tt) {
                            if (valid[tt]) {
                                const float d = v[tt] - mx;
                                E[qb][r] += expm1f(d);
                                S[qb][r] += expf(d);
                            }
                        }
                    }
                }
            }
#pragma unroll
            for (int tt = 0; tt < TG; ++tt) cnt += valid[tt] ? 1.f : 0.f;
        }

        // ---- merge statistics: 16 lanes per row group, then the 4 waves ----
#pragma unroll
        for (int qb = 0; qb < QBM; ++qb) {
            if (qb < QB) {
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    float M = m[qb][r];
                    for (int o = 1; o < 16; o <<= 1) M = fmaxf(M, __shfl_xor(M, o));
                    float e = 0.f, s = 0.f, c = cnt;
                    if (cnt > 0.f) {
                        const float dm = m[qb][r] - M;
                        e = fmaf(cnt, expm1f(dm), E[qb][r] * expf(dm));
                        s = S[qb][r] * expf(dm);
                    }
                    for (int o = 1; o < 16; o <<= 1) {
                        e += __shfl_xor(e, o);
                        s += __shfl_xor(s, o);
                        c += __shfl_xor(c, o);
                    }
                    if (lr == 0) {
                        float* w = wpart + (wave * QC + qb * 16 + 4 * lg + r) * 4;
                        w[0] = (c > 0.f) ? M : -INFINITY;
                        w[1] = e;
                        w[2] = s;
                        w[3] = c;
                    }
                }
            }
        }
        __syncthreads();
        if (tid < QB * 16) {
            float M = -INFINITY;
            for (int w = 0; w < kWaves; ++w) M = fmaxf(M, wpart[(w * QC + tid) * 4]);
            float e = 0.f, s = 0.f;
            for (int w = 0; w < kWaves; ++w) {
                const float* p = wpart + (w * QC + tid) * 4;
                if (p[0] == -INFINITY) continue;     // this wave saw no key
                const float dm = p[0] - M;
                e += fmaf(p[3], expm1f(dm), p[1] * expf(dm));
                s += p[2] * expf(dm);
            }
            st_m[tid] = (tid < rows) ? M : 0.f;
            st_l[tid] = (tid < rows) ? log_mean_exp(e, s, fN) : 0.f;
        }
        __syncthreads();

        // ---- pass 2: column sums of N P - 1 = expm1(z - m - L) --------------
        for (int gi = wave; gi < ngroups; gi += kWaves) {
            BFrag b[TG][NB];
            bool valid[TG];
#pragma unroll
            for (int tt = 0; tt < TG; ++tt) {
                const int key = (gi * TG + tt) * 16 + lr;
                valid[tt] = key < N;
                if constexpr (std::is_same<T, float>::value)
                    load_b_f32<NB>(b[tt], kg + static_cast<int64_t>(key) * D + 4 * lg, valid[tt]);
                else
                    load_b<NB>(b[tt], kg + static_cast<int64_t>(key) * D + 8 * lg, valid[tt]);
            }
            float col[TG];
#pragma unroll
            for (int tt = 0; tt < TG; ++tt) col[tt] = 0.f;
#pragma unroll
            for (int qb = 0; qb < QBM; ++qb) {
                if (qb < QB) {
                    const int row0 = qb * 16 + 4 * lg;
                    const f32x4v mm = *reinterpret_cast<const f32x4v*>(st_m + row0);
                    const f32x4v ll = *reinterpret_cast<const f32x4v*>(st_l + row0);
#pragma unroll
                    for (int tt = 0; tt < TG; ++tt) {
                        const f32x4v z = tile_mma<D>(qs, qb * 16 + lr, lg, b[tt]);
#pragma unroll
                        for (int r = 0; r < 4; ++r) {
                            if (row0 + r < rows)
                                col[tt] += expm1f((z[r] * scale - mm[r]) - ll[r]);
                        }
                    }
                }
            }
#pragma unroll
            for (int tt = 0; tt < TG; ++tt) {
                col[tt] += __shfl_xor(col[tt], 16);
                col[tt] += __shfl_xor(col[tt], 32);
                const int key = (gi * TG + tt) * 16 + lr;
                if (lg == 0 && valid[tt]) colsum[key] += col[tt];
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
    const size_t lds = static_cast<size_t>(C::QC) * C::QS * sizeof(T) +
                       (2 * C::QC + kWaves * C::QC * 4) * sizeof(float) +
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
                       static_cast<int>(blocks));
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
