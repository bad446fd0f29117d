// Score stage, mean-of-probabilities reading: for every text query t a softmax
// over the visual tokens of the scaled logits z[t, n] = Q_t.K_n * scale, then the
// mean over the queries, r_n = mean_t P[t, n]; support as in Eq. 9 (Sec. 4.1).
//
// Unlike the mean-of-logits reading this is a genuine dense contraction
// (N_T x N_V logits per head), computed on the matrix cores with
// v_mfma_f32_16x16x32_bf16 / _f16 (bf16 / fp16 storage) or v_mfma_f32_16x16x4_f32
// (fp32 storage), fp32 accumulation.  One workgroup owns one (image, layer, query head).
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
// Near uniform attention expm1 is a short Taylor series.  In the tight range
// (every |z s - c_t| <= 1/16, the regime of Gaussian keys at the 1/sqrt(d)
// scale) both passes take it to degree 4 (degree 5 in pass 2 when some |L_t|
// widens its range past 1/16), five to seven vector operations per logit and pass.
// The reference is subtracted from the product after the matrix core, not
// started in its accumulator: a product started from -c_t rounds differently from
// the product minus c_t, and exactly uniform attention (identical keys) would then
// give supports of ~1e-11 instead of exactly 0.  Up to 1/8 pass 1 is redone
// with the degree-5 series and pass 2 takes degree 6 (|x - L_t| <= 1/4, since
// L_t lies between the smallest and largest x); every truncation stays within about
// one float32 ulp of the term at the range's edge (degree 4 at 1/16: x^5 / 120,
// 1.07 ulp of x) and far below it for the bulk.  When some
// logit of a query chunk lies further out (peaked attention), the chunk's
// statistics are recomputed online with the running maximum as reference
// (m_t = max_n z s, rescaled as it grows; S_t and E_t relative to it) and pass 2
// uses the library's expm1f wherever a 16 x 16 tile of logits leaves the series'
// range.  The tile is the unit of every such decision (score_prob_common.h), so
// the results do not depend on how many tiles a wave takes at once.
// The query-block loops are not unrolled (the per-lane statistics live in LDS),
// which keeps the kernel's code within the instruction cache.
//
// Heads of at most 64 text queries and 576 tokens take pass 2 in a second form in
// the tight range.  With x = expm1(s z - c_t) and S_t = N + E_t the softmax is
// (1 + x) / S_t, so N P - 1 = w_t x - E_t / S_t with w_t = N / S_t: the column
// sums weight the pass-1 terms instead of re-centring them.  For bf16 keys and
// 385 to 576 tokens (the LLaVA shape) a register-resident kernel keeps every x of
// a wave's 9 key tiles in registers, so pass 2 is one multiply-add per logit, with
// no second product and no second series; the two-pass kernel recomputes x for
// such heads with the same arithmetic, in the same order, so a head's bits do not
// depend on which of the two kernels its batch runs.
//
// Query heads that share a key head (grouped-query attention) run in workgroups
// with consecutive logical ids; the ids are remapped so that those workgroups land
// on the same XCD (blocks are dispatched round-robin over the 8 XCDs) and re-read
// the shared keys from that XCD's L2.
#include <type_traits>

#include "e2s_kernels.h"
#include "score_prob_common.h"

namespace e2s {
namespace {

using prob::kThreads;
using prob::kWaves;
using prob::ScaledSeries;
using prob::tile_mma;

__device__ __forceinline__ int xcd_remap(int bid, int nblocks) {
    const int q = nblocks / 8, r = nblocks % 8;
    const int x = bid % 8, i = bid / 8;
    return x * q + min(x, r) + i;
}

constexpr int64_t kColumnsInLds = 16384;
constexpr size_t kLdsPerCu = 160 * 1024;

// Heads of at most 16 kResMaxQueryBlocks text queries whose key tiles give each
// wave at most kResTiles of them can run register-resident (below).  The two-pass
// body computes such a head's column sums with the same arithmetic, so a head's
// bits do not depend on which kernel a batch runs.
constexpr int kResTiles = 9, kResMinTiles = 7, kResMaxQueryBlocks = 4;
// (the per-query statistics of such a head fit one wave: lane t holds query t)
static_assert(16 * kResMaxQueryBlocks <= kWave, "a head's queries in one wave");
__host__ __device__ constexpr int tiles_per_wave(int64_t N) {
    return static_cast<int>(((N + 15) / 16 + kWaves - 1) / kWaves);
}
__host__ __device__ constexpr bool resident_head(int64_t NT, int64_t N) {
    return NT <= 16 * kResMaxQueryBlocks && tiles_per_wave(N) <= kResTiles;
}

template <typename T, int D> struct ProbCfg;
template <int D> struct ProbCfg<uint16_t, D> {
    static constexpr int QC = 128;           // query rows per LDS chunk
    static constexpr int QS = D + 8;         // padded LDS row (elements)
    static constexpr int NA = D / 32;        // A registers (bf16x8) per key tile
    using AFrag = bf16x8;
};
template <int D> struct ProbCfg<_Float16, D> {
    static constexpr int QC = 128;
    static constexpr int QS = D + 8;
    static constexpr int NA = D / 32;        // A registers (f16x8) per key tile
    using AFrag = f16x8;
};
template <int D> struct ProbCfg<float, D> {
    static constexpr int QC = 64;
    static constexpr int QS = D + 4;
    static constexpr int NA = D / 4;
    using AFrag = float;
};

// A operand (keys) of one 16-key tile for all k steps.
//   bf16, fp16: lane (lr, lg) holds key lr, elements 32 s + 8 lg .. +7 of step s.
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
__device__ __forceinline__ void load_keys(f16x8 (&a)[NS], const _Float16* row) {
#pragma unroll
    for (int s = 0; s < NS; ++s) a[s] = *reinterpret_cast<const f16x8*>(row + 32 * s);
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
__device__ __forceinline__ void load_queries(f16x8 (&b)[D / 32], const _Float16* qs, int qrow,
                                             int lr, int lg) {
    const _Float16* brow = qs + (qrow + lr) * (D + 8) + 8 * lg;
#pragma unroll
    for (int s = 0; s < D / 32; ++s) b[s] = *reinterpret_cast<const f16x8*>(brow + 32 * s);
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

// TG key tiles per group, two groups in flight per wave: 4 tiles (2 workgroups per
// CU by registers) when a chunk has 8 query blocks, else 2 (3 per CU) or 1 (4 per
// CU with 16-bit keys, where the LDS allows it; fp32 keys always take 1, 3 per CU).
template <typename T, int D, int TG>
constexpr int mp_workgroups_per_cu() {
    return TG >= 4 ? 2 : (TG == 1 && !std::is_same<T, float>::value ? 4 : 3);
}
// The two-pass stage of one (image, layer, query head): the body of
// score_mean_prob_kernel, and the fallback of the register-resident kernel below.
template <typename T, int D, int TG, bool GLOBAL>
__device__ __forceinline__ void mean_prob_two_pass(const T* __restrict__ q,
                                                   const T* __restrict__ k,
                                                   float* __restrict__ e_out,
                                                   float* __restrict__ r_out, const BatchGeom& bg,
                                                   int group, float scale, int nblocks, int qcap,
                                                   bool cols_over_stats) {
    using C = ProbCfg<T, D>;
    constexpr int QS = C::QS, NA = C::NA;
    using AFrag = typename C::AFrag;

    extern __shared__ __align__(16) unsigned char smem[];
    // qcap = min(QC, N_T rounded up to 16) query rows per chunk
    const int qbcap = qcap / 16;
    T* qs = reinterpret_cast<T*>(smem);                          // [qcap][QS]
    float* st_m = reinterpret_cast<float*>(qs + qcap * QS);      // [qcap] shift of each query,
                                                                 // or w_t (tight range)
    float* st_c = st_m + qcap;                                   // [qcap] reference c_t
    float* wpart = st_c + qcap;                                  // [kWaves][qcap][4]
    float* lstat = wpart + kWaves * qcap * 4;                    // [3][qbcap][kThreads]
    __shared__ unsigned s_amax;                                  // max |z - c_t| (float bits)
    __shared__ unsigned s_lmax;                                  // max |L_t| (float bits)
    __shared__ float s_fsum;                                     // sum_t E_t / S_t (tight)

    const int64_t bid = xcd_remap(blockIdx.x, nblocks);          // (b*L + l)*H + h
    const int64_t b = bid / (bg.L * bg.H);
    const int lh = static_cast<int>(bid - b * bg.L * bg.H);
    const int l = lh / bg.H, h = lh - l * bg.H;
    const int g = h / group;
    const ImageGeom ig = image_geom(bg, b);
    const int NT = ig.NT, N = ig.N;
    const T* qh = query_rows(q, bg, ig, b, l, h);
    const T* kg = key_rows(k, bg, ig, b, l, g);
    const int64_t qld = query_ld(bg), kld = key_ld(bg);
    const int64_t row = bg.L * bg.H * ig.tok + static_cast<int64_t>(lh) * N;
    // [N] column sums: LDS, or (GLOBAL) the head's output row, overwritten at the
    // end.  cols_over_stats: every head has one query chunk and the sums fit in the
    // per-lane statistics, which are dead once pass 1 has been merged, so the sums
    // take their place (less LDS per workgroup, more workgroups per CU).
    float* colsum = GLOBAL ? e_out + row
                           : (cols_over_stats ? lstat : lstat + 3 * qbcap * kThreads);
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
            load_keys<NA>(a[tt], kg + static_cast<int64_t>(min(key, N - 1)) * kld + koff);
        }
    };

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

    for (int t0 = 0; t0 < NT; t0 += qcap) {
        const int rows = min(qcap, NT - t0);
        const int QB = (rows + 15) / 16;
        __syncthreads();
        // ---- stage this chunk of queries (rows past NT are zero): the thread's
        // packets are requested in two batches, each before its first store (two
        // round trips instead of one per packet, half the registers of one batch);
        // the requests are unconditional (indices past the chunk repeat its last
        // packet), so no branch makes a store wait for more than its batch
        constexpr int EPV = 16 / sizeof(T);                       // elements per 16 bytes
        constexpr int QPT = (C::QC * (D / EPV) + kThreads - 1) / kThreads;
        constexpr int QPB = (QPT + 1) / 2;                        // packets per batch
        const int packets = QB * 16 * (D / EPV);
#pragma unroll 1
        for (int i0 = 0; i0 < QPT; i0 += QPB) {
            f32x4v qv[QPB];
#pragma unroll
            for (int i = 0; i < QPB; ++i) {
                const int idx = min(tid + (i0 + i) * kThreads, packets - 1);
                const int row = idx / (D / EPV), c = idx % (D / EPV);
                qv[i] = *reinterpret_cast<const f32x4v*>(
                    qh + static_cast<int64_t>(t0 + min(row, rows - 1)) * qld + c * EPV);
            }
#pragma unroll
            for (int i = 0; i < QPB; ++i) {
                const int idx = tid + (i0 + i) * kThreads;
                const int row = idx / (D / EPV), c = idx % (D / EPV);
                const f32x4v zero = {0.f, 0.f, 0.f, 0.f};
                if (idx < packets)
                    *reinterpret_cast<f32x4v*>(qs + row * QS + c * EPV) = row < rows ? qv[i] : zero;
            }
        }
        for (int qb = 0; qb < QB; ++qb) lE[qb * kThreads] = 0.f;
        if (tid == 0) {
            s_amax = 0u;
            s_lmax = 0u;
        }
        __syncthreads();

        // ---- reference of each query (block_reference); zero query rows past
        // N_T get 0
        {
            AFrag a0[NA];
            load_keys<NA>(a0, kg + static_cast<int64_t>(min(lr, N - 1)) * kld + koff);
            for (int qb = wave; qb < QB; qb += kWaves) {
                AFrag bq[NA];
                load_queries<D>(bq, qs, qb * 16, lr, lg);
                const float c = prob::block_reference(tile_mma<NA>(a0, bq), N, lr);
                if (lg == 0) st_c[qb * 16 + lr] = c;
            }
        }
        __syncthreads();

        // ---- pass 1: E_t = sum_n expm1(s y) with y = z - c_t / s; groups of keys
        // double-buffered.  First by the degree-4 series (the tight range,
        // |s y| <= 1/16, checked afterwards), else again by the degree-5 series
        // (|s y| <= 1/8), else online (below).
        const ScaledSeries<5> p5(scale);
        const ScaledSeries<6> p6(scale);
        const ScaledSeries<4> p4(scale);
        float amax = 0.f;                                         // largest |y| seen
        auto pass1_group = [&](const AFrag (&a)[TG][NA], int j, auto whole, auto tight,
                               auto split) {
            for (int qb = 0; qb < QB; ++qb) {
                AFrag bq[NA];
                load_queries<D>(bq, qs, qb * 16, lr, lg);
                const float cz = st_c[qb * 16 + lr];
                float E = lE[qb * kThreads];
                if constexpr (decltype(tight)::value) {
#pragma unroll
                    for (int tt = 0; tt < TG; ++tt)
                        prob::series_tile<decltype(whole)::value, decltype(split)::value>(
                            tile_mma<NA>(a[tt], bq), cz, tile_of(j, tt) * 16 + 4 * lg, N, p4, E,
                            amax);
                } else {
#pragma unroll
                    for (int tt = 0; tt < TG; ++tt)
                        prob::series_tile<decltype(whole)::value, false>(
                            tile_mma<NA>(a[tt], bq), cz, tile_of(j, tt) * 16 + 4 * lg, N, p5, E,
                            amax);
                }
                lE[qb * kThreads] = E;
            }
        };
        auto pass1 = [&](auto tight, auto split) {
            stream_groups([&](const AFrag (&a)[TG][NA], int j) {
                // the group's last tile ends at or before N: no key of the group is
                // masked (tile_of is the same for every lane of the wave)
                if (__builtin_amdgcn_readfirstlane(tile_of(j, TG - 1)) * 16 + 16 <= N)
                    pass1_group(a, j, std::true_type{}, tight, split);
                else
                    pass1_group(a, j, std::false_type{}, tight, split);
            });
        };
        // a head the register-resident kernel could take rounds x = expm1(s y) / s
        // before summing it, as that kernel keeps it
        const bool weighted = resident_head(NT, N);
        if (weighted)
            pass1(std::true_type{}, std::true_type{});
        else
            pass1(std::true_type{}, std::false_type{});
        {
            // (non-negative floats order as their bits)
            const float wmax = wave_max(amax);
            if (lane == 0) atomicMax(&s_amax, __float_as_uint(wmax));
        }
        __syncthreads();
        const float amax_s = __uint_as_float(s_amax) * scale;
        const bool tight = amax_s <= prob::kTightRange;
        // |s y| <= 1/8 everywhere keeps the degree-5 series within its range
        const bool far = !(amax_s <= kSeriesRange);
        if (!tight && !far) {
            for (int qb = 0; qb < QB; ++qb) lE[qb * kThreads] = 0.f;
            pass1(std::false_type{}, std::false_type{});
        }

        if (!far) {
            // ---- merge the series sums: the 4 lane groups, then the waves ----
            for (int qb = 0; qb < QB; ++qb) {
                float e = lE[qb * kThreads];
                e += __shfl_xor(e, 16);
                e += __shfl_xor(e, 32);
                if (lg == 0) wpart[(wave * qcap + qb * 16 + lr) * 4] = e;
            }
            __syncthreads();
            float ft = 0.f;
            if (tid < QB * 16) {
                float e = 0.f;
                for (int w = 0; w < kWaves; ++w) e += wpart[(w * qcap + tid) * 4];
                if (tight && weighted) {
                    // S_t = N + E_t: w_t = N / S_t and E_t / S_t (zero rows: 1 and 0)
                    float wt = 1.f;
                    if (tid < rows) {
                        const float Et = scale * e;
                        const float S = fN + Et;
                        wt = fN / S;
                        ft = Et / S;
                    }
                    st_m[tid] = wt;
                } else {
                    // the shift of pass 2 in logit units: c_t + L_t / s
                    float L = 0.f, sh = 0.f;
                    if (tid < rows) {
                        L = log1pf((scale * e) / fN);
                        sh = st_c[tid] + L / scale;
                    }
                    st_m[tid] = sh;
                    atomicMax(&s_lmax, __float_as_uint(fabsf(L)));
                }
            }
            // (a weighted head has at most 64 queries: all in wave 0)
            if (tight && weighted && wave == 0) {
                const float fs = prob::query_sum(ft);
                if (lane == 0) s_fsum = fs;
            }
        } else {
            // ---- pass 1 again, online, tile by tile: running maximum as the
            // reference
            for (int qb = 0; qb < QB; ++qb) {
                lm[qb * kThreads] = -INFINITY;
                lE[qb * kThreads] = 0.f;
                lS[qb * kThreads] = 0.f;
            }
            float cnt = 0.f;                                      // valid keys seen by this lane
            for (int j = 0; j < ngw; ++j) {
                AFrag a[TG][NA];
                load_group(a, j);
                for (int qb = 0; qb < QB; ++qb) {
                    AFrag bq[NA];
                    load_queries<D>(bq, qs, qb * 16, lr, lg);
                    float m = lm[qb * kThreads], E = lE[qb * kThreads], S = lS[qb * kThreads];
                    float c = cnt;
#pragma unroll
                    for (int tt = 0; tt < TG; ++tt) {
                        const int key0 = tile_of(j, tt) * 16 + 4 * lg;
                        prob::online_tile(tile_mma<NA>(a[tt], bq), scale, key0, N, c, m, E, S);
                        c += prob::tile_count(key0, N);
                    }
                    lm[qb * kThreads] = m;
                    lE[qb * kThreads] = E;
                    lS[qb * kThreads] = S;
                }
#pragma unroll
                for (int tt = 0; tt < TG; ++tt) cnt += prob::tile_count(tile_of(j, tt) * 16 + 4 * lg, N);
            }

            // ---- merge statistics: the 4 lane groups of a wave, then the waves ----
            for (int qb = 0; qb < QB; ++qb) {
                const prob::OnlinePart pt =
                    prob::online_wave_part(lm[qb * kThreads], lE[qb * kThreads], lS[qb * kThreads], cnt);
                if (lg == 0) {
                    float* wp = wpart + (wave * qcap + qb * 16 + lr) * 4;
                    wp[0] = pt.M;
                    wp[1] = pt.e;
                    wp[2] = pt.s;
                    wp[3] = pt.c;
                }
            }
            __syncthreads();
            if (tid < QB * 16)
                st_m[tid] = (tid < rows) ? prob::online_shift(wpart + tid * 4, qcap * 4, fN) : 0.f;
        }
        __syncthreads();

        // ---- pass 2: per key, sum over queries of expm1(z s - c_t - L_t) ---------
        // (zero query rows past N_T have z = 0 and shift 0: they add expm1(0) = 0)
        auto add_columns = [&](const float (&col)[TG * 4], int j, float unit) {
#pragma unroll
            for (int i = 0; i < TG * 4; ++i) {
                const float sum = group_sum<16>(col[i]);
                const int key = tile_of(j, i / 4) * 16 + 4 * lg + i % 4;
                // a key's sums are kept by one lane through every chunk, the first
                // chunk starting them (every key below N is written then)
                if (lr == 0 && key < N) {
                    const float prev = (t0 == 0) ? 0.f : colsum[key];
                    colsum[key] = prev + unit * sum;
                }
            }
        };
        // tight: |s (z - shift)| <= amax_s + max |L_t| <= 1/8 (|L_t| <= amax_s): the
        // degree-4 series up to 1/16, else degree 5
        auto pass2_tight = [&](const auto& series) {
            stream_groups([&](const AFrag (&a)[TG][NA], int j) {
                float col[TG][4];
#pragma unroll
                for (int tt = 0; tt < TG; ++tt)
#pragma unroll
                    for (int r = 0; r < 4; ++r) col[tt][r] = 0.f;
                for (int qb = 0; qb < QB; ++qb) {
                    AFrag bq[NA];
                    load_queries<D>(bq, qs, qb * 16, lr, lg);
                    const float sz = st_m[qb * 16 + lr];
#pragma unroll
                    for (int tt = 0; tt < TG; ++tt)
                        prob::column_series_tile(tile_mma<NA>(a[tt], bq), sz, series, col[tt]);
                }
                add_columns(reinterpret_cast<const float(&)[TG * 4]>(col), j, scale);
            });
        };
        if (tight && !weighted) {
            if (amax_s + __uint_as_float(s_lmax) <= prob::kTightRange)
                pass2_tight(p4);
            else
                pass2_tight(p5);
        } else if (tight) {
            // N P - 1 = w_t x - E_t / S_t with x = expm1(s (z - c_t)) recomputed
            // exactly as in pass 1 (the register-resident kernel's arithmetic, in
            // the same order, so both give the same bits)
            const float fsum = s_fsum;
            stream_groups([&](const AFrag (&a)[TG][NA], int j) {
                float col[TG][4];
#pragma unroll
                for (int tt = 0; tt < TG; ++tt)
#pragma unroll
                    for (int r = 0; r < 4; ++r) col[tt][r] = 0.f;
                for (int qb = 0; qb < QB; ++qb) {
                    AFrag bq[NA];
                    load_queries<D>(bq, qs, qb * 16, lr, lg);
                    const float cz = st_c[qb * 16 + lr], wq = st_m[qb * 16 + lr];
#pragma unroll
                    for (int tt = 0; tt < TG; ++tt)
                        prob::column_weighted_tile(tile_mma<NA>(a[tt], bq), cz, p4, wq, col[tt]);
                }
#pragma unroll
                for (int i = 0; i < TG * 4; ++i) {
                    const float sum = group_sum<16>(col[i / 4][i % 4]);
                    const int key = tile_of(j, i / 4) * 16 + 4 * lg + i % 4;
                    if (lr == 0 && key < N) {
                        const float prev = (t0 == 0) ? 0.f : colsum[key];
                        colsum[key] = prev + (scale * sum - fsum);
                    }
                }
            });
        } else if (!far) {
            // y = z - shift; |s y| <= 1/4: the degree-6 series; the column sums are
            // in units of s
            stream_groups([&](const AFrag (&a)[TG][NA], int j) {
                float col[TG][4];
#pragma unroll
                for (int tt = 0; tt < TG; ++tt)
#pragma unroll
                    for (int r = 0; r < 4; ++r) col[tt][r] = 0.f;
                for (int qb = 0; qb < QB; ++qb) {
                    AFrag bq[NA];
                    load_queries<D>(bq, qs, qb * 16, lr, lg);
                    const float sz = st_m[qb * 16 + lr];
#pragma unroll
                    for (int tt = 0; tt < TG; ++tt)
                        prob::column_series_tile(tile_mma<NA>(a[tt], bq), sz, p6, col[tt]);
                }
                add_columns(reinterpret_cast<const float(&)[TG * 4]>(col), j, scale);
            });
        } else {
            for (int j = 0; j < ngw; ++j) {
                AFrag a[TG][NA];
                load_group(a, j);
                float col[TG][4];
#pragma unroll
                for (int tt = 0; tt < TG; ++tt)
#pragma unroll
                    for (int r = 0; r < 4; ++r) col[tt][r] = 0.f;
                for (int qb = 0; qb < QB; ++qb) {
                    AFrag bq[NA];
                    load_queries<D>(bq, qs, qb * 16, lr, lg);
                    const float shift = st_m[qb * 16 + lr];
#pragma unroll
                    for (int tt = 0; tt < TG; ++tt)
                        prob::column_far_tile(tile_mma<NA>(a[tt], bq), scale, shift, col[tt]);
                }
                add_columns(reinterpret_cast<const float(&)[TG * 4]>(col), j, 1.0f);
            }
        }
    }
    __syncthreads();

    const float inv_nt = 1.0f / static_cast<float>(NT);
    for (int n = tid; n < N; n += kThreads) {
        const float u = colsum[n] * inv_nt;
        __builtin_nontemporal_store(u / (2.0f * (2.0f + u)), e_out + row + n);
        if (r_out) r_out[row + n] = (1.0f + u) / fN;
    }
}

template <typename T, int D, int TG, bool GLOBAL>
__global__ __launch_bounds__(kThreads, (mp_workgroups_per_cu<T, D, TG>())) void score_mean_prob_kernel(
    const T* __restrict__ q, const T* __restrict__ k, float* __restrict__ e_out,
    float* __restrict__ r_out, BatchGeom bg, int group, float scale, int nblocks, int qcap,
    bool cols_over_stats) {
    mean_prob_two_pass<T, D, TG, GLOBAL>(q, k, e_out, r_out, bg, group, scale, nblocks, qcap,
                                         cols_over_stats);
}

// Register-resident variant for heads of 16 (QBN - 1) + 1 .. 16 QBN text queries
// whose key tiles give every wave at most MAXT of them (the LLaVA shape: 64
// queries, 576 tokens, 9 tiles per wave).  Pass 1 keeps each x = expm1(s (z - c_t)) of the
// wave's tiles in registers; with S_t = N + E_t (E_t = sum_n x) the softmax is
// P = (1 + x) / S_t, so
//   N P - 1 = (N x - E_t) / S_t = w_t x - E_t / S_t,   w_t = N / S_t,
// and the column sums take one multiply-add per logit: no second product on the
// matrix cores and no second series.  Only the tight range (every |s (z - c_t)|
// <= 1/16, where the degree-4 series is within an ulp) takes this path; any other
// head runs the two-pass body from the start.  u = N r - 1 is then
// (s sum_t w_t x' - sum_t E_t / S_t) / N_T with x = s x' (the series in units of s).
template <typename T, int D, int MAXT, int QBN>
__global__ __launch_bounds__(kThreads, 2) void score_mean_prob_resident_kernel(
    const T* __restrict__ q, const T* __restrict__ k, float* __restrict__ e_out,
    float* __restrict__ r_out, BatchGeom bg, int group, float scale, int nblocks, int qcap,
    bool cols_over_stats) {
    using C = ProbCfg<T, D>;
    constexpr int QS = C::QS, NA = C::NA, QR = 16 * QBN;
    constexpr int KB = 3;                                        // key tiles in registers
    static_assert(QBN >= 1 && QR <= kWave && MAXT >= KB, "resident kernel shape");
    using AFrag = typename C::AFrag;

    extern __shared__ __align__(16) unsigned char smem[];
    T* qs = reinterpret_cast<T*>(smem);                          // [QR][QS]
    float* wpart = reinterpret_cast<float*>(qs + QR * QS);       // [kWaves][QR]
    __shared__ unsigned s_amax;                                  // max |z - c_t| (float bits)

    const int64_t bid = xcd_remap(blockIdx.x, nblocks);          // (b*L + l)*H + h
    const int64_t b = bid / (bg.L * bg.H);
    const int lh = static_cast<int>(bid - b * bg.L * bg.H);
    const int l = lh / bg.H, h = lh - l * bg.H;
    const ImageGeom ig = image_geom(bg, b);
    const int NT = ig.NT, N = ig.N;
    const T* qh = query_rows(q, bg, ig, b, l, h);
    const T* kg = key_rows(k, bg, ig, b, l, h / group);
    const int64_t qld = query_ld(bg), kld = key_ld(bg);
    const int64_t row = bg.L * bg.H * ig.tok + static_cast<int64_t>(lh) * N;
    const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
    const int lr = lane % 16, lg = lane / 16;
    const int ntiles = (N + 15) / 16;
    // this wave's tiles (<= MAXT); the loops run MAXT of them, a tile past the
    // wave's last one repeating that tile with every logit masked, so that no
    // branch separates the loads from their uses
    const int ntw = wave < ntiles ? (ntiles - wave + kWaves - 1) / kWaves : 0;
    constexpr int QB = QBN;                                      // 16 (QBN - 1) < N_T
    const float fN = static_cast<float>(N);
    const int koff = std::is_same<T, float>::value ? 4 * lg : 8 * lg;
    auto key_of = [&](int j) { return (wave + kWaves * j) * 16; };
    auto load_tile = [&](AFrag (&a)[NA], int j) {
        const int jj = min(j, max(ntw - 1, 0));
        load_keys<NA>(a, kg + static_cast<int64_t>(min(key_of(jj) + lr, N - 1)) * kld + koff);
    };

    // the queries are requested first, then keys 0..15 for the references and the
    // wave's first key tiles, so that staging the queries waits for them alone
    constexpr int EPV = 16 / sizeof(T);                          // elements per 16 bytes
    constexpr int QPT = (QR * (D / EPV) + kThreads - 1) / kThreads;   // packets per thread
    f32x4v qv[QPT];
#pragma unroll
    for (int i = 0; i < QPT; ++i) {
        const int idx = min(tid + i * kThreads, QR * (D / EPV) - 1);
        const int r = idx / (D / EPV), c = idx % (D / EPV);
        qv[i] = *reinterpret_cast<const f32x4v*>(qh + static_cast<int64_t>(min(r, NT - 1)) * qld +
                                                 c * EPV);
    }
    __builtin_amdgcn_sched_barrier(0);                           // (the request order)
    AFrag a0[NA];
    load_keys<NA>(a0, kg + static_cast<int64_t>(min(lr, N - 1)) * kld + koff);
    AFrag a[KB][NA];
#pragma unroll
    for (int j = 0; j < KB - 1; ++j) load_tile(a[j], j);
    __builtin_amdgcn_sched_barrier(0);

    // ---- stage the queries (rows past N_T are zero) and their references ----
#pragma unroll
    for (int i = 0; i < QPT; ++i) {
        const int idx = tid + i * kThreads;
        if (idx < QR * (D / EPV)) {
            const int r = idx / (D / EPV), c = idx % (D / EPV);
            const f32x4v zero = {0.f, 0.f, 0.f, 0.f};
            *reinterpret_cast<f32x4v*>(qs + r * QS + c * EPV) = r < NT ? qv[i] : zero;
        }
    }
    if (tid == 0) s_amax = 0u;
    __syncthreads();
    // every wave takes all the references itself (a few products; no barrier)
    float cz[QBN];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
        AFrag bq[NA];
        load_queries<D>(bq, qs, qb * 16, lr, lg);
        cz[qb] = prob::block_reference(tile_mma<NA>(a0, bq), N, lr);
    }

    // ---- pass 1: x = expm1(s y) / s = y P(y), y = z - c_t, kept per logit ------
    // the first QKEEP query blocks' operands stay in registers for every tile (the
    // others are read from LDS per tile); not with two blocks, where the registers
    // would cost a wave per SIMD
    constexpr int QKEEP = QBN == 2 ? 0 : (QBN < 2 ? QBN : 2);
    AFrag bkeep[QKEEP > 0 ? QKEEP : 1][NA];
#pragma unroll
    for (int qb = 0; qb < QKEEP; ++qb) load_queries<D>(bkeep[qb], qs, qb * 16, lr, lg);
    const ScaledSeries<4> p4(scale);
    float x[MAXT][QBN][4];
    float E[QBN];
#pragma unroll
    for (int qb = 0; qb < QBN; ++qb) E[qb] = 0.f;
    float amax = 0.f;
#pragma unroll
    for (int j = 0; j < MAXT; ++j) {
        if (j + KB - 1 < MAXT) load_tile(a[(j + KB - 1) % KB], j + KB - 1);
        const int key0 = key_of(j) + 4 * lg;
        const bool own = j < ntw;
        // MASKED: some key of the tile is past N or the tile is past the wave's last
        // (the same values either way: masking only zeroes such keys)
        auto tile = [&](auto masked) {
#pragma unroll
            for (int qb = 0; qb < QB; ++qb) {
                AFrag bq[NA];
                if (qb < QKEEP) {
#pragma unroll
                    for (int t = 0; t < NA; ++t) bq[t] = bkeep[qb < QKEEP ? qb : 0][t];
                } else {
                    load_queries<D>(bq, qs, qb * 16, lr, lg);
                }
                const f32x4v z = tile_mma<NA>(a[j % KB], bq);
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    float y = z[r] - cz[qb];
                    if constexpr (decltype(masked)::value) y = (own && key0 + r < N) ? y : 0.f;
                    amax = fmaxf(amax, fabsf(y));
                    const float xv = p4(y) * y;
                    x[j][qb][r] = xv;
                    E[qb] += xv;
                }
            }
        };
        if (__builtin_amdgcn_readfirstlane(own && key_of(j) + 16 <= N))
            tile(std::false_type{});
        else
            tile(std::true_type{});
        // keep the tiles in program order: the compiler would otherwise sink each
        // tile's loads down to its first use, which leaves none in flight
        __builtin_amdgcn_sched_barrier(0);
    }
    {
        const float wmax = wave_max(amax);
        if (lane == 0) atomicMax(&s_amax, __float_as_uint(wmax));
    }
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
        float e = E[qb];
        e += __shfl_xor(e, 16);
        e += __shfl_xor(e, 32);
        if (lg == 0) wpart[wave * QR + qb * 16 + lr] = e;
    }
    __syncthreads();
    if (!(__uint_as_float(s_amax) * scale <= prob::kTightRange)) {
        // outside the tight range: the two-pass stage from the start (its LDS is
        // at least this kernel's; every thread has passed the barrier above)
        __syncthreads();
        mean_prob_two_pass<T, D, 1, false>(q, k, e_out, r_out, bg, group, scale, nblocks, qcap,
                                           cols_over_stats);
        return;
    }
    // every wave merges the statistics itself, lane t for query t (no barrier)
    float ft = 0.f, wt = 1.f;                                    // rows past N_T: x = 0
    if (lane < QB * 16) {
        float e = 0.f;
        for (int w = 0; w < kWaves; ++w) e += wpart[w * QR + lane];
        if (lane < NT) {
            const float Et = scale * e;
            const float S = fN + Et;
            wt = fN / S;
            ft = Et / S;
        }
    }
    const float fsum = prob::query_sum(ft);
    float wq[QBN];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) wq[qb] = __shfl(wt, qb * 16 + lr);

    // ---- column sums: per key, sum over the queries of w_t x' -----------------
    const float inv_nt = 1.0f / static_cast<float>(NT);
#pragma unroll
    for (int j = 0; j < MAXT; ++j) {
        float col[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int qb = 0; qb < QB; ++qb)
#pragma unroll
            for (int r = 0; r < 4; ++r) col[r] = fmaf(wq[qb], x[j][qb][r], col[r]);
        // every lane of a 16-lane row ends with the row's four key sums; lane r of
        // the row finishes key key0 + r, so each division runs once per key
        float sr[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) sr[r] = group_sum<16>(col[r]);
        const float sum = lr == 0 ? sr[0] : lr == 1 ? sr[1] : lr == 2 ? sr[2] : sr[3];
        const int key = key_of(j) + 4 * lg + lr;
        if (j < ntw && lr < 4 && key < N) {
            const float u = (scale * sum - fsum) * inv_nt;
            __builtin_nontemporal_store(u / (2.0f * (2.0f + u)), e_out + row + key);
            if (r_out) r_out[row + key] = (1.0f + u) / fN;
        }
    }
}

// LDS of one workgroup: the column sums in LDS up to kColumnsInLds keys, else in
// the output rows; in the statistics' place when every head has one query chunk
// and they fit (over).
template <typename T, int D>
size_t mp_lds(const Dims& d, int qcap, bool& global, bool& over) {
    using C = ProbCfg<T, D>;
    global = d.N > kColumnsInLds;
    const int64_t stats = 3 * (qcap / 16) * kThreads;            // floats
    over = !global && d.NT <= qcap && d.N <= stats;
    return static_cast<size_t>(qcap) * C::QS * sizeof(T) +
           (2 * qcap + kWaves * qcap * 4 + stats) * sizeof(float) +
           (global || over ? 0 : static_cast<size_t>(d.N) * sizeof(float));
}

template <typename T, int D, int TG>
hipError_t launch_mp(const Dims& d, float scale, const void* q, const void* k, float* e,
                     float* r, int qcap, hipStream_t st) {
    bool global = false, over = false;
    const size_t lds = mp_lds<T, D>(d, qcap, global, over);
    auto kern = global ? score_mean_prob_kernel<T, D, TG, true>
                       : score_mean_prob_kernel<T, D, TG, false>;
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
                       static_cast<int>(blocks), qcap, over);
    return hipGetLastError();
}

// The register-resident kernel takes a batch whose largest head qualifies with 7
// to kResTiles key tiles per wave (385 to 576 tokens; every wave runs kResTiles, so
// fewer tiles would waste more of them); every head of such a batch qualifies.
bool resident_fits(const Dims& d) {
    return resident_head(d.NT, d.N) && tiles_per_wave(d.N) >= kResMinTiles;
}

template <typename T, int D, int QBN>
hipError_t launch_mp_resident(const Dims& d, float scale, const void* q, const void* k, float* e,
                              float* r, int qcap, hipStream_t st) {
    using C = ProbCfg<T, D>;
    constexpr int QR = 16 * QBN;
    bool global = false, over = false;
    // room for the two-pass fallback (one tile per group) as well
    const size_t lds = std::max(static_cast<size_t>(QR) * C::QS * sizeof(T) +
                                    static_cast<size_t>(kWaves * QR) * sizeof(float),
                                mp_lds<T, D>(d, qcap, global, over));
    auto kern = score_mean_prob_resident_kernel<T, D, kResTiles, QBN>;
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
                       static_cast<int>(blocks), qcap, over);
    return hipGetLastError();
}

template <typename T, int D>
hipError_t dispatch_mp(const Dims& d, float scale, const void* q, const void* k, float* e,
                       float* r, hipStream_t st) {
    using C = ProbCfg<T, D>;
    // qcap = min(QC, N_T rounded up to 16) query rows per chunk
    const int qcap = static_cast<int>(std::min<int64_t>(C::QC, (d.NT + 15) / 16 * 16));
    if constexpr (std::is_same<T, uint16_t>::value) {
        if (resident_fits(d)) {
            switch ((d.NT + 15) / 16) {
                case 1: return launch_mp_resident<T, D, 1>(d, scale, q, k, e, r, qcap, st);
                case 2: return launch_mp_resident<T, D, 2>(d, scale, q, k, e, r, qcap, st);
                case 3: return launch_mp_resident<T, D, 3>(d, scale, q, k, e, r, qcap, st);
                default: return launch_mp_resident<T, D, 4>(d, scale, q, k, e, r, qcap, st);
            }
        }
    }
    if constexpr (std::is_same<T, float>::value) {
        return launch_mp<T, D, 1>(d, scale, q, k, e, r, qcap, st);
    } else {
        // measured: 4 tiles per group pays when a chunk has 8 query blocks; one tile
        // per group (under 128 VGPRs: 4 workgroups per CU) when the LDS also leaves
        // room for 4 (the LLaVA shape, 34 KiB, before the register-resident kernel
        // took it: stage 413 -> 397 us), else 2 (Qwen2-VL: 50 KiB, 3 per CU, where one
        // tile measured 284 -> 293 us)
        if (qcap >= 128) return launch_mp<T, D, 4>(d, scale, q, k, e, r, qcap, st);
        bool global = false, over = false;
        if (4 * mp_lds<T, D>(d, qcap, global, over) <= kLdsPerCu)
            return launch_mp<T, D, 1>(d, scale, q, k, e, r, qcap, st);
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
    if (dtype == E2S_DTYPE_F16) {
        if (d.D == 128) return dispatch_mp<_Float16, 128>(d, scale, q, k, support_c, r_opt, stream);
        return dispatch_mp<_Float16, 64>(d, scale, q, k, support_c, r_opt, stream);
    }
    if (d.D == 128) return dispatch_mp<float, 128>(d, scale, q, k, support_c, r_opt, stream);
    return dispatch_mp<float, 64>(d, scale, q, k, support_c, r_opt, stream);
}

}  // namespace e2s
