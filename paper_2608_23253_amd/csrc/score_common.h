// Arithmetic of the mean-of-logits score stage shared by the per-head score kernels
// (score.hip) and the per-layer evidence kernel (layer.hip).  Callers run these
// functions with the same thread-to-data mapping, so they produce the same bits
// (the library is compiled without floating-point contraction).
#pragma once

#include "e2s_device.h"

namespace e2s {

// Logit of one key row: lane wl's 8-element dot product, summed over the LPR lanes
// that share the row.
template <int LPR>
__device__ __forceinline__ float row_logit(const float (&qb)[8], const float (&x)[8]) {
    float s = qb[0] * x[0];
#pragma unroll
    for (int m = 1; m < 8; ++m) s = fmaf(qb[m], x[m], s);
    return group_sum<LPR>(s);
}

// expm1 on [-1/8, 1/8]: Taylor series to degree 5 (truncation below 6e-9, under
// one float32 ulp of the result, there).
constexpr float kSeriesRange = 0.125f;
__device__ __forceinline__ float expm1_series(float x) {
    float p = 1.0f / 120.0f;
    p = fmaf(p, x, 1.0f / 24.0f);
    p = fmaf(p, x, 1.0f / 6.0f);
    p = fmaf(p, x, 0.5f);
    p = fmaf(p, x, 1.0f);
    return p * x;
}

// Support e = p - 1/2 of a centred logit dc = a - max - L (Eq. 8-9):
// e = u / (2 (2 + u)) with u = expm1(dc) > -1, so the divisor exceeds 2; it is
// inverted by the hardware reciprocal estimate and one Newton step (within about an
// ulp, at a third of the cost of an IEEE division).
__device__ __forceinline__ float support_from_centred(float dc, bool near) {
    const float u = near ? expm1_series(dc) : expm1f(dc);
    const float d = 2.0f * (2.0f + u);
    float r = __builtin_amdgcn_rcpf(d);
    r = fmaf(r, fmaf(-d, r, 1.0f), r);
    return u * r;
}

// Orders one wave's LDS stores before its later LDS loads of other lanes' data
// (LDS requests of a wave are served in issue order; this keeps the compiler from
// moving loads above the stores).
__device__ __forceinline__ void wave_lds_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// The same for logits kept in global memory (an image whose logits do not fit in
// LDS): workgroup-scope release and acquire order the wave's stores before its
// later loads of other lanes' values (as a workgroup barrier does for global
// memory).
__device__ __forceinline__ void global_logits_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
}

// ---------------------------------------------------------------------------
// Logits on the matrix cores for grouped-query heads (bf16 keys): the fp32 query
// means of up to 16 heads are split exactly into three bf16 terms
// (hi + mid + lo = qbar: each term takes the next 8 significant bits, 24 in all),
// and a 16-key tile meets the three terms in three fp32 accumulators
// (v_mfma_f32_16x16x32_bf16), so a logit carries the same information as the
// fp32 dot product; only the rounding of the sums differs.
// ---------------------------------------------------------------------------
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ uint32_t bf16_bits_rne(float x) {
    const uint32_t u = __float_as_uint(x);
    return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

// x = hi + mid + lo exactly for finite x of normal range: each residual is exact in
// fp32 and carries at most 16, then 8, significant bits.
__device__ __forceinline__ void split_bf16x3(float x, uint16_t& hi, uint16_t& mid, uint16_t& lo) {
    const uint32_t h = bf16_bits_rne(x);
    const float r1 = x - __uint_as_float(h << 16);
    const uint32_t m = bf16_bits_rne(r1);
    const float r2 = r1 - __uint_as_float(m << 16);
    hi = static_cast<uint16_t>(h);
    mid = static_cast<uint16_t>(m);
    lo = static_cast<uint16_t>(bf16_bits_rne(r2));
}

// Logits of one 16-key tile (A operand kt: lane (lr, lg) holds key lr, elements
// 32 s + 8 lg .. + 7 of step s) against up to 16 heads: bh, bm, bo point at this
// lane's head lr row of the hi, mid and lo terms (offset by 8 lg elements; a zero
// row for a column without a head).  Lane (lr, lg) gets the logits of keys
// 4 lg + r against head lr, summed as (lo + mid) + hi.
template <int NS>
__device__ __forceinline__ f32x4 split_tile_logits(const bf16x8 (&kt)[NS], const uint16_t* bh,
                                                   const uint16_t* bm, const uint16_t* bo) {
    f32x4 ch = {0.f, 0.f, 0.f, 0.f}, cm = ch, co = ch;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
        const bf16x8 vh = *reinterpret_cast<const bf16x8*>(bh + 32 * s);
        const bf16x8 vm = *reinterpret_cast<const bf16x8*>(bm + 32 * s);
        const bf16x8 vo = *reinterpret_cast<const bf16x8*>(bo + 32 * s);
        ch = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kt[s], vh, ch, 0, 0, 0);
        cm = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kt[s], vm, cm, 0, 0, 0);
        co = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kt[s], vo, co, 0, 0, 0);
    }
    f32x4 z;
#pragma unroll
    for (int r = 0; r < 4; ++r) z[r] = (co[r] + cm[r]) + ch[r];
    return z;
}

// Lane geometry of the per-wave score stage: 8 elements per lane, LPR lanes per
// row, RPW rows per wave-wide load, KU rows per lane in flight (16 B per lane per
// row for bf16, 32 B for fp32).
template <typename T, int D>
struct WaveRows {
    static constexpr int LPR = D / 8, RPW = kWave / LPR, KU = 16 / sizeof(T);
    static constexpr int BATCH = KU * RPW;   // rows per wave-wide batch
};

// KU key rows base + wrow + u * RPW of one head (kh offset by 8*wl elements; ld
// elements from one row to the next); rows past the end are clamped to the last
// row (in bounds) and discarded later.
template <typename T, int D, int KU>
__device__ __forceinline__ void load_key_batch(Packet<T> (&p)[KU], const T* __restrict__ kh,
                                               int base, int wrow, int N, int64_t ld) {
    constexpr int RPW = WaveRows<T, D>::RPW;
#pragma unroll
    for (int u = 0; u < KU; ++u)
        load_packet(p[u], kh + static_cast<int64_t>(min(base + wrow + u * RPW, N - 1)) * ld);
}

// Logits of one batch: a[n] = qbar . K[n] for the rows of load_key_batch.
template <typename T, int D, int KU>
__device__ __forceinline__ void key_batch_logits(const Packet<T> (&p)[KU], const float (&qb)[8],
                                                 float* a, int base, int wrow, int wl,
                                                 int n_end) {
    constexpr int LPR = WaveRows<T, D>::LPR, RPW = WaveRows<T, D>::RPW;
#pragma unroll
    for (int u = 0; u < KU; ++u) {
        float x[8];
        unpack(p[u], x);
        const float s = row_logit<LPR>(qb, x);
        const int n = base + wrow + u * RPW;
        if (wl == 0 && n < n_end) a[n] = s;
    }
}

// Scale of the summed queries: Eq. 1's logit scale over N_T, rounded once from
// the double quotient (per image, since a ragged batch has one N_T per image).
__device__ __forceinline__ float mean_query_scale(float scale, int NT) {
    return static_cast<float>(static_cast<double>(scale) / static_cast<double>(NT));
}

// Query mean of one head by one wave: lane (wrow, wl) sums rows wrow, wrow + RPW,
// ... of dims 8*wl .. 8*wl+7 in increasing row order; the RPW row sums are then
// combined by a butterfly, so every lane holds the same qbar (times qscale).  qh is
// offset by 8*wl elements; ld elements from one row to the next.  QU rows per lane
// are requested at once; the order of the sums, hence the result, does not depend
// on QU.
template <typename T, int D, int QU = WaveRows<T, D>::KU>
__device__ __forceinline__ void wave_query_mean(const T* __restrict__ qh, int NT, int wrow,
                                                float qscale, float (&qb)[8], int64_t ld) {
    constexpr int LPR = WaveRows<T, D>::LPR, RPW = WaveRows<T, D>::RPW;
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    for (int t0 = 0; t0 < NT; t0 += QU * RPW) {
        Packet<T> p[QU];
#pragma unroll
        for (int u = 0; u < QU; ++u)
            load_packet(p[u], qh + static_cast<int64_t>(min(t0 + wrow + u * RPW, NT - 1)) * ld);
#pragma unroll
        for (int u = 0; u < QU; ++u) {
            float x[8];
            unpack(p[u], x);
            const bool ok = t0 + wrow + u * RPW < NT;
#pragma unroll
            for (int m = 0; m < 8; ++m) acc[m] += ok ? x[m] : 0.f;
        }
    }
#pragma unroll
    for (int m = 0; m < 8; ++m) {
        for (int o = LPR; o < kWave; o <<= 1) acc[m] += __shfl_xor(acc[m], o);
        qb[m] = acc[m] * qscale;
    }
}

// Eq. 8-9 for one head's N logits a[] (LDS, complete and visible to the wave): per
// lane max / min / sums over n = lane, lane + 64, ... in increasing order, then
// butterflies across the wave.  wave_softmax_stats leaves a_n - max in a[] and
// returns L and near; the centred logit of token n is then dc = a[n] - L
// (u = N r - 1 = expm1(dc)).  near: the head's logits span at most kSeriesRange,
// so every a - max and every a - max - L lies in [-kSeriesRange, kSeriesRange]
// (L lies between the smallest a - max and 0) and expm1 is evaluated by the short
// series; otherwise by the library.  L = log(S / N) is taken by log_mean_exp.
// wave_softmax calls emit(n, dc, near) once per token, from lane n % 64.
__device__ __forceinline__ void wave_softmax_stats(float* a, int N, int lane, float& L,
                                                   bool& near) {
    float mx = -INFINITY, lo = INFINITY;
    for (int n = lane; n < N; n += kWave) {
        mx = fmaxf(mx, a[n]);
        lo = fminf(lo, a[n]);
    }
    mx = wave_max(mx);
    lo = -wave_max(-lo);
    near = mx - lo <= kSeriesRange;
    float E = 0.f, S = 0.f;
    if (near) {
        for (int n = lane; n < N; n += kWave) {
            const float d = a[n] - mx;
            a[n] = d;
            const float t = expm1_series(d);
            E += t;
            S += 1.0f + t;
        }
    } else {
        for (int n = lane; n < N; n += kWave) {
            const float d = a[n] - mx;
            a[n] = d;
            E += expm1f(d);
            S += expf(d);
        }
    }
    E = wave_sum(E);
    S = wave_sum(S);
    L = log_mean_exp(E, S, static_cast<float>(N));
}

template <typename Emit>
__device__ __forceinline__ void wave_softmax(float* a, int N, int lane, Emit&& emit) {
    float L;
    bool near;
    wave_softmax_stats(a, N, lane, L, near);
    // near is uniform over the wave: one loop per case, unrolled so that the LDS
    // reads of several tokens are in flight together
    if (near) {
#pragma unroll 4
        for (int n = lane; n < N; n += kWave) emit(n, a[n] - L, true);
    } else {
#pragma unroll 4
        for (int n = lane; n < N; n += kWave) emit(n, a[n] - L, false);
    }
}

// Eq. 8-9 for one head's logits a[] (as for wave_softmax), written to HBM: the
// supports to eo (non-temporal: nothing reads them back soon) and, when ro is
// given, r_n = exp(dc) / N.  Each case is a loop of its own without branches.
template <bool NEAR, bool WITH_R>
__device__ __forceinline__ void store_head_rows(const float* a, int N, int lane, float L,
                                                float* __restrict__ eo, float* __restrict__ ro) {
    const float fN = static_cast<float>(N);
#pragma unroll 4
    for (int n = lane; n < N; n += kWave) {
        const float dc = a[n] - L;
        __builtin_nontemporal_store(support_from_centred(dc, NEAR), eo + n);
        if constexpr (WITH_R) ro[n] = expf(dc) / fN;
    }
}

__device__ __forceinline__ void wave_softmax_store(float* a, int N, int lane,
                                                   float* __restrict__ eo,
                                                   float* __restrict__ ro) {
    float L;
    bool near;
    wave_softmax_stats(a, N, lane, L, near);
    if (near) {
        if (ro) store_head_rows<true, true>(a, N, lane, L, eo, ro);
        else store_head_rows<true, false>(a, N, lane, L, eo, ro);
    } else {
        if (ro) store_head_rows<false, true>(a, N, lane, L, eo, ro);
        else store_head_rows<false, false>(a, N, lane, L, eo, ro);
    }
}

// Eq. 1, 8 and 9 for one query head, computed by one wave with no workgroup
// barrier.  qh: the head's [N_T, d] queries; kh: its key head's [N, d] keys; a: N
// floats owned by the wave, in LDS or (GLOBAL) in global memory (the head's own
// output row, overwritten in place).  The first key batch is requested before
// the query mean, and each later batch before the previous one is used.
template <typename T, int D, bool GLOBAL = false>
__device__ __forceinline__ void wave_head(const T* __restrict__ qh, const T* __restrict__ kh,
                                          int NT, int N, float qscale, float* a, int lane,
                                          float* __restrict__ eo, float* __restrict__ ro,
                                          int64_t qld, int64_t kld) {
    using G = WaveRows<T, D>;
    const int wrow = lane / G::LPR, wl = lane % G::LPR;
    qh += wl * 8;
    kh += wl * 8;
    Packet<T> ka[G::KU], kb[G::KU];
    load_key_batch<T, D>(ka, kh, 0, wrow, N, kld);
    float qb[8];
    wave_query_mean<T, D>(qh, NT, wrow, qscale, qb, qld);
    // the requests are unconditional (rows past N are clamped and never used), so
    // the wait before a batch's first use leaves the next batch's loads pending
    for (int base = 0; base < N; base += 2 * G::BATCH) {
        load_key_batch<T, D>(kb, kh, base + G::BATCH, wrow, N, kld);
        key_batch_logits<T, D>(ka, qb, a, base, wrow, wl, N);
        if (base + G::BATCH >= N) break;
        load_key_batch<T, D>(ka, kh, base + 2 * G::BATCH, wrow, N, kld);
        key_batch_logits<T, D>(kb, qb, a, base + G::BATCH, wrow, wl, N);
    }
    if constexpr (GLOBAL) global_logits_sync();
    else wave_lds_sync();
    wave_softmax_store(a, N, lane, eo, ro);
}

}  // namespace e2s
