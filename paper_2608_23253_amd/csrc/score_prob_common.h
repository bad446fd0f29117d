// Per-tile arithmetic of the mean-of-probabilities score stage (Sec. 3.1 Eq. 1;
// Sec. 4.1 Eq. 8-9 with the softmax taken per text query, then averaged), used
// by score_prob.hip.
//
// A 16 x 16 product tile holds, in lane (lr, lg), the logits of keys
// 16 t + 4 lg + r (r = 0..3) against query lr of a 16-query block.  Every
// decision of the stage (which keys count, the series or the library, when the
// running maximum moves) is taken per tile, and each lane's sums run over its
// tiles in ascending order, so the results do not depend on how many tiles a wave
// takes at once (the library is compiled without floating-point contraction).
#pragma once

#include "e2s_device.h"
#include "score_common.h"

namespace e2s {

typedef float f32x4v __attribute__((ext_vector_type(4)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));

namespace prob {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;

// expm1(s y) = s y P(y) with P the Taylor series of the scaled argument:
// coefficients s^k / (k+1)! for k = 1 .. DEG-1.  Degree 5 on |s y| <= 1/8 and
// degree 6 on |s y| <= 1/4 (truncation x^7 / 5040, below 6e-8 relative there)
// stay under one float32 ulp.  The scale is applied once per sum instead of once
// per logit, and the callers fold the last product into their running sums.
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

// 16 keys x 16 queries on the matrix cores, fp32 accumulation from zero.
template <int NA>
__device__ __forceinline__ f32x4v tile_mma(const bf16x8 (&a)[NA], const bf16x8 (&b)[NA]) {
    f32x4v acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < NA; ++s) acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[s], b[s], acc, 0, 0, 0);
    return acc;
}
template <int NA>
__device__ __forceinline__ f32x4v tile_mma(const f16x8 (&a)[NA], const f16x8 (&b)[NA]) {
    f32x4v acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < NA; ++s) acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(a[s], b[s], acc, 0, 0, 0);
    return acc;
}
template <int NA>
__device__ __forceinline__ f32x4v tile_mma(const float (&a)[NA], const float (&b)[NA]) {
    f32x4v acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < NA; ++s) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a[s], b[s], acc, 0, 0, 0);
    return acc;
}

// Range of the tight path: every centred logit |s (z - c_t)| of a query chunk
// within 1/16.  There expm1 to degree 4 (terms up to x^4 / 24) truncates below
// x^5 / 120, i.e. 1.3e-7 of the term at the edge and far less for the bulk of the
// logits (about 1/100 at the workloads' scale).
constexpr float kTightRange = 0.0625f;

// Reference of a query (in logit units, before the scale): the mean logit
// Q_t.K_n over keys 0..15, summed pairwise so that equal logits give exactly
// their value, or key 0's logit when N < 16.  z: the product of key tile 0 with
// the query block; every lane of the wave gets the value of its query lr.
__device__ __forceinline__ float block_reference(const f32x4v& z, int N, int lr) {
    float sum = (z[0] + z[1]) + (z[2] + z[3]);
    sum += __shfl_xor(sum, 16);
    sum += __shfl_xor(sum, 32);
    const float z0 = __shfl(z[0], lr);            // key 0, from lane (lr, 0)
    return (N >= 16) ? sum * (1.0f / 16.0f) : z0;
}

// Pass 1, near uniform: E += expm1(s y) = s y P(y) (in units of s) for the
// tile's logits with y = z - c_t / s; keys past N count as y = 0.  P: the
// degree-4 series in the tight range (|s y| <= 1/16), else degree 5 (<= 1/8).
// amax: the largest |y| seen, to confirm afterwards that the range held.  WHOLE:
// the caller knows that every key of the tile is below N (the same arithmetic
// without the masking).
// SPLIT: x = y P(y) is rounded before it is added (as the register-resident
// kernel, which keeps x, adds it), else added in one fused step.
template <bool WHOLE, bool SPLIT, typename Series>
__device__ __forceinline__ void series_tile(const f32x4v& z, float cz, int key0, int N,
                                            const Series& p, float& E, float& amax) {
    const bool full = WHOLE || key0 + 4 <= N;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        float y = z[r] - cz;
        if (!full) y = (key0 + r < N) ? y : 0.f;
        amax = fmaxf(amax, fabsf(y));
        if constexpr (SPLIT)
            E += p(y) * y;
        else
            E = fmaf(p(y), y, E);
    }
}

// Pass 1, peaked attention: online statistics of one tile with the running
// maximum m of the scaled logits as reference; E = sum expm1(x), S = sum exp(x)
// over x = z s - m of the valid keys; cnt: valid keys this lane has seen before
// this tile.  The wave-wide tests make the tile's update uniform (series where
// every x of the wave lies within 1/8 of the maximum, else the library).
__device__ __forceinline__ void online_tile(const f32x4v& z, float scale, int key0, int N,
                                            float cnt, float& m, float& E, float& S) {
    float zmax = -INFINITY, zmin = INFINITY, cntt = 0.f;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const bool ok = key0 + r < N;
        zmax = fmaxf(zmax, ok ? z[r] : -INFINITY);
        zmin = fminf(zmin, ok ? z[r] : INFINITY);
        cntt += ok ? 1.f : 0.f;
    }
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
    const bool near = cntt == 0.f || fmaf(zmin, scale, -mx) >= -kSeriesRange;
    if (__all(near)) {
        float el = 0.f;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const float t = expm1_series(fmaf(z[r], scale, -mx));
            el += (key0 + r < N) ? t : 0.f;
        }
        E += el;
        S += cntt + el;
    } else {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            if (key0 + r < N) {
                const float x = fmaf(z[r], scale, -mx);
                const float t = expm1f(x);
                E += t;
                S += (x < -0.5f) ? expf(x) : 1.0f + t;
            }
        }
    }
}

// Valid keys of the tile seen by this lane (0..4).
__device__ __forceinline__ float tile_count(int key0, int N) {
    return static_cast<float>(min(max(N - key0, 0), 4));
}

// Merge of the near-uniform statistics of one query: E = s e with e the sum of
// the four wave partials (in order); S = N + E >= N exp(-1/8) > N / 2, so
// L = log1p(E / N) (as log_mean_exp); the shift of pass 2 in logit units is
// c_t / s + L / s.
__device__ __forceinline__ float near_shift(float cz, float e, float scale, float fN) {
    return cz + log1pf((scale * e) / fN) / scale;
}

// Merge of the online statistics: the four lane groups of a wave (shuffles), then
// the waves (parts p[w] = {M or -inf, e, s, c} in wave order).
struct OnlinePart {
    float M, e, s, c;
};
__device__ __forceinline__ OnlinePart online_wave_part(float m, float E, float S, float cnt) {
    float M = fmaxf(m, __shfl_xor(m, 16));
    M = fmaxf(M, __shfl_xor(M, 32));
    float e = 0.f, s = 0.f;
    if (cnt > 0.f) {
        const float dm = m - M;
        e = fmaf(cnt, expm1f(dm), E * expf(dm));
        s = S * expf(dm);
    }
    float c = cnt;
    e += __shfl_xor(e, 16);
    s += __shfl_xor(s, 16);
    c += __shfl_xor(c, 16);
    e += __shfl_xor(e, 32);
    s += __shfl_xor(s, 32);
    c += __shfl_xor(c, 32);
    return OnlinePart{(c > 0.f) ? M : -INFINITY, e, s, c};
}
// p: the wave parts of one query, 4 floats apart by `stride` floats per wave;
// returns the shift m + L of pass 2 (scaled-logit units).
__device__ __forceinline__ float online_shift(const float* p, int stride, float fN) {
    float M = -INFINITY;
    for (int w = 0; w < kWaves; ++w) M = fmaxf(M, p[w * stride]);
    float e = 0.f, s = 0.f;
    for (int w = 0; w < kWaves; ++w) {
        const float* pw = p + w * stride;
        if (pw[0] == -INFINITY) continue;         // this wave saw no key
        const float dm = pw[0] - M;
        e += fmaf(pw[3], expm1f(dm), pw[1] * expf(dm));
        s += pw[2] * expf(dm);
    }
    return M + log_mean_exp(e, s, fN);
}

// Pass 2, near uniform: col += expm1(s y) / s = y P(y) with y = z - shift, per key
// of the tile, over the query blocks in order; P: the degree-6 series (|s y| <=
// 1/4), or in the tight range degree 4 (|s y| <= 1/16) or 5 (<= 1/8).
template <typename Series>
__device__ __forceinline__ void column_series_tile(const f32x4v& z, float sz, const Series& p,
                                                   float (&col)[4]) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const float y = z[r] - sz;
        col[r] = fmaf(p(y), y, col[r]);
    }
}

// Sum over a head's queries of a per-query value held by lane t of one wave (0 in
// lanes past N_T; at most 64 queries): the butterfly of wave_sum, whose order
// depends only on the lanes, so every kernel that takes it gets the same bits.
__device__ __forceinline__ float query_sum(float v) { return wave_sum(v); }

// Pass 2 in the tight range: col += w_t x with x = expm1(s y) / s = y P(y),
// y = z - c_t, evaluated exactly as pass 1 evaluates it (series_tile), over the
// query blocks in order.  Keys past N are not masked: their sums are never kept.
template <typename Series>
__device__ __forceinline__ void column_weighted_tile(const f32x4v& z, float cz, const Series& p,
                                                     float w, float (&col)[4]) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const float y = z[r] - cz;
        col[r] = fmaf(w, p(y) * y, col[r]);
    }
}

// Pass 2, peaked attention: col += expm1(x) with x = z s - shift, by the series
// where every x of the wave's tile lies within 1/8 of zero, else the library.
__device__ __forceinline__ void column_far_tile(const f32x4v& z, float scale, float shift,
                                                float (&col)[4]) {
    float x[4];
    float xmin = INFINITY, xmax = -INFINITY;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        x[r] = fmaf(z[r], scale, -shift);
        xmin = fminf(xmin, x[r]);
        xmax = fmaxf(xmax, x[r]);
    }
    if (__all(fmaxf(-xmin, xmax) <= kSeriesRange)) {
#pragma unroll
        for (int r = 0; r < 4; ++r) col[r] += expm1_series(x[r]);
    } else {
#pragma unroll
        for (int r = 0; r < 4; ++r) col[r] += expm1f(x[r]);
    }
}

// Support and share of one key from its column sum: u = N r - 1 = sum / N_T in
// centred form (sum = unit times the summed columns, unit = s or 1); e = p - 1/2
// = u / (2 (2 + u)) (Eq. 9), r = (1 + u) / N.
__device__ __forceinline__ float column_u(float sum, float unit, float inv_nt) {
    return (0.f + unit * sum) * inv_nt;
}
__device__ __forceinline__ float support_from_u(float u) { return u / (2.0f * (2.0f + u)); }

}  // namespace prob
}  // namespace e2s
