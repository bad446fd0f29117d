// Device-side helpers shared by the E2S kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>

namespace e2s {

constexpr int kWave = 64;

// ---------------------------------------------------------------------------
// bfloat16 / float loads: 8 consecutive elements of a row as fp32.
// ---------------------------------------------------------------------------
__device__ __forceinline__ float bf16lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// Raw 16-byte packets; converted after the loads are in flight.  Streamed
// operands are read once, so the loads carry the non-temporal hint.
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// Element types: uint16_t holds bfloat16 bits, _Float16 is IEEE half, float.
template <typename T> struct Packet;
template <> struct Packet<uint16_t> { u32x4 a; };
template <> struct Packet<_Float16> { u32x4 a; };
template <> struct Packet<float> { f32x4 a, b; };

__device__ __forceinline__ void load_packet(Packet<uint16_t>& p, const uint16_t* src) {
    p.a = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(src));
}
__device__ __forceinline__ void load_packet(Packet<_Float16>& p, const _Float16* src) {
    p.a = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(src));
}
__device__ __forceinline__ void load_packet(Packet<float>& p, const float* src) {
    p.a = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(src));
    p.b = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(src) + 1);
}
__device__ __forceinline__ void unpack(const Packet<uint16_t>& p, float* x) {
    x[0] = bf16lo(p.a.x); x[1] = bf16hi(p.a.x);
    x[2] = bf16lo(p.a.y); x[3] = bf16hi(p.a.y);
    x[4] = bf16lo(p.a.z); x[5] = bf16hi(p.a.z);
    x[6] = bf16lo(p.a.w); x[7] = bf16hi(p.a.w);
}
__device__ __forceinline__ float f16lo(uint32_t w) {
    return static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(w & 0xFFFFu)));
}
__device__ __forceinline__ float f16hi(uint32_t w) {
    return static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(w >> 16)));
}
__device__ __forceinline__ void unpack(const Packet<_Float16>& p, float* x) {
    x[0] = f16lo(p.a.x); x[1] = f16hi(p.a.x);
    x[2] = f16lo(p.a.y); x[3] = f16hi(p.a.y);
    x[4] = f16lo(p.a.z); x[5] = f16hi(p.a.z);
    x[6] = f16lo(p.a.w); x[7] = f16hi(p.a.w);
}
__device__ __forceinline__ void unpack(const Packet<float>& p, float* x) {
    x[0] = p.a.x; x[1] = p.a.y; x[2] = p.a.z; x[3] = p.a.w;
    x[4] = p.b.x; x[5] = p.b.y; x[6] = p.b.z; x[7] = p.b.w;
}

// ---------------------------------------------------------------------------
// Cross-lane sums inside a DPP row (16 lanes) or half row (8 lanes).  Every lane
// of the group ends with the same, bit-identical total.
// ---------------------------------------------------------------------------
template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, true));
}
constexpr int kQuadSwap1 = 0xB1;       // quad_perm [1,0,3,2]
constexpr int kQuadSwap2 = 0x4E;       // quad_perm [2,3,0,1]
constexpr int kRowHalfMirror = 0x141;  // lane i <- lane 7-i within each 8-lane half
constexpr int kRowMirror = 0x140;      // lane i <- lane 15-i within each 16-lane row

template <int LANES>
__device__ __forceinline__ float group_sum(float v) {
    static_assert(LANES == 8 || LANES == 16, "group of 8 or 16 lanes");
    v += dpp<kQuadSwap1>(v);
    v += dpp<kQuadSwap2>(v);
    v += dpp<kRowHalfMirror>(v);
    if constexpr (LANES == 16) v += dpp<kRowMirror>(v);
    return v;
}

__device__ __forceinline__ float wave_max(float v) {
    for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
    return v;
}
__device__ __forceinline__ float wave_sum(float v) {
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
    return v;
}

// L = log(S / N) for a softmax over N logits shifted by their maximum, with
// S = sum exp(a - max) and E = sum expm1(a - max) = S - N.  With S > N/2 the
// relative error of E is small and log1p(E / N) is exact to a few ulp; below
// that the logits are spread out, E is a sum of terms near -1 that has lost the
// small ones, and S is the accurate sum.
__device__ __forceinline__ float log_mean_exp(float E, float S, float n) {
    return (2.0f * S > n) ? log1pf(E / n) : logf(S / n);
}

// ---------------------------------------------------------------------------
// Order-preserving unsigned images of floating-point values (NaN sorts last).
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t ordered_bits(float x) {
    const uint32_t u = __float_as_uint(x);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ uint64_t ordered_bits(double x) {
    const uint64_t u = static_cast<uint64_t>(__double_as_longlong(x));
    return (u & 0x8000000000000000ull) ? ~u : (u | 0x8000000000000000ull);
}

// ---------------------------------------------------------------------------
// Evidence arithmetic (Sec. 4.1 Eq. 10-11, Sec. 4.2 Eq. 13-16), shared by the
// staged kernels and the fused kernel so that both produce identical bits.
// The library is compiled with -ffp-contract=off: every operation below rounds
// exactly as written.
// ---------------------------------------------------------------------------

// Eq. 10 from s1 = sum_h e_h and s2 = sum_h |e_h - ebar| (e = p - 1/2).
__device__ __forceinline__ float reliability_from_sums(float s1, float s2, float two_over_h) {
    const float clarity = two_over_h * fabsf(s1);
    const float consistency = 1.0f - two_over_h * s2;
    return clarity * consistency;
}

// Eq. 11 with pbar = 1/2 + ebar.
__device__ __forceinline__ void masses_from_reliability(float rho, float ebar, float& mI,
                                                        float& mU, float& mT) {
    mI = rho * (0.5f + ebar);
    mU = rho * (0.5f - ebar);
    mT = 1.0f - rho;
}

// One Dempster step (Eq. 13-16) of the running mass (aI, aU, aT) with (mI, mU, mT).
// Returns K; on total conflict the running mass becomes vacuous and K = 1.  The
// three normalisations share one correctly rounded reciprocal of 1 - K (one
// division sequence instead of three; each mass then carries at most two
// roundings from it).
__device__ __forceinline__ float ds_step(float& aI, float& aU, float& aT, float mI, float mU,
                                         float mT) {
    const float k = aI * mU + aU * mI;
    const float den = 1.0f - k;
    if (den > 0.0f) {
        const float inv = 1.0f / den;
        const float fI = (aI * mI + aI * mT + aT * mI) * inv;
        const float fU = (aU * mU + aU * mT + aT * mU) * inv;
        const float fT = (aT * mT) * inv;
        aI = fI;
        aU = fU;
        aT = fT;
        return k;
    }
    aI = 0.0f;
    aU = 0.0f;
    aT = 1.0f;
    return 1.0f;
}

// c = 1 - q of Eq. 19 using 1 - Pl(I) = m~(U) (Eq. 18).
__device__ __forceinline__ float priority_complement(float aU, float k_last) {
    return aU * (1.0f - k_last);
}

}  // namespace e2s
