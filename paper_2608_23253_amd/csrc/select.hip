// Spatial novelty and global top-K (Sec. 4.3 Eq. 20-23), one workgroup per image.
//
//  1. the image's complements c = 1 - q are staged in LDS (N <= 16384 floats);
//  2. cell representatives (Eq. 20-21): one wave per cell scans the cell's
//     row/column ranges and takes the minimum of the 64-bit key
//     (order-preserving bits of c) << 32 | index, i.e. the highest q with the
//     lowest index on ties;
//  3. adjusted complement c^ = (1 - lambda) c + lambda (1 - b) = 1 - q~ (Eq. 22),
//     evaluated in double precision with explicitly rounded operations; its
//     order-preserving 64-bit image is the ranking key;
//  4. the K-th smallest key T is found by a radix select over 8-bit digits (LDS
//     histogram + one wave's prefix scan per round, at most 8 rounds, fewer once
//     T's bin holds a single key), together with how many tokens equal to T must
//     still be taken; lanes of a wave that fall in the same bin are added with one
//     atomic;
//  5. tokens with key < T, plus the lowest-index tokens with key == T, are kept
//     (Eq. 23); two block-wide scans in token order write them in ascending order.
//
// Ranking by (c^, index) ascending is ranking by (q~ descending, index ascending).
// The greedy formulation (take the best remaining token K times) returns the same
// set; the radix select needs 8 rounds instead of K serial argmax steps.
#include "e2s_device.h"
#include "e2s_kernels.h"

namespace e2s {
namespace {

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int o) {
    const uint32_t lo = __shfl_xor(static_cast<uint32_t>(v), o);
    const uint32_t hi = __shfl_xor(static_cast<uint32_t>(v >> 32), o);
    return (static_cast<uint64_t>(hi) << 32) | lo;
}

__device__ __forceinline__ uint64_t wave_min_u64(uint64_t v) {
    for (int o = 32; o > 0; o >>= 1) {
        const uint64_t w = shfl_xor_u64(v, o);
        v = w < v ? w : v;
    }
    return v;
}

__device__ __forceinline__ uint32_t wave_inclusive_scan(uint32_t x, int lane) {
    for (int o = 1; o < kWave; o <<= 1) {
        const uint32_t y = __shfl_up(x, o);
        if (lane >= o) x += y;
    }
    return x;
}

// Exclusive prefix sum of x over the block in thread order.  buf holds >= waves words.
template <int THREADS>
__device__ uint32_t block_exclusive_scan(uint32_t x, uint32_t* buf) {
    constexpr int kW = THREADS / kWave;
    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    const uint32_t incl = wave_inclusive_scan(x, lane);
    if (lane == kWave - 1) buf[wave] = incl;
    __syncthreads();
    if (wave == 0) {
        const uint32_t v = lane < kW ? buf[lane] : 0u;
        const uint32_t vi = wave_inclusive_scan(v, lane);
        if (lane < kW) buf[lane] = vi - v;
    }
    __syncthreads();
    const uint32_t r = buf[wave] + incl - x;
    __syncthreads();
    return r;
}

template <int THREADS>
__global__ __launch_bounds__(THREADS) void spatial_select_kernel(
    const float* __restrict__ prio_c, int32_t* __restrict__ keep_idx, double* __restrict__ adj_out,
    uint8_t* __restrict__ rep_out, int N, int gh, int gw, int G, float lambda, int K) {
    constexpr int kW = THREADS / kWave;
    extern __shared__ unsigned char smem[];
    float* cs = reinterpret_cast<float*>(smem);                 // [N]
    uint32_t* hist = reinterpret_cast<uint32_t*>(cs + N);       // [256]
    uint32_t* scan = hist + 256;                                // [32]
    uint8_t* rep = reinterpret_cast<uint8_t*>(scan + 32);       // [N]
    __shared__ uint64_t s_prefix;
    __shared__ uint32_t s_rank;
    __shared__ uint32_t s_unique;
    __shared__ uint64_t s_found;

    const int tid = threadIdx.x, lane = tid % kWave, wave = tid / kWave;
    const int64_t b = blockIdx.x;
    const float* cb = prio_c + b * N;
    for (int n = tid; n < N; n += THREADS) {
        cs[n] = cb[n];
        rep[n] = 0;
    }
    __syncthreads();

    // ---- cell representatives ---------------------------------------------
    for (int cell = wave; cell < G * G; cell += kW) {
        const int gr = cell / G, gc = cell - gr * G;
        const int r0 = (gr * gh + G - 1) / G, r1 = ((gr + 1) * gh + G - 1) / G;
        const int c0 = (gc * gw + G - 1) / G, c1 = ((gc + 1) * gw + G - 1) / G;
        const int cw = c1 - c0, cnt = (r1 - r0) * cw;
        uint64_t best = ~0ull;
        for (int j = lane; j < cnt; j += kWave) {
            const int row = r0 + j / cw;
            const int n = row * gw + c0 + (j - (j / cw) * cw);
            const uint64_t key = (static_cast<uint64_t>(ordered_bits(cs[n])) << 32) |
                                 static_cast<uint32_t>(n);
            best = key < best ? key : best;
        }
        best = wave_min_u64(best);
        if (lane == 0 && cnt > 0) rep[static_cast<uint32_t>(best)] = 1;
    }
    __syncthreads();

    const double lam = static_cast<double>(lambda);
    const double oml = 1.0 - lam;
    auto adj = [&](int n) -> double {
        const double t = __dmul_rn(oml, static_cast<double>(cs[n]));
        return rep[n] ? t : __dadd_rn(t, lam);
    };
    if (adj_out || rep_out) {
        for (int n = tid; n < N; n += THREADS) {
            if (adj_out) adj_out[b * N + n] = adj(n);
            if (rep_out) rep_out[b * N + n] = rep[n];
        }
    }
    if (K <= 0) return;

    // ---- radix select of the K-th smallest key ----------------------------
    if (tid == 0) {
        s_prefix = 0;
        s_rank = static_cast<uint32_t>(K);
        s_unique = 0;
    }
    uint64_t mask = 0;
    for (int shift = 56; shift >= 0; shift -= 8) {
        for (int i = tid; i < 256; i += THREADS) hist[i] = 0;
        __syncthreads();
        const uint64_t prefix = s_prefix;
        if (s_unique) {
            // the previous round left one key with this prefix: it is the K-th key
            for (int n = tid; n < N; n += THREADS) {
                const uint64_t kk = ordered_bits(adj(n));
                if ((kk & mask) == prefix) s_found = kk;
            }
            __syncthreads();
            if (tid == 0) s_prefix = s_found;
            __syncthreads();
            break;
        }
        for (int base = 0; base < N; base += THREADS) {
            const int n = base + tid;
            const uint64_t kk = n < N ? ordered_bits(adj(n)) : 0ull;
            const bool match = n < N && (kk & mask) == prefix;
            const uint32_t digit = static_cast<uint32_t>(kk >> shift) & 255u;
            // early rounds put most keys of a wave in one bin: add them with one atomic
            const uint64_t mb = __ballot(match);
            if (mb) {
                const int leader = __ffsll(static_cast<unsigned long long>(mb)) - 1;
                const uint32_t d0 = __shfl(digit, leader);
                const uint64_t same = __ballot(match && digit == d0);
                if (same == mb) {
                    if (lane == leader) atomicAdd(&hist[d0], static_cast<uint32_t>(__popcll(mb)));
                } else if (match) {
                    atomicAdd(&hist[digit], 1u);
                }
            }
        }
        __syncthreads();
        if (wave == 0) {
            const uint32_t h0 = hist[4 * lane], h1 = hist[4 * lane + 1];
            const uint32_t h2 = hist[4 * lane + 2], h3 = hist[4 * lane + 3];
            const uint32_t local = h0 + h1 + h2 + h3;
            const uint32_t incl = wave_inclusive_scan(local, lane);
            const uint32_t rank = s_rank;
            const uint64_t hit = __ballot(incl >= rank);
            const int first = __ffsll(static_cast<unsigned long long>(hit)) - 1;
            if (lane == first) {
                uint32_t cum = incl - local;
                int digit = 4 * lane;
                if (cum + h0 < rank) {
                    cum += h0;
                    ++digit;
                    if (cum + h1 < rank) {
                        cum += h1;
                        ++digit;
                        if (cum + h2 < rank) {
                            cum += h2;
                            ++digit;
                        }
                    }
                }
                s_prefix = prefix | (static_cast<uint64_t>(digit) << shift);
                s_rank = rank - cum;
                s_unique = hist[digit] == 1u;
            }
        }
        mask |= 0xFFull << shift;
        __syncthreads();
    }
    const uint64_t T = s_prefix;
    const uint32_t need_eq = s_rank;   // tokens equal to T still to take, >= 1

    // ---- ordered compaction --------------------------------------------------
    const int chunk = (N + THREADS - 1) / THREADS;
    const int n0 = min(N, tid * chunk), n1 = min(N, n0 + chunk);
    uint32_t eq_local = 0;
    for (int n = n0; n < n1; ++n) eq_local += ordered_bits(adj(n)) == T;
    const uint32_t eq_before = block_exclusive_scan<THREADS>(eq_local, scan);
    uint32_t sel_local = 0, eqr = eq_before;
    for (int n = n0; n < n1; ++n) {
        const uint64_t kk = ordered_bits(adj(n));
        const bool take = kk < T || (kk == T && eqr < need_eq);
        eqr += kk == T;
        sel_local += take;
    }
    uint32_t pos = block_exclusive_scan<THREADS>(sel_local, scan);
    eqr = eq_before;
    int32_t* out = keep_idx + b * K;
    for (int n = n0; n < n1; ++n) {
        const uint64_t kk = ordered_bits(adj(n));
        const bool take = kk < T || (kk == T && eqr < need_eq);
        eqr += kk == T;
        if (take && pos < static_cast<uint32_t>(K)) out[pos++] = n;
    }
}

template <int THREADS>
hipError_t launch_sel(const Dims& d, int cells, float lambda, int keep, const float* c,
                      int32_t* keep_idx, double* adj, uint8_t* rep, hipStream_t st) {
    const size_t lds = static_cast<size_t>(d.N) * sizeof(float) + (256 + 32) * sizeof(uint32_t) +
                       align_up(static_cast<size_t>(d.N), 16);
    auto kern = spatial_select_kernel<THREADS>;
    if (lds > 64 * 1024) {
        hipError_t err = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                             hipFuncAttributeMaxDynamicSharedMemorySize,
                                             static_cast<int>(lds));
        if (err != hipSuccess) return err;
    }
    hipLaunchKernelGGL(kern, dim3(static_cast<unsigned>(d.B)), dim3(THREADS), lds, st, c,
                       keep_idx, adj, rep, static_cast<int>(d.N), static_cast<int>(d.gh),
                       static_cast<int>(d.gw), cells, lambda, keep);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_spatial_select(const Dims& d, int cells, float lambda, int keep,
                                 const float* prio_c, int32_t* keep_idx, double* adj_c,
                                 uint8_t* is_rep, hipStream_t st) {
    if (d.N <= 2048)
        return launch_sel<256>(d, cells, lambda, keep, prio_c, keep_idx, adj_c, is_rep, st);
    return launch_sel<1024>(d, cells, lambda, keep, prio_c, keep_idx, adj_c, is_rep, st);
}

}  // namespace e2s
