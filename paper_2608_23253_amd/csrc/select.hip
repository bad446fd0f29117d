// Spatial novelty and global top-K (Sec. 4.3 Eq. 20-23), one workgroup per image:
// one thread per token (in whole waves) up to 1024 tokens, 1024 threads above.
//
// Thread t owns the consecutive tokens n0 = t * chunk .. n0 + chunk - 1
// (chunk = ceil(N / 1024) above 1024 tokens, else one token) and keeps their values in
// registers throughout.  The work per image is a few KB, so the kernel is bound
// by latency: every step below is shaped to need few dependent LDS round trips
// and workgroup barriers.  An image of more than 16384 tokens is taken in
// segments of 16384 (16 per thread), every pass below visiting the segments in
// order and reloading (or recomputing) their values.
//
//  1. cell representatives (Eq. 20-21): the 64-bit key
//     (order-preserving bits of c) << 32 | index is minimised per cell, i.e. the
//     highest q with the lowest index on ties.  Lanes holding tokens of one cell
//     first combine their keys with DPP row shifts (a segmented minimum inside
//     each 16-lane row); the last lane of each run folds it into the cell's LDS
//     slot with an atomic minimum;
//  2. adjusted complement c^ = (1 - lambda) c + lambda (1 - b) = 1 - q~ (Eq. 22),
//     evaluated in double precision with explicitly rounded operations; its
//     order-preserving 64-bit image is the ranking key;
//  3. the K-th smallest key T is found by a radix select over 8-bit digits,
//     starting at the highest bit in which the image's smallest and largest keys
//     differ, together with how many tokens equal to T must still be taken.  Each
//     round adds the matching keys into an LDS histogram (lanes of a wave that
//     share a bin with one atomic, since same-word LDS atomics serialise), then
//     after one barrier every wave scans the histogram itself and takes the same
//     digit; three histograms in rotation let a round clear the next round's
//     buffer without a second barrier.  The rounds stop once T's bin holds a
//     single key: T is then the one key with the digits chosen so far, and the
//     compaction compares keys with those high bits only (no search for T);
//  4. tokens with key < T, plus the lowest-index tokens with key == T, are kept
//     (Eq. 23); one block-wide scan of the per-thread counts places them in
//     ascending token order.
//
// A pruning operation over a candidate subset (the progressive schedule) passes
// the candidates' raster positions: cells come from the positions, a cell is
// occupied when it holds a candidate, and the token index of every tie rule is
// the candidate index.  A position outside the grid gives its token no cell.
//
// Ranking by (c^, index) ascending is ranking by (q~ descending, index ascending).
// The greedy formulation (take the best remaining token K times) returns the same
// set; the radix select needs a handful of rounds instead of K argmax steps.
#include "e2s_device.h"
#include "e2s_kernels.h"

namespace e2s {
namespace {

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / kWave;
constexpr int kMaxChunk = 16;          // tokens per thread and segment
constexpr int kRowShl1 = 0x101;

template <int CTRL>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t v, uint32_t fill) {
    return static_cast<uint32_t>(__builtin_amdgcn_update_dpp(
        static_cast<int>(fill), static_cast<int>(v), CTRL, 0xF, 0xF, false));
}
template <int CTRL>
__device__ __forceinline__ uint64_t dpp_u64(uint64_t v, uint64_t fill) {
    const uint32_t hi = dpp_u32<CTRL>(static_cast<uint32_t>(v >> 32), static_cast<uint32_t>(fill >> 32));
    const uint32_t lo = dpp_u32<CTRL>(static_cast<uint32_t>(v), static_cast<uint32_t>(fill));
    return (static_cast<uint64_t>(hi) << 32) | lo;
}
__device__ __forceinline__ uint32_t readlane_u32(uint32_t v, int l) {
    return static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(v), l));
}
__device__ __forceinline__ uint64_t readlane_u64(uint64_t v, int l) {
    return (static_cast<uint64_t>(readlane_u32(static_cast<uint32_t>(v >> 32), l)) << 32) |
           readlane_u32(static_cast<uint32_t>(v), l);
}

constexpr int kRowShr1 = 0x111, kRowShr2 = 0x112, kRowShr4 = 0x114, kRowShr8 = 0x118;

// Inclusive prefix sum across the wave: shifts by 1, 2, 4, 8 lanes inside each
// 16-lane DPP row (lanes shifted in from outside the row add 0), then the totals
// of the earlier rows, read from lanes 15, 31 and 47, are added.
__device__ __forceinline__ uint32_t wave_inclusive_scan(uint32_t x, int lane) {
    x += dpp_u32<kRowShr1>(x, 0u);
    x += dpp_u32<kRowShr2>(x, 0u);
    x += dpp_u32<kRowShr4>(x, 0u);
    x += dpp_u32<kRowShr8>(x, 0u);
    const uint32_t t0 = readlane_u32(x, 15), t1 = readlane_u32(x, 31), t2 = readlane_u32(x, 47);
    const int row = lane >> 4;
    return x + (row >= 1 ? t0 : 0u) + (row >= 2 ? t1 : 0u) + (row >= 3 ? t2 : 0u);
}

// One step of the segmented minimum: take the key of the lane S places lower in
// the row when it belongs to the same cell (lanes shifted in from outside the row
// carry cell -1 and the largest key).
template <int CTRL>
__device__ __forceinline__ void seg_min_step(uint64_t& key, int cell) {
    const uint64_t k2 = dpp_u64<CTRL>(key, ~0ull);
    const int c2 = static_cast<int>(dpp_u32<CTRL>(static_cast<uint32_t>(cell), 0xFFFFFFFFu));
    key = (c2 == cell && k2 < key) ? k2 : key;
}

// Wave-wide minimum and maximum of 64-bit values, in every lane: quad swaps and
// half-row / row mirrors inside each 16-lane row, then the four row results.
template <int CTRL>
__device__ __forceinline__ void minmax_step(uint64_t& mn, uint64_t& mx) {
    const uint64_t a = dpp_u64<CTRL>(mn, 0ull), b = dpp_u64<CTRL>(mx, 0ull);
    mn = a < mn ? a : mn;
    mx = b > mx ? b : mx;
}
__device__ __forceinline__ void wave_minmax_u64(uint64_t& mn, uint64_t& mx) {
    minmax_step<kQuadSwap1>(mn, mx);
    minmax_step<kQuadSwap2>(mn, mx);
    minmax_step<kRowHalfMirror>(mn, mx);
    minmax_step<kRowMirror>(mn, mx);
    uint64_t a = readlane_u64(mn, 0), b = readlane_u64(mx, 0);
#pragma unroll
    for (int r = 16; r < kWave; r += 16) {
        const uint64_t ar = readlane_u64(mn, r), br = readlane_u64(mx, r);
        a = ar < a ? ar : a;
        b = br > b ? br : b;
    }
    mn = a;
    mx = b;
}

// Workgroup-shared state of a selection besides the per-cell slots.
struct SelectShared {
    uint32_t hist[3][256];
    uint32_t scan[kWaves];
    uint64_t wlo[kWaves], whi[kWaves];
};

// Token layout of one image's selection.  An image of at most kSegment tokens is
// one segment: thread t owns tokens n0 = t * chunk .. n0 + chunk - 1 (chunk =
// ceil(N / threads)) and keeps their values in registers through every pass.  A
// larger image is cut into segments of kSegment tokens (chunk = kMaxChunk); each
// pass visits the segments in order and has the caller load the segment's values
// again.  Every decision is an exact comparison of integer keys, so the kept set
// does not depend on the layout.
constexpr int kSegment = kThreads * kMaxChunk;

// Selection of one image (Eq. 20-23).  load(n0, cnt, first) fills the caller's
// registers for the tokens n0 .. n0 + cnt - 1 (cnt <= chunk; entries past cnt
// are never used): cv[j] = c, posv[j] = raster position, and whatever keep()
// reads; first is set on the first visit of each token (per-token outputs are
// written then).  best: G*G words of LDS; tok: the image's first token in the
// optional per-token outputs.  Calls keep(slot, n, j) once for every kept token n
// (slot = its rank in ascending token order; j its register).  All threads of the
// workgroup call it.
template <int MAXC, typename Load, typename Keep>
__device__ void select_image(const float (&cv)[MAXC], const int (&posv)[MAXC], Load&& load,
                             uint64_t* best, SelectShared& sh, int64_t tok,
                             double* __restrict__ adj_out, uint8_t* __restrict__ rep_out, int N,
                             int gh, int gw, int G, float lambda, int K, Keep&& keep) {
    const int tid = threadIdx.x, lane = tid % kWave, wave = tid / kWave;
    // images of at most 1024 tokens run with one thread per token, rounded up to
    // whole waves; larger ones with kThreads
    const int nthreads = blockDim.x, nwaves = nthreads / kWave;
    const int nseg = MAXC == kMaxChunk ? (N + kSegment - 1) / kSegment : 1;
    const bool streamed = nseg > 1;
    const int chunk = streamed ? kMaxChunk : (N + nthreads - 1) / nthreads;
    auto first_of = [&](int s) { return min(N, s * kSegment + tid * chunk); };
    auto count_of = [&](int n0) { return max(0, min(N - n0, chunk)); };
    // the tokens of segment s in the registers: a single segment is loaded once,
    // before the barrier below (its memory latency overlaps the LDS set-up), the
    // segments of a larger image on every visit
    auto load_segment = [&](int s, bool first) {
        const int n0 = first_of(s);
        load(n0, count_of(n0), first);
    };
    auto visit = [&](int s, bool first) {
        if (streamed) load_segment(s, first);
    };
    if (!streamed) load_segment(0, true);

    for (int i = tid; i < G * G; i += nthreads) best[i] = ~0ull;
    for (int i = tid; i < 256; i += nthreads) sh.hist[0][i] = 0u;
    __syncthreads();

    int cell[MAXC];
    auto cells_of = [&](int cnt) {
#pragma unroll
        for (int j = 0; j < MAXC; ++j) {
            if (j >= chunk) break;
            const int pos = posv[j];
            const bool placed = j < cnt && pos >= 0 && pos < gh * gw;
            const int row = pos / gw, col = pos - (pos / gw) * gw;
            cell[j] = placed ? (row * G / gh) * G + col * G / gw : -1 - lane;
        }
    };

    // ---- cell representatives (Eq. 20) -----------------------------------
    for (int s = 0; s < nseg; ++s) {
        visit(s, true);
        const int n0 = first_of(s), cnt = count_of(n0);
        cells_of(cnt);
#pragma unroll
        for (int j = 0; j < MAXC; ++j) {
            if (j >= chunk) break;
            const bool placed = cell[j] >= 0;
            uint64_t key = j < cnt ? (static_cast<uint64_t>(ordered_bits(cv[j])) << 32) |
                                         static_cast<uint32_t>(n0 + j)
                                   : ~0ull;
            seg_min_step<kRowShr1>(key, cell[j]);
            seg_min_step<kRowShr2>(key, cell[j]);
            seg_min_step<kRowShr4>(key, cell[j]);
            seg_min_step<kRowShr8>(key, cell[j]);
            // the last lane of each run inside the row holds the run's minimum
            const int next = static_cast<int>(
                __builtin_amdgcn_update_dpp(-1, cell[j], kRowShl1, 0xF, 0xF, false));
            const bool last = next != cell[j];   // lane 15 of a row reads -1
            if (placed && last)
                atomicMin(reinterpret_cast<unsigned long long*>(best + cell[j]),
                          static_cast<unsigned long long>(key));
        }
    }
    __syncthreads();

    // ---- ranking keys (Eq. 21-22) ------------------------------------------
    const double lam = static_cast<double>(lambda);
    const double oml = 1.0 - lam;
    uint64_t kk[MAXC];
    auto keys_of = [&](int n0, int cnt, bool outputs) {
        cells_of(cnt);
#pragma unroll
        for (int j = 0; j < MAXC; ++j) {
            kk[j] = ~0ull;
            if (j >= chunk) break;
            if (j < cnt) {
                const int n = n0 + j;
                const bool rep = cell[j] >= 0 &&
                                 static_cast<uint32_t>(best[cell[j]]) == static_cast<uint32_t>(n);
                const double t = __dmul_rn(oml, static_cast<double>(cv[j]));
                const double adj = rep ? t : __dadd_rn(t, lam);
                kk[j] = ordered_bits(adj);
                if (outputs && adj_out) adj_out[tok + n] = adj;
                if (outputs && rep_out) rep_out[tok + n] = rep ? 1 : 0;
            }
        }
    };
    // later passes over a streamed image recompute the keys of each segment
    auto revisit = [&](int s) {
        if (streamed) {
            visit(s, false);
            const int n0 = first_of(s);
            keys_of(n0, count_of(n0), false);
        }
    };
    uint64_t kmin = ~0ull, kmax = 0ull;
    for (int s = 0; s < nseg; ++s) {
        visit(s, false);
        const int n0 = first_of(s), cnt = count_of(n0);
        keys_of(n0, cnt, true);
#pragma unroll
        for (int j = 0; j < MAXC; ++j) {
            if (j >= chunk) break;
            if (j < cnt) {
                kmin = kk[j] < kmin ? kk[j] : kmin;
                kmax = kk[j] > kmax ? kk[j] : kmax;
            }
        }
    }
    if (K <= 0) return;
    wave_minmax_u64(kmin, kmax);
    if (lane == 0) {
        sh.wlo[wave] = kmin;
        sh.whi[wave] = kmax;
    }
    __syncthreads();
    // the waves' ranges, combined across lanes of every wave at once
    uint64_t lo = lane < nwaves ? sh.wlo[lane] : ~0ull, hi = lane < nwaves ? sh.whi[lane] : 0ull;
    wave_minmax_u64(lo, hi);

    // ---- radix select of the K-th smallest key (Eq. 23) -----------------------
    // The K-th key T is known as (mask, prefix): T & mask == prefix, and no other
    // key carries that prefix unless mask covers every bit (then T == prefix).  So
    // a key is below T iff (key & mask) < prefix, and equals T iff
    // (key & mask) == prefix.  need_eq: how many keys equal to T are taken.
    uint64_t mask = ~0ull, prefix = lo;     // all keys equal: T = lo, take K of them
    uint32_t need_eq = static_cast<uint32_t>(K);
    if (lo != hi) {
        const int top = 63 - __clzll(static_cast<long long>(lo ^ hi));
        mask = top == 63 ? 0ull : (~0ull << (top + 1));
        prefix = lo & mask;                 // bits above top: common to every key
        uint32_t rank = static_cast<uint32_t>(K);
        int shift = top >= 7 ? top - 7 : 0;
        for (int round = 0;; ++round) {
            uint32_t* h = sh.hist[round % 3];
            // the buffer after this one was last read before the previous barrier
            for (int i = tid; i < 256; i += nthreads) sh.hist[(round + 1) % 3][i] = 0u;
            for (int s = 0; s < nseg; ++s) {
                revisit(s);
                const int cnt = count_of(first_of(s));
#pragma unroll
                for (int j = 0; j < MAXC; ++j) {
                    if (j >= chunk) break;
                    const bool match = j < cnt && (kk[j] & mask) == prefix;
                    const uint32_t digit = static_cast<uint32_t>(kk[j] >> shift) & 255u;
                    uint64_t mb = __ballot(match);
                    for (int it = 0; it < 2 && mb; ++it) {
                        const int leader = __ffsll(static_cast<unsigned long long>(mb)) - 1;
                        const uint32_t d0 = readlane_u32(digit, leader);
                        const uint64_t same = __ballot(match && digit == d0);
                        if (lane == leader) atomicAdd(&h[d0], static_cast<uint32_t>(__popcll(same)));
                        mb &= ~same;
                    }
                    if ((mb >> lane) & 1ull) atomicAdd(&h[digit], 1u);
                }
            }
            __syncthreads();
            // every wave finds the bin that holds the rank-th matching key
            const uint32_t h0 = h[4 * lane], h1 = h[4 * lane + 1];
            const uint32_t h2 = h[4 * lane + 2], h3 = h[4 * lane + 3];
            const uint32_t local = h0 + h1 + h2 + h3;
            const uint32_t incl = wave_inclusive_scan(local, lane);
            const int first = __ffsll(static_cast<unsigned long long>(__ballot(incl >= rank))) - 1;
            uint32_t cum = readlane_u32(incl - local, first);
            const uint32_t g0 = readlane_u32(h0, first), g1 = readlane_u32(h1, first);
            const uint32_t g2 = readlane_u32(h2, first), g3 = readlane_u32(h3, first);
            uint32_t digit = 4 * first, cnt_d = g0;
            if (cum + g0 < rank) {
                cum += g0;
                ++digit;
                cnt_d = g1;
                if (cum + g1 < rank) {
                    cum += g1;
                    ++digit;
                    cnt_d = g2;
                    if (cum + g2 < rank) {
                        cum += g2;
                        ++digit;
                        cnt_d = g3;
                    }
                }
            }
            prefix |= static_cast<uint64_t>(digit) << shift;
            rank -= cum;
            mask |= 0xFFull << shift;
            if (cnt_d == 1u) {              // one key carries this prefix: the K-th
                need_eq = 1u;
                break;
            }
            if (shift == 0) {               // every bit is fixed: T == prefix
                need_eq = rank;
                break;
            }
            shift = shift >= 8 ? shift - 8 : 0;
        }
    }

    // ---- ordered compaction ----------------------------------------------------
    // per segment (at most 16384 tokens) both prefix sums ride in one word; the
    // counts of earlier segments are carried
    uint32_t lt_carry = 0, eq_carry = 0;
    for (int s = 0; s < nseg; ++s) {
        revisit(s);
        const int n0 = first_of(s), cnt = count_of(n0);
        uint32_t lt = 0, eq = 0;
#pragma unroll
        for (int j = 0; j < MAXC; ++j) {
            if (j >= chunk) break;
            if (j < cnt) {
                lt += (kk[j] & mask) < prefix;
                eq += (kk[j] & mask) == prefix;
            }
        }
        const uint32_t packed = (lt << 16) | eq;
        const uint32_t incl = wave_inclusive_scan(packed, lane);
        if (lane == kWave - 1) sh.scan[wave] = incl;
        __syncthreads();
        uint32_t before = incl - packed, total = 0;
        for (int w = 0; w < nwaves; ++w) {
            const uint32_t v = sh.scan[w];
            if (w < wave) before += v;
            total += v;
        }
        uint32_t lt_run = lt_carry + (before >> 16), eq_run = eq_carry + (before & 0xFFFFu);
#pragma unroll
        for (int j = 0; j < MAXC; ++j) {
            if (j >= chunk) break;
            if (j < cnt) {
                uint32_t pos = static_cast<uint32_t>(K);
                const uint64_t hk = kk[j] & mask;
                if (hk < prefix) {
                    pos = lt_run + (eq_run < need_eq ? eq_run : need_eq);
                    ++lt_run;
                } else if (hk == prefix) {
                    if (eq_run < need_eq) pos = lt_run + eq_run;
                    ++eq_run;
                }
                if (pos < static_cast<uint32_t>(K)) keep(static_cast<int>(pos), n0 + j, j);
            }
        }
        lt_carry += total >> 16;
        eq_carry += total & 0xFFFFu;
        if (streamed) __syncthreads();      // sh.scan is written again for the next segment
    }
}

template <int MAXC>
__global__ __launch_bounds__(kThreads) void spatial_select_kernel(
    const float* __restrict__ prio_c, int32_t* __restrict__ keep_idx, double* __restrict__ adj_out,
    uint8_t* __restrict__ rep_out, int N, int gh, int gw, int G, float lambda, int K) {
    extern __shared__ uint64_t best[];
    __shared__ SelectShared sh;
    const int64_t b = blockIdx.x;
    const float* cb = prio_c + b * N;
    float cv[MAXC];
    int posv[MAXC];
    auto load = [&](int n0, int cnt, bool) {
#pragma unroll
        for (int j = 0; j < MAXC; ++j) {
            cv[j] = j < cnt ? cb[n0 + j] : 0.f;
            posv[j] = n0 + j;
        }
    };
    select_image<MAXC>(cv, posv, load, best, sh, b * N, adj_out, rep_out, N, gh, gw, G, lambda, K,
                       [&](int slot, int n, int) { keep_idx[b * K + slot] = n; });
}

// Raster positions of the tokens n0 .. n0 + cnt - 1 (candidate positions when
// given).
template <int MAXC>
__device__ __forceinline__ void token_positions(int (&posv)[MAXC], const int32_t* cand_pos,
                                                int64_t tok, int n0, int cnt) {
#pragma unroll
    for (int j = 0; j < MAXC; ++j)
        posv[j] = cand_pos ? (j < cnt ? cand_pos[tok + n0 + j] : -1) : n0 + j;
}

// How an operation fuses its layers (Eq. 11-19); the ablation variants change one
// step each (e2s.h).  m_prev, when given, is the candidates' fused mass from
// earlier operations: every layer is combined onto it.
struct FusionPlan {
    bool unit_rho;   // rho = 1 (no head reliability)
    bool carried;    // combine onto m_prev
    bool protect;    // Eq. 19's conflict factor
    int l_first, l_end;
};
__device__ __forceinline__ FusionPlan fusion_plan(const SelectArgs& a, const float* m_prev, int L) {
    const bool last_only = a.variant == E2S_VARIANT_NO_LAYER_FUSION;
    FusionPlan f;
    f.unit_rho = a.variant == E2S_VARIANT_NO_HEAD_RELIABILITY;
    f.carried = m_prev != nullptr && !last_only;
    f.protect = a.variant != E2S_VARIANT_NO_CONFLICT;
    f.l_first = last_only ? L - 1 : 0;
    f.l_end = L;
    return f;
}

// Eq. 11-19 for the tokens n0 .. n0 + cnt - 1 (cnt <= MAXC) of the image whose
// tokens start at `tok`: the fused masses (aI, aU, aT) and the conflict kl of the
// last combination (0 when nothing was combined), from the per-layer rho and
// pbar_c.  The per-token arithmetic is that of the staged mass and Dempster
// kernels and does not depend on MAXC.  With up to 2 tokens per call every
// layer's inputs are requested at once; with up to 4, each layer's before the
// previous layer is combined.
template <int MAXC>
__device__ __forceinline__ void fuse_tokens(const float* __restrict__ rho,
                                            const float* __restrict__ pbar_c,
                                            const float* __restrict__ m_prev, const FusionPlan& f,
                                            int L, int64_t tok, int N, int n0, int cnt,
                                            float (&aI)[MAXC], float (&aU)[MAXC],
                                            float (&aT)[MAXC], float (&kl)[MAXC]) {
    const int l_first = f.l_first, l_end = f.l_end;
    auto load_layer = [&](int l, float (&rr)[MAXC], float (&ee)[MAXC]) {
        const int64_t base = L * tok + static_cast<int64_t>(l) * N;
#pragma unroll
        for (int j = 0; j < MAXC; ++j) {
            if (j >= cnt) break;
            const int64_t i = base + n0 + j;
            rr[j] = f.unit_rho ? 1.0f : rho[i];
            ee[j] = pbar_c[i];
        }
    };
    // the first layer's masses (combined onto the carried mass, if any)
    auto start = [&](const float (&r)[MAXC], const float (&e)[MAXC]) {
#pragma unroll
        for (int j = 0; j < MAXC; ++j) {
            if (j >= cnt) break;
            kl[j] = 0.f;
            if (f.carried) {
                const int64_t i = 3 * (tok + n0 + j);
                aI[j] = m_prev[i];
                aU[j] = m_prev[i + 1];
                aT[j] = m_prev[i + 2];
                float mI, mU, mT;
                masses_from_reliability(r[j], e[j], mI, mU, mT);
                kl[j] = ds_step(aI[j], aU[j], aT[j], mI, mU, mT);
            } else {
                masses_from_reliability(r[j], e[j], aI[j], aU[j], aT[j]);
            }
        }
    };
    // one further layer combined (Eq. 13-16)
    auto step = [&](const float (&r)[MAXC], const float (&e)[MAXC]) {
#pragma unroll
        for (int j = 0; j < MAXC; ++j) {
            if (j >= cnt) break;
            float mI, mU, mT;
            masses_from_reliability(r[j], e[j], mI, mU, mT);
            kl[j] = ds_step(aI[j], aU[j], aT[j], mI, mU, mT);
        }
    };
    constexpr int kAhead = MAXC <= 2 ? 8 : 0;
    if (kAhead > 0 && l_end - l_first <= kAhead) {
        float ra[kAhead > 0 ? kAhead : 1][MAXC], ea[kAhead > 0 ? kAhead : 1][MAXC];
#pragma unroll
        for (int t = 0; t < kAhead; ++t)
            if (l_first + t < l_end) load_layer(l_first + t, ra[t], ea[t]);
        start(ra[0], ea[0]);
#pragma unroll
        for (int t = 1; t < kAhead; ++t)
            if (l_first + t < l_end) step(ra[t], ea[t]);
    } else {
        constexpr bool kPrefetch = MAXC <= 4;
        float r[MAXC], e[MAXC];
        load_layer(l_first, r, e);
        start(r, e);
        if (kPrefetch && l_first + 1 < l_end) load_layer(l_first + 1, r, e);
        for (int l = l_first + 1; l < l_end; ++l) {
            float r2[MAXC], e2[MAXC];
            if (!kPrefetch) load_layer(l, r, e);
            else if (l + 1 < l_end) load_layer(l + 1, r2, e2);
            step(r, e);
            if (kPrefetch && l + 1 < l_end) {
#pragma unroll
                for (int j = 0; j < MAXC; ++j) {
                    r[j] = r2[j];
                    e[j] = e2[j];
                }
            }
        }
    }
}

// The fused masses and c of one token into the optional per-token outputs.
__device__ __forceinline__ void write_fused(const SelectArgs& a, int64_t i, float aI, float aU,
                                            float aT, float c) {
    if (a.fused) {
        a.fused[3 * i + 0] = aI;
        a.fused[3 * i + 1] = aU;
        a.fused[3 * i + 2] = aT;
    }
    if (a.prio_c) a.prio_c[i] = c;
}

// Eq. 11-19 for every token of the batch, one token per thread, ahead of the
// selection: pre[token] = (aI, aU, aT, kl), plus the optional per-token outputs.
// Used for images of more than 2048 tokens, where the per-image selection
// workgroup would otherwise do this work for four or more tokens per thread on one
// CU.  The values are those fuse_tokens gives inside the selection kernel.
constexpr int kFuseThreads = 256;
__global__ __launch_bounds__(kFuseThreads) void ds_fuse_kernel(
    const float* __restrict__ rho, const float* __restrict__ pbar_c,
    const float* __restrict__ m_prev, SelectArgs a, BatchGeom bg, f32x4* __restrict__ pre,
    int tiles) {
    const int64_t b = blockIdx.x / tiles;
    const int n = static_cast<int>(blockIdx.x - b * tiles) * kFuseThreads + threadIdx.x;
    const ImageGeom ig = image_geom(bg, b);
    if (n >= ig.N) return;
    const FusionPlan f = fusion_plan(a, m_prev, bg.L);
    float aI[1], aU[1], aT[1], kl[1];
    fuse_tokens<1>(rho, pbar_c, m_prev, f, bg.L, ig.tok, ig.N, n, 1, aI, aU, aT, kl);
    const int64_t i = ig.tok + n;
    f32x4 v = {aI[0], aU[0], aT[0], kl[0]};
    pre[i] = v;
    write_fused(a, i, aI[0], aU[0], aT[0], priority_complement(aU[0], f.protect ? kl[0] : 0.0f));
}

// Dempster fusion across the layers (Eq. 11-19) from per-layer reliability and
// mean support (fuse_tokens), or its results from ds_fuse_kernel when `pre` is
// given, then the selection: the tail of a pruning operation after the per-layer
// evidence.  For an image of more than 16384 tokens the fusion is recomputed (or
// reread) on every visit of a segment (the same arithmetic, so the same values).
template <int MAXC>
__global__ __launch_bounds__(kThreads) void ds_select_kernel(
    const float* __restrict__ rho, const float* __restrict__ pbar_c,
    const float* __restrict__ m_prev, const f32x4* __restrict__ pre, SelectArgs a,
    BatchGeom bg) {
    extern __shared__ uint64_t best[];
    __shared__ SelectShared sh;
    const int64_t b = blockIdx.x;
    const ImageGeom ig = image_geom(bg, b);
    const int L = bg.L, N = ig.N, gh = ig.gh, gw = ig.gw, K = ig.K;
    const int64_t tok = ig.tok;
    const FusionPlan f = fusion_plan(a, m_prev, L);

    float aI[MAXC], aU[MAXC], aT[MAXC];
    float cv[MAXC];
    int posv[MAXC];
    auto load = [&](int n0, int cnt, bool first) {
        float kl[MAXC];
        if (pre) {
#pragma unroll
            for (int j = 0; j < MAXC; ++j) {
                if (j >= cnt) break;
                const f32x4 v = pre[tok + n0 + j];
                aI[j] = v.x;
                aU[j] = v.y;
                aT[j] = v.z;
                kl[j] = v.w;
            }
        } else {
            fuse_tokens<MAXC>(rho, pbar_c, m_prev, f, L, tok, N, n0, cnt, aI, aU, aT, kl);
        }
        token_positions<MAXC>(posv, a.cand_pos, tok, n0, cnt);
#pragma unroll
        for (int j = 0; j < MAXC; ++j) {
            if (j >= cnt) break;
            cv[j] = priority_complement(aU[j], f.protect ? kl[j] : 0.0f);
            if (first && !pre) write_fused(a, tok + n0 + j, aI[j], aU[j], aT[j], cv[j]);
        }
    };
    select_image<MAXC>(cv, posv, load, best, sh, tok, nullptr, nullptr, N, gh, gw, a.cells,
                       a.lambda, K, [&](int slot, int n, int j) {
                           const int64_t o = ig.keep_off + slot;
                           a.keep_idx[o] = n;
                           if (a.keep_pos) a.keep_pos[o] = posv[j];
                           if (a.m_out) {
                               a.m_out[3 * o + 0] = aI[j];
                               a.m_out[3 * o + 1] = aU[j];
                               a.m_out[3 * o + 2] = aT[j];
                           }
                       });
}

// Ablation A1 (attention top-K): the K tokens of largest attention averaged over
// the layers and heads, from the supports e = p - 1/2: with u = N r - 1,
// e = u / (2 (2 + u)), so u = 4e / (1 - 2e) and the ranking by mean r is the
// ranking by sum_{l,h} u.  Layers in order, heads in order within a layer.  No
// spatial term; carried masses (m_out) are written vacuous.
template <int MAXC>
__global__ __launch_bounds__(kThreads) void attention_select_kernel(
    const float* __restrict__ support_c, SelectArgs a, BatchGeom bg) {
    extern __shared__ uint64_t best[];
    __shared__ SelectShared sh;
    const int64_t b = blockIdx.x;
    const ImageGeom ig = image_geom(bg, b);
    const int L = bg.L, H = bg.H, N = ig.N, gh = ig.gh, gw = ig.gw, K = ig.K;
    const int64_t tok = ig.tok;
    float cv[MAXC];
    int posv[MAXC];
    auto load = [&](int n0, int cnt, bool) {
#pragma unroll
        for (int j = 0; j < MAXC; ++j) {
            if (j >= cnt) break;
            const float* eb = support_c + L * H * tok + n0 + j;
            float s = 0.f;
            for (int lh = 0; lh < L * H; lh += 8) {
                float ev[8];
#pragma unroll
                for (int u = 0; u < 8; ++u)
                    ev[u] = lh + u < L * H ? eb[(lh + u) * static_cast<int64_t>(N)] : 0.f;
#pragma unroll
                for (int u = 0; u < 8; ++u)
                    if (lh + u < L * H) s += (4.0f * ev[u]) / (1.0f - 2.0f * ev[u]);
            }
            cv[j] = -s;
        }
        token_positions<MAXC>(posv, a.cand_pos, tok, n0, cnt);
    };
    select_image<MAXC>(cv, posv, load, best, sh, tok, nullptr, nullptr, N, gh, gw, a.cells, 0.0f,
                       K, [&](int slot, int n, int j) {
                           const int64_t o = ig.keep_off + slot;
                           a.keep_idx[o] = n;
                           if (a.keep_pos) a.keep_pos[o] = posv[j];
                           if (a.m_out) {
                               a.m_out[3 * o + 0] = 0.0f;
                               a.m_out[3 * o + 1] = 0.0f;
                               a.m_out[3 * o + 2] = 1.0f;
                           }
                       });
}

// Tokens per thread, rounded up to the kernel variant's register budget.
int chunk_class(const Dims& d) {
    const int64_t chunk = (d.N + kThreads - 1) / kThreads;
    return chunk <= 1 ? 1 : chunk <= 2 ? 2 : chunk <= 4 ? 4 : chunk <= 8 ? 8 : kMaxChunk;
}

// Workgroup size of the selection kernels: one thread per token, in whole waves,
// for images of at most kThreads tokens (fewer waves to synchronise, and each
// wave's scan of the histogram is not repeated by idle waves); kThreads above.
// Every decision is an exact comparison of integer keys, so the kept set does not
// depend on it.
unsigned select_threads(const Dims& d) {
    if (d.N > kThreads) return kThreads;
    return static_cast<unsigned>((d.N + kWave - 1) / kWave * kWave);
}

template <typename Kern>
hipError_t allow_lds(Kern kern, size_t lds) {
    if (lds <= 64 * 1024) return hipSuccess;
    return hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                               hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
}

template <int MAXC>
hipError_t launch_dssel(const Dims& d, const SelectArgs& a, const float* rho, const float* pbar_c,
                        const float* m_prev, f32x4* pre, hipStream_t st) {
    const size_t lds = static_cast<size_t>(a.cells) * a.cells * sizeof(uint64_t);
    auto kern = ds_select_kernel<MAXC>;
    hipError_t err = allow_lds(kern, lds);
    if (err != hipSuccess) return err;
    const BatchGeom bg = batch_geom(d, a.keep);
    if (pre) {
        const int64_t tiles = (d.N + kFuseThreads - 1) / kFuseThreads;
        hipLaunchKernelGGL(ds_fuse_kernel, dim3(static_cast<unsigned>(d.B * tiles)),
                           dim3(kFuseThreads), 0, st, rho, pbar_c, m_prev, a, bg, pre,
                           static_cast<int>(tiles));
        err = hipGetLastError();
        if (err != hipSuccess) return err;
    }
    hipLaunchKernelGGL(kern, dim3(static_cast<unsigned>(d.B)), dim3(select_threads(d)), lds, st, rho, pbar_c,
                       m_prev, static_cast<const f32x4*>(pre), a, bg);
    return hipGetLastError();
}

template <int MAXC>
hipError_t launch_attsel(const Dims& d, const SelectArgs& a, const float* support_c,
                         hipStream_t st) {
    const size_t lds = static_cast<size_t>(a.cells) * a.cells * sizeof(uint64_t);
    auto kern = attention_select_kernel<MAXC>;
    hipError_t err = allow_lds(kern, lds);
    if (err != hipSuccess) return err;
    hipLaunchKernelGGL(kern, dim3(static_cast<unsigned>(d.B)), dim3(select_threads(d)), lds, st, support_c,
                       a, batch_geom(d, a.keep));
    return hipGetLastError();
}

template <int MAXC>
hipError_t launch_sel(const Dims& d, int cells, float lambda, int keep, const float* prio_c,
                      int32_t* keep_idx, double* adj_c, uint8_t* is_rep, hipStream_t st) {
    const size_t lds = static_cast<size_t>(cells) * cells * sizeof(uint64_t);
    auto kern = spatial_select_kernel<MAXC>;
    hipError_t err = allow_lds(kern, lds);
    if (err != hipSuccess) return err;
    hipLaunchKernelGGL(kern, dim3(static_cast<unsigned>(d.B)), dim3(select_threads(d)), lds, st, prio_c,
                       keep_idx, adj_c, is_rep, static_cast<int>(d.N), static_cast<int>(d.gh),
                       static_cast<int>(d.gw), cells, lambda, keep);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_ds_select(const Dims& d, const SelectArgs& a, const float* rho,
                            const float* pbar_c, const float* m_prev, void* fuse_scratch,
                            hipStream_t st) {
    // four or more tokens per thread: the fusion runs device-wide first when the
    // caller lends room for it (d.tokens x 16 bytes)
    const int cc = chunk_class(d);
    f32x4* pre = cc >= 4 ? static_cast<f32x4*>(fuse_scratch) : nullptr;
    switch (cc) {
        case 1: return launch_dssel<1>(d, a, rho, pbar_c, m_prev, nullptr, st);
        case 2: return launch_dssel<2>(d, a, rho, pbar_c, m_prev, nullptr, st);
        case 4: return launch_dssel<4>(d, a, rho, pbar_c, m_prev, pre, st);
        case 8: return launch_dssel<8>(d, a, rho, pbar_c, m_prev, pre, st);
        default: return launch_dssel<kMaxChunk>(d, a, rho, pbar_c, m_prev, pre, st);
    }
}

hipError_t launch_attention_select(const Dims& d, const SelectArgs& a, const float* support_c,
                                   hipStream_t st) {
    switch (chunk_class(d)) {
        case 1: return launch_attsel<1>(d, a, support_c, st);
        case 2: return launch_attsel<2>(d, a, support_c, st);
        case 4: return launch_attsel<4>(d, a, support_c, st);
        case 8: return launch_attsel<8>(d, a, support_c, st);
        default: return launch_attsel<kMaxChunk>(d, a, support_c, st);
    }
}

hipError_t launch_spatial_select(const Dims& d, int cells, float lambda, int keep,
                                 const float* prio_c, int32_t* keep_idx, double* adj_c,
                                 uint8_t* is_rep, hipStream_t st) {
    switch (chunk_class(d)) {
        case 1: return launch_sel<1>(d, cells, lambda, keep, prio_c, keep_idx, adj_c, is_rep, st);
        case 2: return launch_sel<2>(d, cells, lambda, keep, prio_c, keep_idx, adj_c, is_rep, st);
        case 4: return launch_sel<4>(d, cells, lambda, keep, prio_c, keep_idx, adj_c, is_rep, st);
        case 8: return launch_sel<8>(d, cells, lambda, keep, prio_c, keep_idx, adj_c, is_rep, st);
        default:
            return launch_sel<kMaxChunk>(d, cells, lambda, keep, prio_c, keep_idx, adj_c, is_rep, st);
    }
}

}  // namespace e2s
