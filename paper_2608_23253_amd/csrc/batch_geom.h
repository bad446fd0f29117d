// Where each image of a batch lives and how large it is, as seen by the kernels.
//
// A uniform batch (e2s_prune and the staged entry points) has every image of one
// shape, its tensors packed image after image:
//   Q [B, L, H, N_T, d], K [B, L, Hkv, N, d], per-token arrays [B, ..., N], keep [B, K].
// A ragged batch (e2s_prune_ragged) reads image b's sizes and offsets from a
// device table of e2s_image records; its per-token arrays hold image b's tokens
// from token_offset on, and every [L, ...] block of a per-token array (supports,
// rho, pbar_c in the workspace) starts at L * token_offset (times H for the
// supports).  Both forms give a kernel the same ImageGeom, so one kernel body
// serves both; for a uniform batch the offsets are the packed ones.
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>

#include "e2s.h"

namespace e2s {

struct BatchGeom {
    const e2s_image* images;   // device table (ragged), or null (uniform)
    int L, H, Hkv, D;          // shared by every image
    int NT, N, gh, gw, K;      // the uniform batch's per-image sizes
    bool has_views;            // Q and K given as per-layer views (uniform batch)
    e2s_qk_views views;
};

struct ImageGeom {
    int64_t q_off;             // elements from q to the image's Q block [L, H, N_T, d]
    int64_t k_off;             // elements from k to its K block [L, Hkv, N, d]
    int64_t tok;               // its first token in per-token arrays
    int64_t keep_off;          // its first entry in keep_idx
    int NT, N, gh, gw, K;
};

__device__ __forceinline__ ImageGeom image_geom(const BatchGeom& g, int64_t b) {
    ImageGeom r;
    if (g.images != nullptr) {
        // the table is read-only for the whole launch and b is uniform over the
        // workgroup: read it through the constant address space (scalar loads,
        // which do not occupy the vector memory counter the kernels wait on)
        typedef const __attribute__((address_space(4))) e2s_image ConstImage;
        ConstImage* im = (ConstImage*)g.images + b;
        r.q_off = im->q_offset;
        r.k_off = im->k_offset;
        r.tok = im->token_offset;
        r.keep_off = im->keep_offset;
        r.NT = im->num_text;
        r.gh = im->grid_h;
        r.gw = im->grid_w;
        r.N = r.gh * r.gw;
        r.K = im->keep;
    } else {
        r.NT = g.NT;
        r.N = g.N;
        r.gh = g.gh;
        r.gw = g.gw;
        r.K = g.K;
        r.q_off = b * g.L * g.H * static_cast<int64_t>(g.NT) * g.D;
        r.k_off = b * g.L * g.Hkv * static_cast<int64_t>(g.N) * g.D;
        r.tok = b * g.N;
        r.keep_off = b * g.K;
    }
    return r;
}

// First element of the rows [N_T, d] of query head h (image b, layer l), and the
// element stride between consecutive rows: packed blocks, or the caller's views.
template <typename T>
__device__ __forceinline__ const T* query_rows(const T* q, const BatchGeom& g, const ImageGeom& ig,
                                               int64_t b, int l, int h) {
    if (g.has_views)
        return static_cast<const T*>(g.views.q[l]) + b * g.views.q_stride_image +
               h * g.views.q_stride_head;
    return q + ig.q_off + (static_cast<int64_t>(l) * g.H + h) * ig.NT * g.D;
}
__device__ __forceinline__ int64_t query_ld(const BatchGeom& g) {
    return g.has_views ? g.views.q_stride_text : g.D;
}
// The same for the rows [N, d] of key head kv.
template <typename T>
__device__ __forceinline__ const T* key_rows(const T* k, const BatchGeom& g, const ImageGeom& ig,
                                             int64_t b, int l, int kv) {
    if (g.has_views)
        return static_cast<const T*>(g.views.k[l]) + b * g.views.k_stride_image +
               kv * g.views.k_stride_head;
    return k + ig.k_off + (static_cast<int64_t>(l) * g.Hkv + kv) * ig.N * g.D;
}
__device__ __forceinline__ int64_t key_ld(const BatchGeom& g) {
    return g.has_views ? g.views.k_stride_token : g.D;
}

}  // namespace e2s
