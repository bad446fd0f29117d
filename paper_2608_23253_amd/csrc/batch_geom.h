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

}  // namespace e2s
