// Kernel launchers used by the C ABI (host side).  Arguments are validated by
// the caller; each launcher only enqueues work on `stream` and reports the
// runtime's launch status.
#pragma once

#include <hip/hip_runtime.h>

#include "batch_geom.h"
#include "e2s_validate.h"

namespace e2s {

// The kernels' view of a validated call's batch (keep: K of a uniform selection).
inline BatchGeom batch_geom(const Dims& d, int keep = 0) {
    BatchGeom g{};
    g.images = d.images;
    g.L = static_cast<int>(d.L);
    g.H = static_cast<int>(d.H);
    g.Hkv = static_cast<int>(d.Hkv);
    g.D = static_cast<int>(d.D);
    g.NT = static_cast<int>(d.NT);
    g.N = static_cast<int>(d.N);
    g.gh = static_cast<int>(d.gh);
    g.gw = static_cast<int>(d.gw);
    g.K = keep;
    g.has_views = d.views != nullptr;
    if (d.views) g.views = *d.views;
    return g;
}

// Score stage, mean-of-logits reading (Eq. 1 then Eq. 8, 9).
hipError_t launch_score_mean_logit(const Dims& d, int dtype, float scale, const void* q,
                                   const void* k, float* support_c, float* r_opt,
                                   hipStream_t stream);

// Score stage, mean-of-probabilities reading (per-query softmax, then the mean).
hipError_t launch_score_mean_prob(const Dims& d, int dtype, float scale, const void* q,
                                  const void* k, float* support_c, float* r_opt,
                                  hipStream_t stream);

// Eq. 10.
hipError_t launch_head_reliability(const Dims& d, const float* support_c, float* rho,
                                   float* pbar_c, hipStream_t stream);
// Eq. 11.
hipError_t launch_head_masses(const Dims& d, const float* rho, const float* pbar_c,
                              float* mass, hipStream_t stream);
// Eq. 12-19 from the layer masses.
hipError_t launch_ds_combine(const Dims& d, const float* mass, float* fused, float* conflict,
                             float* prio_c, hipStream_t stream);
// Eq. 10-19 in one pass over the supports.
hipError_t launch_fuse_evidence(const Dims& d, const float* support_c, float* fused,
                                float* conflict, float* prio_c, hipStream_t stream);
// Eq. 20-23.
hipError_t launch_spatial_select(const Dims& d, int cells, float lambda, int keep,
                                 const float* prio_c, int32_t* keep_idx, double* adj_c,
                                 uint8_t* is_rep, hipStream_t stream);

// Score + reliability of a whole layer per workgroup (mean-of-logits reading, one
// query head per key head), writing rho and pbar_c [B, L, N]; applicable when
// layer_evidence_fits(d).
bool layer_evidence_fits(const Dims& d);
hipError_t launch_layer_evidence(const Dims& d, int dtype, float scale, const void* q,
                                 const void* k, float* rho, float* pbar_c, hipStream_t stream);
// Arguments of the selection tail of a pruning operation.
struct SelectArgs {
    int cells;                 // G
    float lambda;              // Eq. 22 (0 for the no-spatial-novelty variant)
    int keep;                  // K
    int variant;               // e2s_variant
    const int32_t* cand_pos;   // [B, N] raster positions of the candidates, or null (0..N-1)
    int32_t* keep_idx;         // [B, K] kept candidate indices, ascending
    int32_t* keep_pos;         // [B, K] their raster positions, or null
    float* m_out;              // [B, K, 3] their fused masses, or null
    float* fused;              // [B, N, 3] fused masses, or null
    float* prio_c;             // [B, N] c = 1 - q, or null
};
// Eq. 11-19 from rho, pbar_c (onto m_prev [B, N, 3] when given), then Eq. 20-23.
// fuse_scratch: null, or 16-byte aligned device memory of d.tokens x 16 bytes that
// the call may use to run the fusion device-wide before the per-image selection
// (for images of more than 2048 tokens; the results are the same either way).
hipError_t launch_ds_select(const Dims& d, const SelectArgs& a, const float* rho,
                            const float* pbar_c, const float* m_prev, void* fuse_scratch,
                            hipStream_t stream);
// Attention top-K (ablation A1) from the supports [B, L, H, N].
hipError_t launch_attention_select(const Dims& d, const SelectArgs& a, const float* support_c,
                                   hipStream_t stream);

// Streaming read of bytes / 16 packets (e2s_read_probe), arguments validated.
hipError_t launch_read_probe(const void* buf, size_t bytes, int workgroups, uint32_t* sink,
                             hipStream_t stream);

// Token compaction (e2s_compact_tokens), arguments validated.
hipError_t launch_compact(const e2s_compact_shape& s, const int32_t* keep, const void* src,
                          void* dst, hipStream_t stream);

}  // namespace e2s
