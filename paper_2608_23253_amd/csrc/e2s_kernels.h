// Kernel launchers used by the C ABI (host side).  Arguments are validated by
// the caller; each launcher only enqueues work on `stream` and reports the
// runtime's launch status.
#pragma once

#include <hip/hip_runtime.h>

#include "e2s_validate.h"

namespace e2s {

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
// Eq. 11-19 from rho, pbar_c, then Eq. 20-23; fused and prio_c may be null.
hipError_t launch_ds_select(const Dims& d, int cells, float lambda, int keep, const float* rho,
                            const float* pbar_c, int32_t* keep_idx, float* fused, float* prio_c,
                            hipStream_t stream);

}  // namespace e2s
