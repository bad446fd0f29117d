// Host-side argument checks of the C ABI (see e2s_validate.h).
#include "e2s_validate.h"

#include <cmath>
#include <limits>

namespace e2s {

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

e2s_status check_aligned(const void* ptr, size_t align) {
    return (reinterpret_cast<uintptr_t>(ptr) % align) == 0 ? E2S_OK : E2S_ERR_MISALIGNED;
}

e2s_status check_shape(const e2s_shape* s, Dims* out) {
    if (s == nullptr) return E2S_ERR_NULL_POINTER;
    if (s->batch < 1 || s->num_layers < 1 || s->num_heads < 1 || s->num_kv_heads < 1 ||
        s->head_dim < 1 || s->num_text < 1 || s->grid_h < 1 || s->grid_w < 1)
        return E2S_ERR_BAD_SHAPE;
    if (s->num_heads % s->num_kv_heads != 0) return E2S_ERR_BAD_SHAPE;
    Dims d;
    d.B = s->batch;
    d.L = s->num_layers;
    d.H = s->num_heads;
    d.Hkv = s->num_kv_heads;
    d.D = s->head_dim;
    d.NT = s->num_text;
    d.gh = s->grid_h;
    d.gw = s->grid_w;
    d.N = d.gh * d.gw;
    d.group = d.H / d.Hkv;
    if (d.N > kMaxVisual) return E2S_ERR_UNSUPPORTED;
    if (d.H > kMaxHeads) return E2S_ERR_UNSUPPORTED;
    if (d.D != 64 && d.D != 128) return E2S_ERR_UNSUPPORTED;
    // Every tensor of the call must be indexable with 63-bit element offsets and
    // the grids must stay below 2^31 workgroups.
    const double big = static_cast<double>(std::numeric_limits<int64_t>::max() / 16);
    const double qel = static_cast<double>(d.B) * d.L * d.H * d.NT * d.D;
    const double kel = static_cast<double>(d.B) * d.L * d.Hkv * d.N * d.D;
    const double eel = static_cast<double>(d.B) * d.L * d.H * d.N;
    if (qel > big || kel > big || eel > big) return E2S_ERR_BAD_SHAPE;
    if (static_cast<double>(d.B) * d.L * d.H > 2147483647.0) return E2S_ERR_BAD_SHAPE;
    if (static_cast<double>(d.B) * d.N > 2147483647.0) return E2S_ERR_BAD_SHAPE;
    if (out) *out = d;
    return E2S_OK;
}

e2s_status check_score_params(const e2s_params* p) {
    if (p == nullptr) return E2S_ERR_NULL_POINTER;
    if (p->dtype != E2S_DTYPE_F32 && p->dtype != E2S_DTYPE_BF16) return E2S_ERR_BAD_PARAM;
    if (p->mode != E2S_SCORE_MEAN_LOGIT && p->mode != E2S_SCORE_MEAN_PROB)
        return E2S_ERR_BAD_PARAM;
    if (!std::isfinite(p->scale) || p->scale < 0.0f) return E2S_ERR_BAD_PARAM;
    return E2S_OK;
}

e2s_status check_select_params(const e2s_params* p, const Dims& d) {
    if (p == nullptr) return E2S_ERR_NULL_POINTER;
    if (p->cells < 1 || p->cells > d.gh || p->cells > d.gw) return E2S_ERR_BAD_PARAM;
    if (!std::isfinite(p->lambda) || p->lambda < 0.0f || p->lambda > 1.0f)
        return E2S_ERR_BAD_PARAM;
    if (p->keep < 0 || p->keep > d.N) return E2S_ERR_BAD_PARAM;
    if (p->variant < E2S_VARIANT_FULL || p->variant > E2S_VARIANT_NO_SPATIAL_NOVELTY)
        return E2S_ERR_BAD_PARAM;
    return E2S_OK;
}

size_t support_region_bytes(const Dims& d) {
    return align_up(static_cast<size_t>(d.B * d.L * d.H * d.N) * sizeof(float), 256);
}

size_t layer_region_bytes(const Dims& d) {
    return align_up(static_cast<size_t>(d.B * d.L * d.N) * sizeof(float), 256);
}

size_t prune_workspace_bytes(const Dims& d) {
    return support_region_bytes(d) + 2 * layer_region_bytes(d);
}

}  // namespace e2s
