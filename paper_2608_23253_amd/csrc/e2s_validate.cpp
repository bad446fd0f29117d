// Host-side argument checks of the C ABI (see e2s_validate.h).
#include "e2s_validate.h"

#include <algorithm>
#include <cmath>
#include <limits>
#include <vector>

namespace e2s {

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

e2s_status check_aligned(const void* ptr, size_t align) {
    return (reinterpret_cast<uintptr_t>(ptr) % align) == 0 ? E2S_OK : E2S_ERR_MISALIGNED;
}

// A grid may hold fewer than 2^32 work-items.  The kernels launch at most 1024
// threads per (image, layer, head) unit and 256 per (image, layer, 64-token tile);
// blh and bl_tiles count those units.
static bool grids_fit(double blh, double bl_tiles) {
    return blh * 1024.0 < 4294967296.0 && bl_tiles * 256.0 < 4294967296.0;
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
    // Every tensor of the call must be indexable with 63-bit element offsets.
    const double big = static_cast<double>(std::numeric_limits<int64_t>::max() / 16);
    const double qel = static_cast<double>(d.B) * d.L * d.H * d.NT * d.D;
    const double kel = static_cast<double>(d.B) * d.L * d.Hkv * d.N * d.D;
    const double eel = static_cast<double>(d.B) * d.L * d.H * d.N;
    if (qel > big || kel > big || eel > big) return E2S_ERR_BAD_SHAPE;
    if (!grids_fit(static_cast<double>(d.B) * d.L * d.H,
                   static_cast<double>(d.B) * d.L * ((d.N + 63) / 64)))
        return E2S_ERR_UNSUPPORTED;
    d.tokens = d.B * d.N;
    if (out) *out = d;
    return E2S_OK;
}

e2s_status check_views(const e2s_qk_views* v, const Dims& d, int elem_bytes) {
    if (v == nullptr) return E2S_ERR_NULL_POINTER;
    if (d.L > E2S_MAX_VIEW_LAYERS) return E2S_ERR_UNSUPPORTED;
    for (int64_t l = 0; l < d.L; ++l) {
        if (v->q[l] == nullptr || v->k[l] == nullptr) return E2S_ERR_NULL_POINTER;
        if (check_aligned(v->q[l], 16) != E2S_OK || check_aligned(v->k[l], 16) != E2S_OK)
            return E2S_ERR_MISALIGNED;
    }
    const int64_t strides[6] = {v->q_stride_image, v->q_stride_head, v->q_stride_text,
                                v->k_stride_image, v->k_stride_head, v->k_stride_token};
    for (int64_t st : strides) {
        if (st < 0) return E2S_ERR_BAD_SHAPE;
        if (st > std::numeric_limits<int64_t>::max() / 64) return E2S_ERR_BAD_SHAPE;
        if ((st * elem_bytes) % 16 != 0) return E2S_ERR_MISALIGNED;
    }
    // element offsets of the last row of each view stay in 63-bit range
    const double big = static_cast<double>(std::numeric_limits<int64_t>::max() / 16);
    const double qend = static_cast<double>(d.B) * v->q_stride_image +
                        static_cast<double>(d.H) * v->q_stride_head +
                        static_cast<double>(d.NT) * v->q_stride_text;
    const double kend = static_cast<double>(d.B) * v->k_stride_image +
                        static_cast<double>(d.Hkv) * v->k_stride_head +
                        static_cast<double>(d.N) * v->k_stride_token;
    if (qend > big || kend > big) return E2S_ERR_BAD_SHAPE;
    return E2S_OK;
}

namespace {
// Ranges [start, start + len) of the records with len > 0 must not overlap.
bool disjoint(std::vector<std::pair<int64_t, int64_t>> r) {
    std::sort(r.begin(), r.end());
    for (size_t i = 1; i < r.size(); ++i)
        if (r[i].first < r[i - 1].first + r[i - 1].second) return false;
    return true;
}
}  // namespace

e2s_status check_ragged(const e2s_ragged_shape* s, const e2s_image* images, int elem_bytes,
                        Dims* out, int64_t* min_side) {
    if (s == nullptr || images == nullptr) return E2S_ERR_NULL_POINTER;
    if (s->batch < 1 || s->num_layers < 1 || s->num_heads < 1 || s->num_kv_heads < 1 ||
        s->head_dim < 1)
        return E2S_ERR_BAD_SHAPE;
    if (s->num_heads % s->num_kv_heads != 0) return E2S_ERR_BAD_SHAPE;
    Dims d;
    d.B = s->batch;
    d.L = s->num_layers;
    d.H = s->num_heads;
    d.Hkv = s->num_kv_heads;
    d.D = s->head_dim;
    d.group = d.H / d.Hkv;
    d.gh = 0;
    d.gw = 0;
    if (d.H > kMaxHeads) return E2S_ERR_UNSUPPORTED;
    if (d.D != 64 && d.D != 128) return E2S_ERR_UNSUPPORTED;
    const double big = static_cast<double>(std::numeric_limits<int64_t>::max() / 16);
    const int64_t align_el = elem_bytes > 0 ? 16 / elem_bytes : 1;
    int64_t nt_max = 0, n_max = 0, span = 0, side = std::numeric_limits<int64_t>::max();
    std::vector<std::pair<int64_t, int64_t>> toks, keeps;
    toks.reserve(static_cast<size_t>(d.B));
    for (int64_t b = 0; b < d.B; ++b) {
        const e2s_image& im = images[b];
        if (im.grid_h < 1 || im.grid_w < 1 || im.num_text < 1) return E2S_ERR_BAD_SHAPE;
        const int64_t n = static_cast<int64_t>(im.grid_h) * im.grid_w;
        if (n > kMaxVisual) return E2S_ERR_UNSUPPORTED;
        if (im.keep < 0 || im.keep > n) return E2S_ERR_BAD_PARAM;
        if (im.q_offset < 0 || im.k_offset < 0 || im.token_offset < 0 || im.keep_offset < 0)
            return E2S_ERR_BAD_SHAPE;
        if (im.q_offset % align_el != 0 || im.k_offset % align_el != 0) return E2S_ERR_MISALIGNED;
        const double qel = static_cast<double>(im.q_offset) +
                           static_cast<double>(d.L) * d.H * im.num_text * d.D;
        const double kel = static_cast<double>(im.k_offset) + static_cast<double>(d.L) * d.Hkv * n * d.D;
        const double tel = (static_cast<double>(im.token_offset) + n) * d.L * d.H;
        const double kp = static_cast<double>(im.keep_offset) + im.keep;
        if (qel > big || kel > big || tel > big || kp > 2147483647.0) return E2S_ERR_BAD_SHAPE;
        nt_max = std::max<int64_t>(nt_max, im.num_text);
        n_max = std::max(n_max, n);
        span = std::max(span, im.token_offset + n);
        side = std::min<int64_t>(side, std::min(im.grid_h, im.grid_w));
        toks.emplace_back(im.token_offset, n);
        if (im.keep > 0) keeps.emplace_back(im.keep_offset, im.keep);
    }
    if (!disjoint(toks) || !disjoint(keeps)) return E2S_ERR_BAD_SHAPE;
    if (!grids_fit(static_cast<double>(d.B) * d.L * d.H,
                   static_cast<double>(d.B) * d.L * ((n_max + 63) / 64)))
        return E2S_ERR_UNSUPPORTED;
    d.NT = nt_max;
    d.N = n_max;
    d.tokens = span;
    if (out) *out = d;
    if (min_side) *min_side = side;
    return E2S_OK;
}

e2s_status check_score_params(const e2s_params* p) {
    if (p == nullptr) return E2S_ERR_NULL_POINTER;
    if (p->dtype != E2S_DTYPE_F32 && p->dtype != E2S_DTYPE_BF16 && p->dtype != E2S_DTYPE_F16)
        return E2S_ERR_BAD_PARAM;
    if (p->mode != E2S_SCORE_MEAN_LOGIT && p->mode != E2S_SCORE_MEAN_PROB)
        return E2S_ERR_BAD_PARAM;
    if (!std::isfinite(p->scale) || p->scale < 0.0f) return E2S_ERR_BAD_PARAM;
    return E2S_OK;
}

e2s_status check_select_params(const e2s_params* p, const Dims& d) {
    if (p == nullptr) return E2S_ERR_NULL_POINTER;
    if (p->cells < 1 || p->cells > d.gh || p->cells > d.gw) return E2S_ERR_BAD_PARAM;
    if (p->cells > kMaxCells) return E2S_ERR_UNSUPPORTED;
    if (!std::isfinite(p->lambda) || p->lambda < 0.0f || p->lambda > 1.0f)
        return E2S_ERR_BAD_PARAM;
    if (p->keep < 0 || p->keep > d.N) return E2S_ERR_BAD_PARAM;
    if (p->variant < E2S_VARIANT_FULL || p->variant > E2S_VARIANT_NO_SPATIAL_NOVELTY)
        return E2S_ERR_BAD_PARAM;
    return E2S_OK;
}

e2s_status check_compact(const e2s_compact_shape* s) {
    if (s == nullptr) return E2S_ERR_NULL_POINTER;
    if (s->batch < 1 || s->rows < 1 || s->num_tokens < 1 || s->keep < 0 || s->channels < 1)
        return E2S_ERR_BAD_SHAPE;
    if (s->elem_bytes != 2 && s->elem_bytes != 4) return E2S_ERR_BAD_PARAM;
    if ((static_cast<int64_t>(s->channels) * s->elem_bytes) % 16 != 0) return E2S_ERR_MISALIGNED;
    const double big = static_cast<double>(std::numeric_limits<int64_t>::max() / 16);
    const double counts[3] = {static_cast<double>(s->batch), static_cast<double>(s->rows),
                              static_cast<double>(s->num_tokens)};
    const double dcounts[3] = {static_cast<double>(s->batch), static_cast<double>(s->rows),
                               static_cast<double>(s->keep)};
    double src_end = s->channels, dst_end = s->channels;
    for (int i = 0; i < 3; ++i) {
        if (s->src_stride[i] < 0 || s->dst_stride[i] < 0) return E2S_ERR_BAD_SHAPE;
        // (the products below stay in range: elem_bytes <= 4)
        if (s->src_stride[i] > std::numeric_limits<int64_t>::max() / 16 ||
            s->dst_stride[i] > std::numeric_limits<int64_t>::max() / 16)
            return E2S_ERR_BAD_SHAPE;
        if ((s->src_stride[i] * s->elem_bytes) % 16 != 0 ||
            (s->dst_stride[i] * s->elem_bytes) % 16 != 0)
            return E2S_ERR_MISALIGNED;
        src_end += (counts[i] - 1) * static_cast<double>(s->src_stride[i]);
        dst_end += (dcounts[i] - 1) * static_cast<double>(s->dst_stride[i]);
    }
    if (src_end * s->elem_bytes > big || dst_end * s->elem_bytes > big) return E2S_ERR_BAD_SHAPE;
    return E2S_OK;
}

size_t support_region_bytes(const Dims& d) {
    return align_up(static_cast<size_t>(d.L * d.H * d.tokens) * sizeof(float), 256);
}

size_t layer_region_bytes(const Dims& d) {
    return align_up(static_cast<size_t>(d.L * d.tokens) * sizeof(float), 256);
}

size_t prune_workspace_bytes(const Dims& d) {
    return support_region_bytes(d) + 2 * layer_region_bytes(d);
}

}  // namespace e2s
