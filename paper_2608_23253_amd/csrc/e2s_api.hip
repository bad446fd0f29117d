// extern "C" entry points of libe2s.so (declared and documented in include/e2s.h).
// Each call validates every argument on the host before it touches the HIP
// runtime, then enqueues its kernels on the caller's stream.
#include <atomic>
#include <cmath>
#include <mutex>

#include "e2s.h"
#include "e2s_kernels.h"
#include "e2s_validate.h"

// Workspace of e2s_prune_noalloc (callers that cannot allocate).  In host code
// `scratch` names a host-side stand-in, not device memory: kernels and copies get
// the device address that scratch_address() looks up once per device.
static __device__ __align__(256) unsigned char scratch[E2S_NOALLOC_SCRATCH_BYTES];

namespace {

using e2s::Dims;

e2s_status from_hip(hipError_t err) {
    if (err == hipSuccess) return E2S_OK;
    if (err == hipErrorNotSupported) return E2S_ERR_UNSUPPORTED;
    return E2S_ERR_LAUNCH;
}

#define E2S_TRY(expr)                          \
    do {                                       \
        const e2s_status st_ = (expr);         \
        if (st_ != E2S_OK) return st_;         \
    } while (0)

e2s_status need(const void* p) { return p ? E2S_OK : E2S_ERR_NULL_POINTER; }
e2s_status aligned_opt(const void* p, size_t a) { return p ? e2s::check_aligned(p, a) : E2S_OK; }

float effective_scale(const e2s_params* p, const Dims& d) {
    if (p->scale != 0.0f) return p->scale;
    return static_cast<float>(1.0 / std::sqrt(static_cast<double>(d.D)));
}

e2s_status check_score_call(const e2s_shape* shape, const e2s_params* params, const void* q,
                            const void* k, const float* support_c, const float* r_opt,
                            Dims* d) {
    E2S_TRY(e2s::check_shape(shape, d));
    E2S_TRY(e2s::check_score_params(params));
    E2S_TRY(need(q));
    E2S_TRY(need(k));
    E2S_TRY(need(support_c));
    E2S_TRY(e2s::check_aligned(q, 16));
    E2S_TRY(e2s::check_aligned(k, 16));
    E2S_TRY(e2s::check_aligned(support_c, 4));
    E2S_TRY(aligned_opt(r_opt, 4));
    return E2S_OK;
}

e2s_status run_score(const Dims& d, const e2s_params* params, const void* q, const void* k,
                     float* support_c, float* r_opt, hipStream_t st) {
    const float scale = effective_scale(params, d);
    if (params->mode == E2S_SCORE_MEAN_LOGIT)
        return from_hip(e2s::launch_score_mean_logit(d, params->dtype, scale, q, k, support_c,
                                                     r_opt, st));
    return from_hip(
        e2s::launch_score_mean_prob(d, params->dtype, scale, q, k, support_c, r_opt, st));
}

// Compute units of the current device (cached per device).
int device_cus() {
    // calls may come from several host threads; every writer stores the same value
    static std::atomic<int> cached[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
    int n = cached[dev].load(std::memory_order_relaxed);
    if (n == 0) {
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
            return 0;
        cached[dev].store(n, std::memory_order_relaxed);
    }
    return n;
}

// Eq. 1, 8-10: per-layer rho and pbar_c, on chip when a layer fits and there are
// enough layers to occupy the device with one workgroup each, else through the
// supports in `workspace` (both give the same bits).
e2s_status run_layer_reliability(const Dims& d, const e2s_params* params, const void* q,
                                 const void* k, void* workspace, float* rho, float* pbar_c,
                                 hipStream_t st) {
    if (params->mode == E2S_SCORE_MEAN_LOGIT && e2s::layer_evidence_fits(d) &&
        d.B * d.L >= device_cus())
        return from_hip(e2s::launch_layer_evidence(d, params->dtype, effective_scale(params, d), q,
                                                   k, rho, pbar_c, st));
    float* support_c = static_cast<float*>(workspace);
    E2S_TRY(run_score(d, params, q, k, support_c, nullptr, st));
    return from_hip(e2s::launch_head_reliability(d, support_c, rho, pbar_c, st));
}

e2s::SelectArgs select_args(const e2s_params* p, int32_t* keep_idx, float* fused,
                            float* prio_c) {
    e2s::SelectArgs a{};
    a.cells = p->cells;
    a.lambda = p->variant == E2S_VARIANT_NO_SPATIAL_NOVELTY ? 0.0f : p->lambda;
    a.keep = p->keep;
    a.variant = p->variant;
    a.keep_idx = keep_idx;
    a.fused = fused;
    a.prio_c = prio_c;
    return a;
}

// A pruning operation after validation: the evidence (or, for attention top-K, the
// supports) of the operation's layers, then the selection tail.  d.N is the
// candidate count.
e2s_status run_operation(const Dims& d, const e2s_params* params, const void* q, const void* k,
                         void* workspace, const e2s::SelectArgs& a, const float* m_prev,
                         hipStream_t st) {
    char* ws = static_cast<char*>(workspace);
    if (params->variant == E2S_VARIANT_ATTENTION_TOPK) {
        float* support_c = reinterpret_cast<float*>(ws);
        E2S_TRY(run_score(d, params, q, k, support_c, nullptr, st));
        return from_hip(e2s::launch_attention_select(d, a, support_c, st));
    }
    float* rho = reinterpret_cast<float*>(ws + e2s::support_region_bytes(d));
    float* pbar_c =
        reinterpret_cast<float*>(ws + e2s::support_region_bytes(d) + e2s::layer_region_bytes(d));
    E2S_TRY(run_layer_reliability(d, params, q, k, workspace, rho, pbar_c, st));
    // the supports region is free again (the reliability stage has read it) and
    // lends the selection room for its device-wide fusion when it is large enough
    const bool room = e2s::support_region_bytes(d) >= static_cast<size_t>(d.tokens) * 16;
    return from_hip(e2s::launch_ds_select(d, a, rho, pbar_c, m_prev, room ? ws : nullptr, st));
}

e2s_status check_score_inputs(const e2s_shape* shape, const e2s_params* params, const void* q,
                              const void* k, void* workspace, size_t workspace_bytes, Dims* d) {
    E2S_TRY(e2s::check_shape(shape, d));
    E2S_TRY(e2s::check_score_params(params));
    E2S_TRY(need(q));
    E2S_TRY(need(k));
    E2S_TRY(need(workspace));
    E2S_TRY(e2s::check_aligned(q, 16));
    E2S_TRY(e2s::check_aligned(k, 16));
    E2S_TRY(e2s::check_aligned(workspace, 256));
    if (workspace_bytes < e2s::prune_workspace_bytes(*d)) return E2S_ERR_WORKSPACE_TOO_SMALL;
    return E2S_OK;
}

constexpr int kMaxDevices = 64;

// The current device's address of `scratch`: looked up with that device current on
// the first call, then reused (each device holds its own copy of the array).
e2s_status scratch_address(void** out) {
    static std::mutex mu;
    static void* addr[kMaxDevices] = {};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices)
        return E2S_ERR_SCRATCH_TOO_SMALL;
    std::lock_guard<std::mutex> lock(mu);
    if (addr[dev] == nullptr) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr)
            return E2S_ERR_SCRATCH_TOO_SMALL;
        addr[dev] = p;
    }
    *out = addr[dev];
    return E2S_OK;
}

}  // namespace

extern "C" {

int32_t e2s_abi_version(void) { return E2S_ABI_VERSION; }

e2s_status e2s_read_probe(const void* buf, size_t bytes, int32_t workgroups, uint32_t* sink,
                          void* stream) {
    E2S_TRY(need(buf));
    E2S_TRY(need(sink));
    E2S_TRY(e2s::check_aligned(buf, 16));
    E2S_TRY(e2s::check_aligned(sink, 4));
    if (bytes == 0 || bytes % 16 != 0) return E2S_ERR_BAD_SHAPE;
    if (workgroups < 1 || workgroups > 65535) return E2S_ERR_BAD_PARAM;
    return from_hip(e2s::launch_read_probe(buf, bytes, workgroups, sink,
                                           static_cast<hipStream_t>(stream)));
}

const char* e2s_status_string(e2s_status status) {
    switch (status) {
        case E2S_OK: return "E2S_OK";
        case E2S_ERR_NULL_POINTER: return "E2S_ERR_NULL_POINTER: a required pointer is NULL";
        case E2S_ERR_BAD_SHAPE: return "E2S_ERR_BAD_SHAPE: a count is out of range or inconsistent";
        case E2S_ERR_BAD_PARAM: return "E2S_ERR_BAD_PARAM: dtype, mode, scale, cells, lambda or keep";
        case E2S_ERR_UNSUPPORTED: return "E2S_ERR_UNSUPPORTED: valid but not implemented by this library";
        case E2S_ERR_MISALIGNED: return "E2S_ERR_MISALIGNED: a pointer violates the alignment rule";
        case E2S_ERR_WORKSPACE_TOO_SMALL: return "E2S_ERR_WORKSPACE_TOO_SMALL: workspace below e2s_prune_workspace_size";
        case E2S_ERR_LAUNCH: return "E2S_ERR_LAUNCH: the HIP runtime refused a kernel launch";
        case E2S_ERR_SCRATCH_TOO_SMALL: return "E2S_ERR_SCRATCH_TOO_SMALL: the call needs more than the library's static scratch (E2S_NOALLOC_SCRATCH_BYTES), or its device address was unavailable";
    }
    return "unknown e2s_status";
}

e2s_status e2s_score_heads(const e2s_shape* shape, const e2s_params* params, const void* q,
                           const void* k, float* support_c, float* r_opt, void* stream) {
    Dims d;
    E2S_TRY(check_score_call(shape, params, q, k, support_c, r_opt, &d));
    return run_score(d, params, q, k, support_c, r_opt, static_cast<hipStream_t>(stream));
}

e2s_status e2s_head_reliability(const e2s_shape* shape, const float* support_c, float* rho,
                                float* pbar_c, void* stream) {
    Dims d;
    E2S_TRY(e2s::check_shape(shape, &d));
    E2S_TRY(need(support_c));
    E2S_TRY(need(rho));
    E2S_TRY(need(pbar_c));
    E2S_TRY(e2s::check_aligned(support_c, 4));
    E2S_TRY(e2s::check_aligned(rho, 4));
    E2S_TRY(e2s::check_aligned(pbar_c, 4));
    return from_hip(e2s::launch_head_reliability(d, support_c, rho, pbar_c,
                                                 static_cast<hipStream_t>(stream)));
}

e2s_status e2s_head_masses(const e2s_shape* shape, const float* rho, const float* pbar_c,
                           float* mass, void* stream) {
    Dims d;
    E2S_TRY(e2s::check_shape(shape, &d));
    E2S_TRY(need(rho));
    E2S_TRY(need(pbar_c));
    E2S_TRY(need(mass));
    E2S_TRY(e2s::check_aligned(rho, 4));
    E2S_TRY(e2s::check_aligned(pbar_c, 4));
    E2S_TRY(e2s::check_aligned(mass, 4));
    return from_hip(e2s::launch_head_masses(d, rho, pbar_c, mass, static_cast<hipStream_t>(stream)));
}

e2s_status e2s_ds_combine_layers(const e2s_shape* shape, const float* mass, float* fused,
                                 float* conflict, float* prio_c, void* stream) {
    Dims d;
    E2S_TRY(e2s::check_shape(shape, &d));
    E2S_TRY(need(mass));
    E2S_TRY(need(prio_c));
    E2S_TRY(e2s::check_aligned(mass, 4));
    E2S_TRY(e2s::check_aligned(prio_c, 4));
    E2S_TRY(aligned_opt(fused, 4));
    E2S_TRY(aligned_opt(conflict, 4));
    return from_hip(e2s::launch_ds_combine(d, mass, fused, conflict, prio_c,
                                           static_cast<hipStream_t>(stream)));
}

e2s_status e2s_fuse_evidence(const e2s_shape* shape, const float* support_c, float* fused,
                             float* conflict, float* prio_c, void* stream) {
    Dims d;
    E2S_TRY(e2s::check_shape(shape, &d));
    E2S_TRY(need(support_c));
    E2S_TRY(need(prio_c));
    E2S_TRY(e2s::check_aligned(support_c, 4));
    E2S_TRY(e2s::check_aligned(prio_c, 4));
    E2S_TRY(aligned_opt(fused, 4));
    E2S_TRY(aligned_opt(conflict, 4));
    return from_hip(e2s::launch_fuse_evidence(d, support_c, fused, conflict, prio_c,
                                              static_cast<hipStream_t>(stream)));
}

e2s_status e2s_spatial_select(const e2s_shape* shape, const e2s_params* params,
                              const float* prio_c, int32_t* keep_idx, double* adj_c_opt,
                              uint8_t* is_rep_opt, void* stream) {
    Dims d;
    E2S_TRY(e2s::check_shape(shape, &d));
    E2S_TRY(e2s::check_select_params(params, d));
    E2S_TRY(need(prio_c));
    if (params->keep > 0) E2S_TRY(need(keep_idx));
    E2S_TRY(e2s::check_aligned(prio_c, 4));
    E2S_TRY(aligned_opt(keep_idx, 4));
    E2S_TRY(aligned_opt(adj_c_opt, 8));
    return from_hip(e2s::launch_spatial_select(d, params->cells, params->lambda, params->keep,
                                               prio_c, keep_idx, adj_c_opt, is_rep_opt,
                                               static_cast<hipStream_t>(stream)));
}

e2s_status e2s_prune_workspace_size(const e2s_shape* shape, const e2s_params* params,
                                    size_t* bytes) {
    Dims d;
    E2S_TRY(e2s::check_shape(shape, &d));
    E2S_TRY(need(params));
    E2S_TRY(need(bytes));
    *bytes = e2s::prune_workspace_bytes(d);
    return E2S_OK;
}

e2s_status e2s_layer_reliability(const e2s_shape* shape, const e2s_params* params,
                                 const void* q, const void* k, void* workspace,
                                 size_t workspace_bytes, float* rho, float* pbar_c,
                                 void* stream) {
    Dims d;
    E2S_TRY(check_score_inputs(shape, params, q, k, workspace, workspace_bytes, &d));
    E2S_TRY(need(rho));
    E2S_TRY(need(pbar_c));
    E2S_TRY(e2s::check_aligned(rho, 4));
    E2S_TRY(e2s::check_aligned(pbar_c, 4));
    return run_layer_reliability(d, params, q, k, workspace, rho, pbar_c,
                                 static_cast<hipStream_t>(stream));
}

e2s_status e2s_fuse_select(const e2s_shape* shape, const e2s_params* params, const float* rho,
                           const float* pbar_c, int32_t* keep_idx, float* fused_opt,
                           float* prio_c_opt, void* stream) {
    Dims d;
    E2S_TRY(e2s::check_shape(shape, &d));
    E2S_TRY(e2s::check_select_params(params, d));
    E2S_TRY(need(rho));
    E2S_TRY(need(pbar_c));
    if (params->keep > 0) E2S_TRY(need(keep_idx));
    E2S_TRY(e2s::check_aligned(rho, 4));
    E2S_TRY(e2s::check_aligned(pbar_c, 4));
    E2S_TRY(aligned_opt(keep_idx, 4));
    E2S_TRY(aligned_opt(fused_opt, 4));
    E2S_TRY(aligned_opt(prio_c_opt, 4));
    if (params->variant == E2S_VARIANT_ATTENTION_TOPK) return E2S_ERR_UNSUPPORTED;
    return from_hip(e2s::launch_ds_select(d, select_args(params, keep_idx, fused_opt, prio_c_opt),
                                          rho, pbar_c, nullptr, nullptr,
                                          static_cast<hipStream_t>(stream)));
}

e2s_status e2s_prune(const e2s_shape* shape, const e2s_params* params, const void* q,
                     const void* k, void* workspace, size_t workspace_bytes, int32_t* keep_idx,
                     float* fused_opt, float* prio_c_opt, void* stream) {
    Dims d;
    E2S_TRY(check_score_inputs(shape, params, q, k, workspace, workspace_bytes, &d));
    E2S_TRY(e2s::check_select_params(params, d));
    if (params->keep > 0) E2S_TRY(need(keep_idx));
    E2S_TRY(aligned_opt(keep_idx, 4));
    E2S_TRY(aligned_opt(fused_opt, 4));
    E2S_TRY(aligned_opt(prio_c_opt, 4));

    return run_operation(d, params, q, k, workspace,
                         select_args(params, keep_idx, fused_opt, prio_c_opt), nullptr,
                         static_cast<hipStream_t>(stream));
}

e2s_status e2s_prune_noalloc(const e2s_shape* shape, const e2s_params* params, const void* q,
                             const void* k, int32_t* keep_idx, float* fused_opt,
                             float* prio_c_opt, void* stream) {
    Dims d;
    E2S_TRY(e2s::check_shape(shape, &d));
    E2S_TRY(e2s::check_score_params(params));
    E2S_TRY(need(q));
    E2S_TRY(need(k));
    E2S_TRY(e2s::check_aligned(q, 16));
    E2S_TRY(e2s::check_aligned(k, 16));
    E2S_TRY(e2s::check_select_params(params, d));
    if (params->keep > 0) E2S_TRY(need(keep_idx));
    E2S_TRY(aligned_opt(keep_idx, 4));
    E2S_TRY(aligned_opt(fused_opt, 4));
    E2S_TRY(aligned_opt(prio_c_opt, 4));
    if (e2s::prune_workspace_bytes(d) > E2S_NOALLOC_SCRATCH_BYTES) return E2S_ERR_SCRATCH_TOO_SMALL;
    void* ws = nullptr;
    E2S_TRY(scratch_address(&ws));
    return run_operation(d, params, q, k, ws,
                         select_args(params, keep_idx, fused_opt, prio_c_opt), nullptr,
                         static_cast<hipStream_t>(stream));
}

e2s_status e2s_prune_views(const e2s_shape* shape, const e2s_params* params,
                           const e2s_qk_views* views, void* workspace, size_t workspace_bytes,
                           int32_t* keep_idx, float* fused_opt, float* prio_c_opt, void* stream) {
    Dims d;
    E2S_TRY(e2s::check_shape(shape, &d));
    E2S_TRY(e2s::check_score_params(params));
    E2S_TRY(e2s::check_views(views, d, params->dtype == E2S_DTYPE_F32 ? 4 : 2));
    E2S_TRY(need(workspace));
    E2S_TRY(e2s::check_aligned(workspace, 256));
    if (workspace_bytes < e2s::prune_workspace_bytes(d)) return E2S_ERR_WORKSPACE_TOO_SMALL;
    E2S_TRY(e2s::check_select_params(params, d));
    if (params->keep > 0) E2S_TRY(need(keep_idx));
    E2S_TRY(aligned_opt(keep_idx, 4));
    E2S_TRY(aligned_opt(fused_opt, 4));
    E2S_TRY(aligned_opt(prio_c_opt, 4));
    d.views = views;
    // the kernels read Q and K through the views; the packed pointers are unused
    return run_operation(d, params, nullptr, nullptr, workspace,
                         select_args(params, keep_idx, fused_opt, prio_c_opt), nullptr,
                         static_cast<hipStream_t>(stream));
}

e2s_status e2s_prune_stage(const e2s_shape* shape, const e2s_params* params, int32_t num_cand,
                           const void* q, const void* k, const int32_t* cand_pos_opt,
                           const float* m_prev_opt, void* workspace, size_t workspace_bytes,
                           int32_t* keep_idx, int32_t* keep_pos_opt, float* m_out_opt,
                           void* stream) {
    Dims d;
    // the workspace of the full grid bounds that of any candidate subset
    E2S_TRY(check_score_inputs(shape, params, q, k, workspace, workspace_bytes, &d));
    if (num_cand < 1 || num_cand > d.N) return E2S_ERR_BAD_SHAPE;
    if (cand_pos_opt == nullptr && num_cand != d.N) return E2S_ERR_BAD_SHAPE;
    d.N = num_cand;
    d.tokens = d.B * d.N;
    E2S_TRY(e2s::check_select_params(params, d));
    if (params->keep > 0) E2S_TRY(need(keep_idx));
    E2S_TRY(aligned_opt(cand_pos_opt, 4));
    E2S_TRY(aligned_opt(m_prev_opt, 4));
    E2S_TRY(aligned_opt(keep_idx, 4));
    E2S_TRY(aligned_opt(keep_pos_opt, 4));
    E2S_TRY(aligned_opt(m_out_opt, 4));
    e2s::SelectArgs a = select_args(params, keep_idx, nullptr, nullptr);
    a.cand_pos = cand_pos_opt;
    a.keep_pos = keep_pos_opt;
    a.m_out = m_out_opt;
    return run_operation(d, params, q, k, workspace, a, m_prev_opt,
                         static_cast<hipStream_t>(stream));
}

e2s_status e2s_prune_ragged_workspace_size(const e2s_ragged_shape* shape,
                                           const e2s_image* images_host, size_t* bytes) {
    Dims d;
    E2S_TRY(e2s::check_ragged(shape, images_host, 0, &d, nullptr));
    E2S_TRY(need(bytes));
    *bytes = e2s::prune_workspace_bytes(d);
    return E2S_OK;
}

e2s_status e2s_prune_ragged(const e2s_ragged_shape* shape, const e2s_params* params,
                            const e2s_image* images_host, const e2s_image* images_dev,
                            const void* q, const void* k, void* workspace,
                            size_t workspace_bytes, int32_t* keep_idx, float* fused_opt,
                            float* prio_c_opt, void* stream) {
    E2S_TRY(e2s::check_score_params(params));
    Dims d;
    int64_t min_side = 0;
    const int elem = params->dtype == E2S_DTYPE_F32 ? 4 : 2;
    E2S_TRY(e2s::check_ragged(shape, images_host, elem, &d, &min_side));
    E2S_TRY(need(images_dev));
    E2S_TRY(need(q));
    E2S_TRY(need(k));
    E2S_TRY(need(workspace));
    E2S_TRY(e2s::check_aligned(images_dev, 8));
    E2S_TRY(e2s::check_aligned(q, 16));
    E2S_TRY(e2s::check_aligned(k, 16));
    E2S_TRY(e2s::check_aligned(workspace, 256));
    if (workspace_bytes < e2s::prune_workspace_bytes(d)) return E2S_ERR_WORKSPACE_TOO_SMALL;
    // selection parameters: cells within every image's grid; keep is per image
    if (params->cells < 1 || params->cells > min_side) return E2S_ERR_BAD_PARAM;
    if (params->cells > e2s::kMaxCells) return E2S_ERR_UNSUPPORTED;
    if (!std::isfinite(params->lambda) || params->lambda < 0.0f || params->lambda > 1.0f)
        return E2S_ERR_BAD_PARAM;
    if (params->variant < E2S_VARIANT_FULL || params->variant > E2S_VARIANT_NO_SPATIAL_NOVELTY)
        return E2S_ERR_BAD_PARAM;
    bool any_keep = false;
    for (int64_t b = 0; b < d.B; ++b) any_keep = any_keep || images_host[b].keep > 0;
    if (any_keep) E2S_TRY(need(keep_idx));
    E2S_TRY(aligned_opt(keep_idx, 4));
    E2S_TRY(aligned_opt(fused_opt, 4));
    E2S_TRY(aligned_opt(prio_c_opt, 4));
    d.images = images_dev;
    return run_operation(d, params, q, k, workspace,
                         select_args(params, keep_idx, fused_opt, prio_c_opt), nullptr,
                         static_cast<hipStream_t>(stream));
}

e2s_status e2s_compact_tokens(const e2s_compact_shape* shape, const int32_t* keep_idx,
                              const void* src, void* dst, void* stream) {
    E2S_TRY(e2s::check_compact(shape));
    if (shape->keep == 0) return E2S_OK;
    E2S_TRY(need(keep_idx));
    E2S_TRY(need(src));
    E2S_TRY(need(dst));
    E2S_TRY(e2s::check_aligned(keep_idx, 4));
    E2S_TRY(e2s::check_aligned(src, 16));
    E2S_TRY(e2s::check_aligned(dst, 16));
    return from_hip(e2s::launch_compact(*shape, keep_idx, src, dst,
                                        static_cast<hipStream_t>(stream)));
}

}  // extern "C"
