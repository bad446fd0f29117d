/*
 * e2s.h - C ABI of the E2S-Pruner token-scoring path on AMD Instinct MI355X (gfx950).
 *
 * The path (arXiv 2608.23253, Sec. 3.1 and 4) takes, for every image of a batch,
 * the text-query and visual-key projections of L source layers and returns the
 * K visual tokens to keep:
 *
 *   score      text->visual attention per head, normalized over the visual tokens,
 *              mapped to a support p in [0,1)                   (Eq. 1, 8, 9)
 *   reliability head clarity x consistency, mean support        (Eq. 10)
 *   masses     (m(I), m(U), m(Theta)) per token and layer        (Eq. 11)
 *   fusion     Dempster's rule across the layers with the conflict
 *              of every step exported; retention priority q      (Eq. 12-19)
 *   select     cell representatives, novelty bonus, global top-K (Eq. 20-23)
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Every tensor argument is a DEVICE pointer to memory the caller allocated and
 *    owns.  The library never allocates, frees, copies between host and device,
 *    or synchronises.  Each call first validates all arguments on the host; an
 *    invalid call returns an error and enqueues nothing.  A valid call enqueues
 *    its kernels on `stream` (a hipStream_t; NULL = the null stream) and returns
 *    E2S_OK without waiting.  Errors inside a kernel are not reported.
 *  - Tensors are dense, row-major (last index fastest) with the layouts given
 *    below.  q and k must be 16-byte aligned, float/int outputs 4-byte aligned,
 *    double outputs 8-byte aligned.  Outputs must not overlap inputs or each other.
 *  - The library is stateless and reentrant; calls on different streams may
 *    run concurrently when they share no workspace and no output.  There is no
 *    global error state.  The one exception is e2s_prune_noalloc, whose workspace
 *    is a static device array of the library (one per GPU, shared by its calls).
 *  - The kernels run on the current HIP device; every pointer of a call must be
 *    memory of that device and `stream` one of its streams.
 *  - Centred quantities: the support p is exported as e = p - 1/2 and the
 *    retention priority q as c = 1 - q (Eq. 19 rewritten with Eq. 18 as
 *    c = m~(U) * (1 - K)).  Near the uniform-attention point p = 1/2 and q = 1,
 *    so the centred forms keep the digits that decide the ranking.
 *  - NaN or Inf in q/k give undefined values for that image only.
 *
 * Shape symbols: B batch, L source layers, H query heads, Hkv key heads
 * (H % Hkv == 0; query head h reads key head floor(h*Hkv/H)), d head_dim,
 * N_T text queries, N = N_V = grid_h * grid_w visual tokens in row-major
 * raster order, K tokens kept.
 */
#ifndef E2S_H
#define E2S_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define E2S_ABI_VERSION 9

#if defined(__GNUC__) || defined(__clang__)
#define E2S_API __attribute__((visibility("default")))
#else
#define E2S_API
#endif

typedef enum {
    E2S_OK = 0,
    E2S_ERR_NULL_POINTER = 1,         /* a required pointer is NULL                    */
    E2S_ERR_BAD_SHAPE = 2,            /* a count is out of range or inconsistent       */
    E2S_ERR_BAD_PARAM = 3,            /* dtype, mode, scale, cells, lambda or keep     */
    E2S_ERR_UNSUPPORTED = 4,          /* valid per the paper, not implemented here     */
    E2S_ERR_MISALIGNED = 5,           /* a pointer violates the alignment rule         */
    E2S_ERR_WORKSPACE_TOO_SMALL = 6,  /* e2s_prune workspace below the required size   */
    E2S_ERR_LAUNCH = 7,               /* the HIP runtime refused a kernel launch       */
    E2S_ERR_SCRATCH_TOO_SMALL = 8     /* e2s_prune_noalloc: the call needs more than
                                         E2S_NOALLOC_SCRATCH_BYTES of scratch, or the
                                         scratch's device address was not available     */
} e2s_status;

typedef enum { E2S_DTYPE_F32 = 0, E2S_DTYPE_BF16 = 1, E2S_DTYPE_F16 = 2 } e2s_dtype;

/* The two readings of how the text queries are reduced (Sec. 3.1, Eq. 1 and Eq. 8):
 *  MEAN_LOGIT: a_n = mean_t Q_t.K_n * scale (Eq. 1), r = softmax over n of a (Eq. 8).
 *  MEAN_PROB:  r_n = mean_t softmax over n of (Q_t.K_n * scale).              */
typedef enum { E2S_SCORE_MEAN_LOGIT = 0, E2S_SCORE_MEAN_PROB = 1 } e2s_score_mode;

typedef struct {
    int32_t batch;         /* B >= 1                                   */
    int32_t num_layers;    /* L >= 1 source layers, fused in order      */
    int32_t num_heads;     /* H >= 1, at most 128                      */
    int32_t num_kv_heads;  /* Hkv >= 1, H % Hkv == 0                   */
    int32_t head_dim;      /* d: 64 or 128                             */
    int32_t num_text;      /* N_T >= 1                                 */
    int32_t grid_h;        /* visual grid rows >= 1                    */
    int32_t grid_w;        /* visual grid cols >= 1; N = grid_h*grid_w <= 2^20  */
} e2s_shape;
/* Launch limits (E2S_ERR_UNSUPPORTED beyond them, for every entry point that takes
 * an e2s_shape or e2s_image records): B*L*H < 2^22 and B*L*ceil(N/64) < 2^24, N
 * being the largest image's token count; each keeps a kernel grid under 2^32
 * work-items. */

/* The full method and the ablation variants of the paper's ablation study (Sec. 5,
 * Table 2), each removing or replacing one component.  Honoured by e2s_prune and
 * e2s_prune_stage (all) and e2s_fuse_select (all but ATTENTION_TOPK, which needs
 * the per-head supports); the staged entry points always compute the full method.
 *  ATTENTION_TOPK      (A1) keep the K tokens of largest attention r averaged over
 *                      the layers and heads; no evidence, no spatial term
 *  NO_HEAD_RELIABILITY (A2) rho = 1 in Eq. 11 (Bayesian layer masses)
 *  NO_LAYER_FUSION     (A3) the last layer's masses only: no Dempster combination
 *                      with earlier layers or operations, so K = 0 and q = Pl
 *  NO_CONFLICT         (A4) q = Pl(I) instead of Eq. 19
 *  NO_SPATIAL_NOVELTY  (A5) lambda = 0 in Eq. 22                                  */
typedef enum {
    E2S_VARIANT_FULL = 0,
    E2S_VARIANT_ATTENTION_TOPK = 1,
    E2S_VARIANT_NO_HEAD_RELIABILITY = 2,
    E2S_VARIANT_NO_LAYER_FUSION = 3,
    E2S_VARIANT_NO_CONFLICT = 4,
    E2S_VARIANT_NO_SPATIAL_NOVELTY = 5
} e2s_variant;

typedef struct {
    int32_t dtype;   /* e2s_dtype of q and k                                     */
    int32_t mode;    /* e2s_score_mode                                           */
    float scale;     /* logit scale of Eq. 1; 0 selects 1/sqrt(head_dim)         */
    int32_t cells;   /* G: cells per side, 1 <= G <= min(grid_h, grid_w, 128) (paper: 4);
                        above 128: E2S_ERR_UNSUPPORTED */
    float lambda;    /* novelty weight of Eq. 22, finite, in [0, 1] (paper: 0.1) */
    int32_t keep;    /* K of Eq. 23, 0 <= K <= N                                 */
    int32_t variant; /* an e2s_variant; 0 is the full method                       */
} e2s_params;

/* Score stage (Sec. 3.1 Eq. 1; Sec. 4.1 Eq. 8-9).
 *   q  [B, L, H,   N_T, d]  dtype per params->dtype
 *   k  [B, L, Hkv, N,   d]  same dtype
 *   support_c [B, L, H, N] f32 out: e = p - 1/2 with p = N r / (1 + N r)
 *   r_opt     [B, L, H, N] f32 out or NULL: r, the normalized attention
 * Uses params->dtype, mode and scale (cells, lambda, keep are not checked). */
E2S_API e2s_status e2s_score_heads(const e2s_shape* shape, const e2s_params* params,
                           const void* q, const void* k,
                           float* support_c, float* r_opt, void* stream);

/* Head reliability (Sec. 4.1 Eq. 10) from support_c [B, L, H, N]:
 *   rho    [B, L, N] f32 out: (2/H)|sum_h e_h| * (1 - (2/H) sum_h |e_h - ebar|)
 *   pbar_c [B, L, N] f32 out: ebar = mean_h e_h = pbar - 1/2                       */
E2S_API e2s_status e2s_head_reliability(const e2s_shape* shape, const float* support_c,
                                float* rho, float* pbar_c, void* stream);

/* Layer masses (Sec. 4.1 Eq. 11) from rho, pbar_c [B, L, N]:
 *   mass [B, L, N, 3] f32 out: (rho (1/2 + ebar), rho (1/2 - ebar), 1 - rho)  = (I, U, Theta) */
E2S_API e2s_status e2s_head_masses(const e2s_shape* shape, const float* rho, const float* pbar_c,
                           float* mass, void* stream);

/* Dempster fusion across the L layers in index order (Sec. 4.2 Eq. 12-19).
 *   mass     [B, L, N, 3] f32 in (each triple a mass function over {I}, {U}, Theta)
 *   fused    [B, N, 3]    f32 out: m~ after the last layer
 *   conflict [B, L, N]    f32 out: K^(l) of Eq. 13, row l = 0 is 0
 *   prio_c   [B, N]       f32 out: c = 1 - q = m~(U) (1 - K^(L))
 * Total conflict (1 - K <= 0) makes the running mass vacuous (0, 0, 1) and records
 * K = 1, so q = 1 there (Eq. 19).  fused and conflict may be NULL (not written). */
E2S_API e2s_status e2s_ds_combine_layers(const e2s_shape* shape, const float* mass, float* fused,
                                 float* conflict, float* prio_c, void* stream);

/* Reliability, masses and fusion in one pass over support_c (Eq. 10-19); the
 * results are bit-identical to the three staged calls above.
 *   support_c [B, L, H, N] in; fused [B, N, 3], conflict [B, L, N] (both may be NULL),
 *   prio_c [B, N] out. */
E2S_API e2s_status e2s_fuse_evidence(const e2s_shape* shape, const float* support_c, float* fused,
                             float* conflict, float* prio_c, void* stream);

/* Spatial novelty and top-K (Sec. 4.3 Eq. 20-23) from prio_c [B, N]:
 *   cells: cell(n) = floor(row*G/grid_h)*G + floor(col*G/grid_w), row = n / grid_w,
 *   col = n % grid_w; the representative of a cell is its token of lowest c (highest
 *   q), lowest index on ties; adjusted complement c^ = (1-lambda) c + lambda (1-b),
 *   evaluated in double precision; the K tokens of smallest (c^, index) are kept.
 *   keep_idx   [B, K] int32 out, ascending token indices; may be NULL iff K == 0
 *   adj_c_opt  [B, N] double out or NULL: c^ = 1 - q~
 *   is_rep_opt [B, N] uint8 out or NULL: b of Eq. 21
 * Uses params->cells, lambda and keep. */
E2S_API e2s_status e2s_spatial_select(const e2s_shape* shape, const e2s_params* params,
                              const float* prio_c, int32_t* keep_idx, double* adj_c_opt,
                              uint8_t* is_rep_opt, void* stream);

/* Score and head reliability in one call (Sec. 3.1 Eq. 1; Sec. 4.1 Eq. 8-10):
 *   rho, pbar_c [B, L, N] f32 out, bit-identical to e2s_score_heads followed by
 *   e2s_head_reliability.
 * With the MEAN_LOGIT reading, H == Hkv, one layer's supports on chip
 * (H * (N + d) * 4 <= 153600 bytes) and at least as many (image, layer) pairs as
 * the device has compute units, one workgroup per (image, layer) keeps the
 * supports in local memory and only rho and pbar_c reach device memory; otherwise
 * the two staged kernels run with the supports in `workspace`.
 *   workspace: 256-byte aligned, >= e2s_prune_workspace_size bytes, contents
 *   undefined on return.
 * Uses params->dtype, mode and scale. */
E2S_API e2s_status e2s_layer_reliability(const e2s_shape* shape, const e2s_params* params,
                                 const void* q, const void* k, void* workspace,
                                 size_t workspace_bytes, float* rho, float* pbar_c,
                                 void* stream);

/* Masses, fusion and selection in one call (Sec. 4.1 Eq. 11; Sec. 4.2 Eq. 12-19;
 * Sec. 4.3 Eq. 20-23) from rho, pbar_c [B, L, N]; one workgroup per image.  With
 * the full method the results are bit-identical to e2s_head_masses ->
 * e2s_ds_combine_layers -> e2s_spatial_select.
 *   keep_idx [B, K] int32 out (NULL iff K == 0); fused_opt [B, N, 3] and
 *   prio_c_opt [B, N] f32 out or NULL.
 * Uses params->cells, lambda, keep and variant (ATTENTION_TOPK: E2S_ERR_UNSUPPORTED). */
E2S_API e2s_status e2s_fuse_select(const e2s_shape* shape, const e2s_params* params,
                           const float* rho, const float* pbar_c, int32_t* keep_idx,
                           float* fused_opt, float* prio_c_opt, void* stream);

/* Bytes of device workspace e2s_prune and e2s_layer_reliability need for this
 * shape (host-only query). */
E2S_API e2s_status e2s_prune_workspace_size(const e2s_shape* shape, const e2s_params* params,
                                    size_t* bytes);

/* The whole path (Algorithm 1 with every source layer fused before one top-K):
 * e2s_layer_reliability -> e2s_fuse_select on `stream`, with the intermediates in
 * `workspace` (256-byte aligned, >= e2s_prune_workspace_size bytes, contents
 * undefined on return); the result equals the staged calls bit for bit.
 *   keep_idx [B, K] int32 out (NULL iff K == 0); fused_opt [B, N, 3] and
 *   prio_c_opt [B, N] f32 out or NULL (not written by ATTENTION_TOPK).
 * Honours params->variant. */
E2S_API e2s_status e2s_prune(const e2s_shape* shape, const e2s_params* params, const void* q,
                     const void* k, void* workspace, size_t workspace_bytes,
                     int32_t* keep_idx, float* fused_opt, float* prio_c_opt, void* stream);

/* One pruning operation of Algorithm 1 over the current candidate tokens: the
 * progressive schedule (Sec. 4, Algorithm 1; Sec. 5.1) calls it once per pruning
 * layer with the survivors of the previous call.  shape describes the ORIGINAL
 * grid (cells of Eq. 20) and the operation's L evidence layers; num_cand = N_l
 * candidates, 1 <= N_l <= grid_h * grid_w, 0 <= params->keep <= N_l.
 *   q        [B, L, H, N_T, d]    text queries at the operation's layers
 *   k        [B, L, Hkv, N_l, d]  keys of the candidates, in candidate order
 *   cand_pos_opt [B, N_l] int32 or NULL: raster positions of the candidates,
 *            ascending (then index ties are position ties); NULL means positions
 *            0 .. N_l-1.  A cell is occupied when it holds a candidate; a position
 *            outside the grid gives its token no cell.
 *   m_prev_opt [B, N_l, 3] f32 or NULL: the candidates' fused masses after the
 *            previous operation (its m_out); every layer is combined onto them
 *   keep_idx [B, K] int32 out: kept candidate indices, ascending (NULL iff K == 0)
 *   keep_pos_opt [B, K] int32 out or NULL: their raster positions
 *   m_out_opt [B, K, 3] f32 out or NULL: their fused masses, the next call's m_prev
 * N_l is the N_l of Eq. 9 and the softmax of Eq. 8 runs over the candidates.
 * workspace: 256-byte aligned, >= e2s_prune_workspace_size(shape, params) bytes.
 * With num_cand = grid_h * grid_w and NULL optional arguments the result equals
 * e2s_prune's. */
E2S_API e2s_status e2s_prune_stage(const e2s_shape* shape, const e2s_params* params,
                           int32_t num_cand, const void* q, const void* k,
                           const int32_t* cand_pos_opt, const float* m_prev_opt,
                           void* workspace, size_t workspace_bytes, int32_t* keep_idx,
                           int32_t* keep_pos_opt, float* m_out_opt, void* stream);

/* ---------------------------------------------------------------------------
 * Ragged batches: every image with its own grid, text length and budget.
 * Vision-language models with dynamic resolution give each image its own patch
 * grid (Qwen2-VL, Sec. 5 of the paper), and prompts differ in length.  The path
 * is defined per image (Algorithm 1; Eq. 1-23 never mix images), so a ragged
 * batch computes, for every image b, exactly what e2s_prune computes for that
 * image alone.
 * ------------------------------------------------------------------------- */

/* One image of a ragged batch.  Offsets count elements of the array they index,
 * so the images may sit anywhere in the caller's buffers (packed, or with gaps).
 * q_offset and k_offset must keep the image's blocks 16-byte aligned (multiples
 * of 8 elements for bf16, 4 for f32). */
typedef struct {
    int32_t grid_h;        /* image b's grid rows >= 1                             */
    int32_t grid_w;        /* grid cols >= 1; N_b = grid_h * grid_w <= 2^20        */
    int32_t num_text;      /* N_T,b >= 1 text queries                              */
    int32_t keep;          /* K_b, 0 <= K_b <= N_b                                 */
    int64_t q_offset;      /* q + q_offset: the image's Q block [L, H, N_T,b, d]   */
    int64_t k_offset;      /* k + k_offset: its K block [L, Hkv, N_b, d]           */
    int64_t token_offset;  /* its N_b tokens in fused_opt / prio_c_opt start here;
                              the images' ranges [token_offset, token_offset + N_b)
                              must not overlap                                     */
    int64_t keep_offset;   /* its K_b kept indices in keep_idx start here; ranges
                              [keep_offset, keep_offset + K_b) must not overlap    */
} e2s_image;               /* 48 bytes */

typedef struct {
    int32_t batch;         /* B >= 1 images                                        */
    int32_t num_layers;    /* L >= 1                                               */
    int32_t num_heads;     /* H >= 1, at most 128                                  */
    int32_t num_kv_heads;  /* Hkv >= 1, H % Hkv == 0                               */
    int32_t head_dim;      /* d: 64 or 128                                         */
} e2s_ragged_shape;

/* Bytes of device workspace e2s_prune_ragged needs: the supports [L, H, .] and
 * rho, pbar_c [L, .] of every image, each image's block at L*H*token_offset
 * (resp. L*token_offset), i.e. (L*H + 2L) * T floats in three 256-byte aligned
 * regions, T = max over b of token_offset + N_b (host-only query). */
E2S_API e2s_status e2s_prune_ragged_workspace_size(const e2s_ragged_shape* shape,
                                                   const e2s_image* images_host,
                                                   size_t* bytes);

/* e2s_prune over a ragged batch.  images_host [B] (host memory) is validated and
 * sizes the launches; images_dev [B] (device memory, 8-byte aligned) must hold
 * the same records: the kernels read it.  Per image b, with its own N_b, N_T,b
 * and K_b, the results are those of e2s_prune on that image alone, bit for bit:
 *   keep_idx + keep_offset   [K_b] int32 out, ascending token indices of image b
 *   fused_opt + 3*token_offset [N_b, 3], prio_c_opt + token_offset [N_b] f32 out
 *   (both may be NULL; not written by ATTENTION_TOPK)
 * params->keep is ignored (each image has its own); params->cells must not
 * exceed any image's grid_h or grid_w.  keep_idx may be NULL iff every K_b is 0.
 * workspace: 256-byte aligned, >= e2s_prune_ragged_workspace_size bytes. */
E2S_API e2s_status e2s_prune_ragged(const e2s_ragged_shape* shape, const e2s_params* params,
                                    const e2s_image* images_host, const e2s_image* images_dev,
                                    const void* q, const void* k, void* workspace,
                                    size_t workspace_bytes, int32_t* keep_idx,
                                    float* fused_opt, float* prio_c_opt, void* stream);

/* ---------------------------------------------------------------------------
 * Token compaction: the model side of a pruning operation.  Algorithm 1 goes on
 * with the retained visual tokens only (its Ensure: V_keep; Sec. 4, and Sec. 5.1
 * for the layers after each pruning layer), so the caller's per-token vectors -
 * hidden states, and key/value cache rows - of the kept tokens are gathered
 * into shorter arrays.  A plain gather: no arithmetic of the method.
 * ------------------------------------------------------------------------- */
typedef struct {
    int32_t batch;          /* B >= 1 images                                          */
    int32_t rows;           /* R >= 1 rows per image (e.g. layers x KV heads, or 1)   */
    int32_t num_tokens;     /* N >= 1 tokens per row in src                           */
    int32_t keep;           /* K >= 0 tokens kept per image                           */
    int32_t channels;       /* C >= 1 elements per token vector, contiguous           */
    int32_t elem_bytes;     /* 2 or 4                                                 */
    int64_t src_stride[3];  /* elements between consecutive images, rows and tokens  */
    int64_t dst_stride[3];  /* the same for dst                                       */
} e2s_compact_shape;

/* dst[b, r, j, :] = src[b, r, keep_idx[b*K + j], :] for every image b, row r and
 * j < K (keep_idx [B, K] int32, e.g. e2s_prune's output; device memory).  An index
 * outside [0, N) leaves its dst vector unwritten.  src and dst are 16-byte
 * aligned, C * elem_bytes and every stride * elem_bytes are multiples of 16, and
 * dst must not overlap src.  Strides let src be a slice of a larger buffer (the
 * visual tokens of a key/value cache [B, Hkv, S, d] are a [B, Hkv, N, d] slice
 * with strides Hkv*S*d, S*d, d). */
E2S_API e2s_status e2s_compact_tokens(const e2s_compact_shape* shape, const int32_t* keep_idx,
                                      const void* src, void* dst, void* stream);

/* ---------------------------------------------------------------------------
 * Inputs in place: the source layers' text queries and visual keys read where the
 * model holds them.  Algorithm 1 takes, at every source layer, the attention
 * queries of the text tokens and the keys of the visual tokens (Sec. 3.1 Eq. 1);
 * in a running model these are per-layer projection outputs and key/value-cache
 * rows (after the rotary embedding), which e2s_prune would need copied into its
 * packed [B, L, H, N_T, d] and [B, L, Hkv, N, d] arrays.  Here each layer has a
 * base pointer and the rows are found by element strides, so no copy is made.
 * ------------------------------------------------------------------------- */
#define E2S_MAX_VIEW_LAYERS 16

typedef struct {
    /* Per source layer l < L: Q[b, l, h, t, :] = q[l] + b * q_stride_image +
     * h * q_stride_head + t * q_stride_text, and K[b, l, g, n, :] = k[l] +
     * b * k_stride_image + g * k_stride_head + n * k_stride_token, each a row of
     * d contiguous elements of params->dtype.  Every base and every stride times
     * the element size must be 16-byte aligned; strides are >= 0 and may differ
     * from the packed ones (the visual tokens of a cache [B, Hkv, S, d] starting
     * at token v0: k[l] = cache_l + v0 * d, strides Hkv*S*d, S*d, d; token-major
     * projections [B, T, H, d]: strides T*H*d, d, H*d).  Entries l >= L unused. */
    const void* q[E2S_MAX_VIEW_LAYERS];
    const void* k[E2S_MAX_VIEW_LAYERS];
    int64_t q_stride_image, q_stride_head, q_stride_text;
    int64_t k_stride_image, k_stride_head, k_stride_token;
} e2s_qk_views;

/* e2s_prune with Q and K given as views (L <= E2S_MAX_VIEW_LAYERS, else
 * E2S_ERR_UNSUPPORTED); everything else as e2s_prune, including the workspace
 * (e2s_prune_workspace_size) and the results, which equal e2s_prune's on packed
 * copies of the same values bit for bit.  The views struct is read on the host
 * during the call; the rows it points to are device memory that the call only
 * reads. */
E2S_API e2s_status e2s_prune_views(const e2s_shape* shape, const e2s_params* params,
                                   const e2s_qk_views* views, void* workspace,
                                   size_t workspace_bytes, int32_t* keep_idx, float* fused_opt,
                                   float* prio_c_opt, void* stream);

/* ---------------------------------------------------------------------------
 * For callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc): e2s_prune without the
 * caller's workspace.
 * ------------------------------------------------------------------------- */

/* Size of the library's static device scratch: one array per GPU, held from the
 * first e2s_prune_noalloc call on that GPU until the process ends. */
#define E2S_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)

/* e2s_prune with its workspace taken from the library's static scratch instead of
 * an argument.  Everything else (arguments, validation, kernels, results) is
 * e2s_prune's: the results equal e2s_prune's bit for bit.  The call allocates
 * nothing: no hipMalloc or hipFree, no allocating library routine.  Its first call
 * on a device, with that device current, looks up that device's copy of the
 * scratch (hipGetSymbolAddress) and keeps the address for later calls.
 *   A shape whose e2s_prune_workspace_size exceeds E2S_NOALLOC_SCRATCH_BYTES (e.g.
 *   more than 64 LLaVA-shaped images per call) returns E2S_ERR_SCRATCH_TOO_SMALL
 *   and enqueues nothing; so does a failed address lookup.
 *   Every call on one GPU shares that GPU's scratch, which keeps the last call's
 *   contents (the kernels write every scratch byte before they read it, so no
 *   call needs it cleared).  Calls that overlap in time on one GPU (other streams,
 *   other host threads) race on it: order them on one stream, or use e2s_prune
 *   with a workspace each. */
E2S_API e2s_status e2s_prune_noalloc(const e2s_shape* shape, const e2s_params* params,
                                     const void* q, const void* k, int32_t* keep_idx,
                                     float* fused_opt, float* prio_c_opt, void* stream);

/* Measurement helper, not a step of the method: a streaming read of device memory,
 * which the benchmark times to report the achievable read bandwidth beside the
 * nominal HBM peak.  `workgroups` workgroups of 256 threads each read one
 * contiguous share of buf[0 .. bytes) (16-byte aligned, bytes > 0 and a multiple
 * of 16) with 16-byte non-temporal loads and combine the words with XOR; the
 * 4-byte `sink` (device memory) is written only when that XOR equals a fixed
 * value, so the loads cannot be dropped and nothing else is written.
 * workgroups: 1 .. 65535.  Enqueued on `stream`. */
E2S_API e2s_status e2s_read_probe(const void* buf, size_t bytes, int32_t workgroups,
                                  uint32_t* sink, void* stream);

/* Static description of a status code (never NULL). */
E2S_API const char* e2s_status_string(e2s_status status);

/* E2S_ABI_VERSION of the built library. */
E2S_API int32_t e2s_abi_version(void);

#ifdef __cplusplus
}
#endif
#endif /* E2S_H */
