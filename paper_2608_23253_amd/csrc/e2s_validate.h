// Host-side argument checks of the C ABI.  Pure C++, no HIP: every entry point
// runs these before it touches the runtime, so an invalid call enqueues nothing.
#pragma once

#include <cstddef>
#include <cstdint>

#include "e2s.h"

namespace e2s {

// Derived sizes of one call.  All products are computed in 64 bits.
struct Dims {
    int64_t B, L, H, Hkv, D, NT, gh, gw, N;
    int64_t group;  // H / Hkv query heads per key head
    // Ragged batch: the device table of per-image records; NT and N are then the
    // largest N_T,b and N_b (launch sizes), gh and gw unused.  Null: uniform.
    const e2s_image* images = nullptr;
    // Q and K as per-layer views (host struct, copied into the kernel arguments),
    // or null (packed arrays).
    const e2s_qk_views* views = nullptr;
    // Token span of the per-token arrays: B * N (uniform), or the largest
    // token_offset + N_b (ragged); sizes the workspace.
    int64_t tokens = 0;
};

// Visual tokens per image.  Up to 16384 the per-image kernels keep an image's
// values on chip; beyond, they stream it (logits and column sums in the output
// rows, the selection in segments of 16384 tokens).
constexpr int64_t kMaxVisual = 1 << 20;
// Cells per side of the spatial grid: the selection keeps one 64-bit word per cell
// in LDS (128 KiB at G = 128).
constexpr int64_t kMaxCells = 128;
constexpr int64_t kMaxHeads = 128;     // per-token head supports held in registers

e2s_status check_shape(const e2s_shape* s, Dims* out);
// Views of Q and K for dtype (element size) and the validated shape.
e2s_status check_views(const e2s_qk_views* v, const Dims& d, int elem_bytes);
e2s_status check_score_params(const e2s_params* p);
e2s_status check_select_params(const e2s_params* p, const Dims& d);
e2s_status check_aligned(const void* ptr, size_t align);

// A ragged batch: the shape, every image record (sizes, offsets, alignment of the
// Q and K blocks for elements of elem_bytes bytes; 0 skips that check, disjoint
// token and keep ranges), giving Dims with the largest N_T,b and N_b and the
// token span.  min_side: the smallest grid side over the images.
e2s_status check_ragged(const e2s_ragged_shape* s, const e2s_image* images, int elem_bytes,
                        Dims* out, int64_t* min_side);

// Token compaction: counts, element size, 16-byte granularity of the vectors and
// strides, and that the largest offset of each array fits 63 bits.
e2s_status check_compact(const e2s_compact_shape* s);

// Workspace of e2s_layer_reliability and e2s_prune: the supports e [B,L,H,N] f32
// (used only when a layer's supports do not stay on chip), then rho and pbar_c
// [B,L,N] f32 (e2s_prune), each region rounded up to 256 bytes.
size_t support_region_bytes(const Dims& d);
size_t layer_region_bytes(const Dims& d);
size_t prune_workspace_bytes(const Dims& d);
size_t align_up(size_t x, size_t a);

}  // namespace e2s
