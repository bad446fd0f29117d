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
};

constexpr int64_t kMaxVisual = 16384;  // one image's scores fit in a workgroup's LDS
constexpr int64_t kMaxHeads = 128;     // per-token head supports held in registers

e2s_status check_shape(const e2s_shape* s, Dims* out);
e2s_status check_score_params(const e2s_params* p);
e2s_status check_select_params(const e2s_params* p, const Dims& d);
e2s_status check_aligned(const void* ptr, size_t align);

// Workspace of e2s_layer_reliability and e2s_prune: the supports e [B,L,H,N] f32
// (used only when a layer's supports do not stay on chip), then rho and pbar_c
// [B,L,N] f32 (e2s_prune), each region rounded up to 256 bytes.
size_t support_region_bytes(const Dims& d);
size_t layer_region_bytes(const Dims& d);
size_t prune_workspace_bytes(const Dims& d);
size_t align_up(size_t x, size_t a);

}  // namespace e2s
