// Randomized exercise of the C ABI's host-side argument checks (e2s_validate.cpp),
// built with AddressSanitizer and UndefinedBehaviorSanitizer by
// tests/test_validate_sanitized.py.  Every check is called on random, often
// extreme, arguments; the sanitizers turn any out-of-bounds access, signed
// overflow or other undefined behaviour into a failure.  A few fixed cases pin the
// expected status codes.
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <limits>
#include <random>
#include <vector>

#include "e2s_validate.h"

namespace {

std::mt19937_64 rng(2608);

int64_t pick64() {
    static const int64_t edges[] = {0, 1, -1, 2, 7, 8, 16, 63, 64, 128, 1023, 1024, 65535,
                                    1 << 20, (1 << 20) + 1, int64_t(1) << 31,
                                    std::numeric_limits<int32_t>::max(),
                                    std::numeric_limits<int64_t>::max(),
                                    std::numeric_limits<int64_t>::min(),
                                    std::numeric_limits<int64_t>::max() / 16,
                                    std::numeric_limits<int64_t>::max() / 64 + 1};
    const int n = sizeof(edges) / sizeof(edges[0]);
    switch (rng() % 3) {
        case 0: return edges[rng() % n];
        case 1: return static_cast<int64_t>(rng() % 4096) - 8;
        default: return static_cast<int64_t>(rng());
    }
}
int32_t pick32() {
    const int64_t v = pick64();
    if (v > std::numeric_limits<int32_t>::max()) return std::numeric_limits<int32_t>::max();
    if (v < std::numeric_limits<int32_t>::min()) return std::numeric_limits<int32_t>::min();
    return static_cast<int32_t>(v);
}
float pickf() {
    static const float edges[] = {0.f, 0.1f, 1.f, -0.f, -1.f, 1.0000001f, 0.5f,
                                  std::numeric_limits<float>::infinity(),
                                  std::numeric_limits<float>::quiet_NaN(), 1e30f, -1e-30f};
    return edges[rng() % (sizeof(edges) / sizeof(edges[0]))];
}

int failures = 0;
void expect(bool ok, const char* what) {
    if (!ok) {
        std::printf("FAIL: %s\n", what);
        ++failures;
    }
}

}  // namespace

int main() {
    using namespace e2s;
    // fixed cases
    e2s_shape good{2, 3, 4, 2, 64, 5, 6, 7};
    Dims d;
    expect(check_shape(&good, &d) == E2S_OK && d.N == 42 && d.tokens == 84, "good shape");
    e2s_shape bad = good;
    bad.num_heads = 5;
    expect(check_shape(&bad, &d) == E2S_ERR_BAD_SHAPE, "H % Hkv");
    bad = good;
    bad.head_dim = 96;
    expect(check_shape(&bad, &d) == E2S_ERR_UNSUPPORTED, "head_dim 96");
    bad = good;
    bad.grid_h = 2048;
    bad.grid_w = 1024;
    expect(check_shape(&bad, &d) == E2S_ERR_UNSUPPORTED, "N > 2^20");
    e2s_compact_shape cs{2, 1, 8, 4, 8, 2, {64, 64, 8}, {32, 32, 8}};
    expect(check_compact(&cs) == E2S_OK, "good compaction");
    cs.src_stride[2] = std::numeric_limits<int64_t>::max();
    expect(check_compact(&cs) != E2S_OK, "huge compaction stride");

    // random cases
    long n_ok = 0;
    for (int it = 0; it < 200000; ++it) {
        e2s_shape s{pick32(), pick32(), pick32(), pick32(), pick32(), pick32(), pick32(), pick32()};
        if (rng() % 2) {
            s = good;
            reinterpret_cast<int32_t*>(&s)[rng() % 8] = pick32();
        }
        Dims dd;
        const e2s_status st = check_shape(&s, &dd);
        if (st == E2S_OK) {
            ++n_ok;
            expect(dd.N == int64_t(s.grid_h) * s.grid_w && dd.group * dd.Hkv == dd.H, "dims");
            e2s_params p{int32_t(rng() % 4) - 1, int32_t(rng() % 3) - 1, pickf(), pick32(), pickf(),
                         pick32(), int32_t(rng() % 8) - 1};
            (void)check_score_params(&p);
            (void)check_select_params(&p, dd);
            size_t ws = prune_workspace_bytes(dd);
            expect(ws >= support_region_bytes(dd), "workspace");
            if (dd.L <= E2S_MAX_VIEW_LAYERS) {
                e2s_qk_views v{};
                for (int l = 0; l < E2S_MAX_VIEW_LAYERS; ++l) {
                    v.q[l] = reinterpret_cast<const void*>(uintptr_t(16) * (1 + rng() % 1024));
                    v.k[l] = reinterpret_cast<const void*>(uintptr_t(16) * (1 + rng() % 1024) +
                                                           (rng() % 8 == 0 ? 2 : 0));
                }
                v.q_stride_image = pick64();
                v.q_stride_head = pick64();
                v.q_stride_text = pick64();
                v.k_stride_image = pick64();
                v.k_stride_head = pick64();
                v.k_stride_token = pick64();
                (void)check_views(&v, dd, (rng() % 2) ? 2 : 4);
            }
        }
        // ragged batches
        const int B = 1 + int(rng() % 6);
        e2s_ragged_shape rs{B, pick32(), pick32(), pick32(), (rng() % 2) ? 64 : pick32()};
        if (rng() % 2) rs = e2s_ragged_shape{B, 2, 4, 2, 64};
        std::vector<e2s_image> ims(B);
        int64_t tok = 0;
        for (int b = 0; b < B; ++b) {
            e2s_image& im = ims[b];
            im.grid_h = (rng() % 4) ? int32_t(1 + rng() % 40) : pick32();
            im.grid_w = (rng() % 4) ? int32_t(1 + rng() % 40) : pick32();
            im.num_text = (rng() % 4) ? int32_t(1 + rng() % 200) : pick32();
            im.keep = (rng() % 4) ? int32_t(rng() % 50) : pick32();
            im.q_offset = (rng() % 4) ? int64_t(8 * (rng() % 100000)) : pick64();
            im.k_offset = (rng() % 4) ? int64_t(8 * (rng() % 100000)) : pick64();
            im.token_offset = (rng() % 4) ? tok : pick64();
            im.keep_offset = (rng() % 4) ? int64_t(b * 64) : pick64();
            // the next packed offset (kept small: only valid-looking grids advance it)
            if (im.grid_h > 0 && im.grid_w > 0 && im.grid_h <= 4096 && im.grid_w <= 4096)
                tok += int64_t(im.grid_h) * im.grid_w;
        }
        Dims rd;
        int64_t side = 0;
        if (check_ragged(&rs, ims.data(), (rng() % 2) ? 2 : 4, &rd, &side) == E2S_OK) {
            expect(rd.N >= 1 && rd.tokens >= rd.N && side >= 1, "ragged dims");
            (void)prune_workspace_bytes(rd);
        }
        // compaction
        e2s_compact_shape c{pick32(), pick32(), pick32(), pick32(), pick32(),
                            (rng() % 2) ? 2 : pick32(),
                            {pick64(), pick64(), pick64()},
                            {pick64(), pick64(), pick64()}};
        if (rng() % 2) {
            c = cs;
            c.src_stride[2] = 8;
            reinterpret_cast<int32_t*>(&c)[rng() % 6] = pick32();
            c.dst_stride[rng() % 3] = pick64();
        }
        (void)check_compact(&c);
        (void)check_aligned(reinterpret_cast<const void*>(uintptr_t(rng())), size_t(1) << (rng() % 9));
    }
    std::printf("%ld valid shapes among 200000 random calls; %d failures\n", n_ok, failures);
    return failures == 0 ? 0 : 1;
}
