"""GPU parity of the ragged-batch entry point e2s_prune_ragged.

A ragged batch gives every image its own grid, text length and budget.  The path
never mixes images (Eq. 1-23 are per image), so each image's result must be the
one e2s_prune returns for that image alone, bit for bit, and must match the CPU
oracle under the same rule as the uniform path (fused masses within 1e-4 absolute
and within 1e-7 + 2e-3 |ref| per element, kept sets exact or differing only inside
the 1e-5 tie window).

Cases mix grids (ragged tails, a 2x3 grid at G = 2), text lengths (1 to 150, so the
mean-of-probabilities kernel takes one or two query chunks, 2 or 4 key tiles at a
time), budgets (0 to N_b), one query head per key head and grouped-query heads
(groups of 4, 7 and 16), bf16, fp16 and fp32 storage, d = 64 and 128, near-uniform and
peaked attention, packed and gapped layouts, and a batch large enough that every
(image, layer) gets its own workgroup on the on-chip layer path.
"""
import ctypes

import numpy as np
import pytest

import oracle as O
import synth
from _helpers import assert_mass_bar, check_keep_wellformed, compare_sets, log, to_device

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
E = pytest.importorskip("paper_2608_23253_amd")

MODES = ["mean_logit", "mean_prob"]


def _base(name, **kw):
    base = dict(name=name, config_id=70, batch=1, num_layers=2, num_heads=4, num_kv_heads=4,
                head_dim=64, num_text=8, grid_h=8, grid_w=8, keep=16, lambdas=(0.1,),
                dtype="bf16", salient_count=3, clusters=0, shift_sigmas=2.0)
    base.update(kw)
    return synth.Config(**base)


# (base config, [(grid_h, grid_w, num_text, keep)], cells)
CASES = {
    "mha_bf16_d128": (_base("mha_bf16_d128", config_id=71, num_layers=3, num_heads=6,
                            num_kv_heads=6, head_dim=128),
                      [(7, 9, 5, 20), (8, 8, 16, 16), (3, 5, 1, 0), (12, 10, 40, 30),
                       (4, 4, 2, 16), (11, 13, 150, 37)], 3),
    "gqa7_bf16_d128": (_base("gqa7_bf16_d128", config_id=72, num_heads=14, num_kv_heads=2,
                             head_dim=128),
                       [(16, 20, 33, 40), (9, 7, 3, 9), (21, 17, 64, 100), (5, 5, 130, 5)], 4),
    "gqa16_bf16_d64": (_base("gqa16_bf16_d64", config_id=73, num_heads=32, num_kv_heads=2),
                       [(6, 6, 7, 9), (10, 12, 20, 24), (13, 9, 4, 0)], 4),
    "gqa8_f32_d64": (_base("gqa8_f32_d64", config_id=74, dtype="f32", num_layers=1,
                           num_heads=8, num_kv_heads=1),
                     [(5, 13, 3, 7), (8, 8, 9, 64), (2, 3, 1, 2)], 2),
    "gqa4_f16_d128": (_base("gqa4_f16_d128", config_id=44, dtype="f16", num_heads=8,
                            num_kv_heads=2, head_dim=128),
                      [(9, 12, 20, 30), (5, 6, 3, 0), (14, 11, 70, 40)], 3),
    "mha_f32_d128": (_base("mha_f32_d128", config_id=75, dtype="f32", num_heads=3,
                           num_kv_heads=3, head_dim=128),
                     [(6, 7, 4, 10), (9, 9, 17, 20)], 3),
    # more than 16384 tokens: the batch streams every image's selection in segments
    # and (above 24576 tokens) keeps its logits in the output rows, the images alone
    # mostly not
    "large_gqa2_bf16_d128": (_base("large_gqa2_bf16_d128", config_id=81, num_layers=1,
                                   num_heads=4, num_kv_heads=2, head_dim=128, salient_count=40,
                                   clusters=3),
                             [(160, 170, 5, 2000), (12, 9, 7, 20), (140, 130, 30, 900),
                              (4, 4, 2, 3)], 4),
    # peaked attention (the online statistics of the mean-of-probabilities kernel);
    # N_T = 100 gives the batch query chunks of 112 rows, the images alone smaller
    # ones
    "heavy_mixed_bf16_d128": (_base("heavy_mixed_bf16_d128", config_id=78, num_heads=4,
                                    num_kv_heads=4, head_dim=128, value_std=2.0,
                                    shift_sigmas=4.0, salient_count=6),
                              [(12, 12, 16, 24), (24, 24, 64, 100), (9, 11, 100, 20),
                               (5, 7, 3, 0), (3, 5, 1, 4)], 3),
}


def _images(cfg, dims):
    out = []
    for b, dd in enumerate(dims):
        gh, gw, nt, keep = dd
        ic = cfg.replace(grid_h=gh, grid_w=gw, num_text=nt, keep=keep)
        q, k, _ = synth.gen_image(ic, b)
        out.append((q, k))
    return out


def _layout(cfg, dims, gaps=False):
    """Image records: packed, or (gaps) in reverse order with padding between the
    blocks of every array."""
    L, H, Hkv, D = cfg.num_layers, cfg.num_heads, cfg.num_kv_heads, cfg.head_dim
    arr = (E.Image * len(dims))()
    qo = ko = to = kk = 0
    order = list(range(len(dims)))[::-1] if gaps else list(range(len(dims)))
    for b in order:
        gh, gw, nt, keep = dims[b]
        n = gh * gw
        if gaps:
            qo, ko, to, kk = qo + 8 * 3, ko + 8 * 5, to + 7, kk + 3
        arr[b] = E.Image(gh, gw, nt, keep, qo, ko, to, kk)
        qo += L * H * nt * D
        ko += L * Hkv * n * D
        to += n
        kk += keep
    return arr, qo, ko


def _upload(cfg, imgs, arr, qtot, ktot):
    q = np.zeros(qtot, np.float32)
    k = np.zeros(ktot, np.float32)
    for b, (qb, kb) in enumerate(imgs):
        q[arr[b].q_offset:arr[b].q_offset + qb.size] = qb.reshape(-1)
        k[arr[b].k_offset:arr[b].k_offset + kb.size] = kb.reshape(-1)
    return to_device(q, cfg.dtype), to_device(k, cfg.dtype)


def _run(cfg, dims, cells, mode, gaps=False, variant="full", lam=0.1):
    L, H, Hkv, D = cfg.num_layers, cfg.num_heads, cfg.num_kv_heads, cfg.head_dim
    imgs = _images(cfg, dims)
    arr, qtot, ktot = _layout(cfg, dims, gaps)
    qd, kd = _upload(cfg, imgs, arr, qtot, ktot)
    keep, fused, prio = E.prune_ragged(qd, kd, arr, L, H, Hkv, D, cells, lam, mode,
                                       want_fused=True, want_prio=True, variant=variant)
    torch.cuda.synchronize()
    return imgs, arr, keep, fused, prio


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("name", list(CASES))
def test_ragged_matches_each_image_alone_and_the_oracle(name, mode):
    cfg, dims, cells = CASES[name]
    log(f"[case] ragged {name} mode={mode} dims={dims}")
    imgs, arr, keep, fused, prio = _run(cfg, dims, cells, mode, gaps=(name == "mha_bf16_d128"))
    keep_all = keep.cpu().numpy()
    fused_all, prio_all = fused.cpu().numpy(), prio.cpu().numpy()
    for b, ((qb, kb), (gh, gw, nt, K)) in enumerate(zip(imgs, dims)):
        im = arr[b]
        n = gh * gw
        kb_keep = keep_all[im.keep_offset:im.keep_offset + K]
        kb_fused = fused_all[im.token_offset:im.token_offset + n]
        kb_prio = prio_all[im.token_offset:im.token_offset + n]
        # the same image alone through the uniform entry point: the same bits
        a_keep, a_fused, a_prio = E.prune(to_device(qb[None], cfg.dtype),
                                          to_device(kb[None], cfg.dtype), gh, gw, K, cells, 0.1,
                                          mode, want_fused=True, want_prio=True)
        torch.cuda.synchronize()
        assert a_keep[0].cpu().numpy().tolist() == kb_keep.tolist(), f"image {b}: kept set"
        np.testing.assert_array_equal(a_fused[0].cpu().numpy(), kb_fused)
        np.testing.assert_array_equal(a_prio[0].cpu().numpy(), kb_prio)
        # the oracle
        check_keep_wellformed(kb_keep[None], n, K)
        ref = O.prune_image(qb, kb, gh, gw, K, cells, 0.1, mode)
        err = np.abs(kb_fused.astype(np.float64) - ref.fused)
        assert_mass_bar(kb_fused, ref.fused, f"image {b}: fused masses")
        cmp = compare_sets(kb_keep, ref)
        log(f"  image {b} {gh}x{gw} N_T={nt} K={K}: set {cmp.verdict} swaps={cmp.swaps} "
            f"max|d fused|={err.max():.2e}")
        assert cmp.verdict != "fail"


def test_ragged_uniform_batch_equals_prune():
    """A ragged call whose images all have one shape, packed, equals e2s_prune on the
    [B, ...] tensors bit for bit (here on the on-chip layer path: B * L >= CUs)."""
    cfg = _base("uniform_as_ragged", config_id=76, batch=64, num_layers=4, num_heads=6,
                num_kv_heads=6, head_dim=128, num_text=12, grid_h=9, grid_w=10, keep=25)
    q, k, _ = synth.gen_batch(cfg)
    qd, kd = to_device(q, "bf16"), to_device(k, "bf16")
    for mode in MODES:
        u_keep, u_fused, u_prio = E.prune(qd, kd, 9, 10, 25, 3, 0.1, mode, want_fused=True,
                                          want_prio=True)
        arr, _, _, _, _ = E.packed_images([(9, 10, 12, 25)] * 64, 4, 6, 6, 128)
        r_keep, r_fused, r_prio = E.prune_ragged(qd.reshape(-1), kd.reshape(-1), arr, 4, 6, 6,
                                                 128, 3, 0.1, mode, want_fused=True,
                                                 want_prio=True)
        torch.cuda.synchronize()
        assert torch.equal(u_keep.reshape(-1), r_keep)
        assert torch.equal(u_fused.reshape(-1, 3), r_fused)
        assert torch.equal(u_prio.reshape(-1), r_prio)


def test_ragged_layer_path_mixed_grids():
    """Enough (image, layer) pairs for the on-chip layer path, with mixed grids and
    text lengths: every image equals itself alone."""
    cfg = _base("layer_path_ragged", config_id=77, num_layers=4, num_heads=6, num_kv_heads=6,
                head_dim=128)
    rng = np.random.default_rng(77)
    dims = [(int(rng.integers(3, 14)), int(rng.integers(3, 14)), int(rng.integers(1, 40)), 0)
            for _ in range(70)]
    dims = [(gh, gw, nt, int(rng.integers(0, gh * gw + 1))) for gh, gw, nt, _ in dims]
    imgs, arr, keep, fused, prio = _run(cfg, dims, 3, "mean_logit")
    keep_all, prio_all = keep.cpu().numpy(), prio.cpu().numpy()
    for b in range(0, 70, 7):
        gh, gw, nt, K = dims[b]
        qb, kb = imgs[b]
        a_keep, _, a_prio = E.prune(to_device(qb[None], "bf16"), to_device(kb[None], "bf16"), gh,
                                    gw, K, 3, 0.1, "mean_logit", want_prio=True)
        torch.cuda.synchronize()
        im = arr[b]
        assert a_keep[0].cpu().numpy().tolist() == \
            keep_all[im.keep_offset:im.keep_offset + K].tolist()
        np.testing.assert_array_equal(a_prio[0].cpu().numpy(),
                                      prio_all[im.token_offset:im.token_offset + gh * gw])


@pytest.mark.parametrize("variant", ["a1_attention_topk", "a3_no_layer_fusion"])
def test_ragged_variants(variant):
    cfg, dims, cells = CASES["gqa7_bf16_d128"]
    imgs, arr, keep, _, _ = _run(cfg, dims, cells, "mean_logit", variant=variant)
    keep_all = keep.cpu().numpy()
    for b, ((qb, kb), (gh, gw, nt, K)) in enumerate(zip(imgs, dims)):
        a_keep, _, _ = E.prune(to_device(qb[None], "bf16"), to_device(kb[None], "bf16"), gh, gw,
                               K, cells, 0.1, "mean_logit", variant=variant)
        torch.cuda.synchronize()
        im = arr[b]
        assert a_keep[0].cpu().numpy().tolist() == \
            keep_all[im.keep_offset:im.keep_offset + K].tolist()


def test_ragged_workload_every_image():
    """The Qwen2-VL dynamic-resolution workload at full size: every image against
    the oracle (the launch configuration the benchmark times)."""
    rc = synth.ragged_by_name("qwen2vl_dynamic")
    qs, ks, _, dims = synth.gen_ragged(rc)
    cfg = rc.base
    L, H, Hkv, D = cfg.num_layers, cfg.num_heads, cfg.num_kv_heads, cfg.head_dim
    arr, qtot, ktot, _, _ = E.packed_images(dims, L, H, Hkv, D)
    qd, kd = _upload(cfg, list(zip(qs, ks)), arr, qtot, ktot)
    for mode in MODES:
        keep, fused, _ = E.prune_ragged(qd, kd, arr, L, H, Hkv, D, 4, 0.1, mode,
                                        want_fused=True)
        torch.cuda.synchronize()
        keep_all, fused_all = keep.cpu().numpy(), fused.cpu().numpy()
        counts = {}
        for b in range(len(dims)):
            gh, gw, nt, K = dims[b]
            im = arr[b]
            ref = O.prune_image(qs[b], ks[b], gh, gw, K, 4, 0.1, mode)
            got_f = fused_all[im.token_offset:im.token_offset + gh * gw]
            err = assert_mass_bar(got_f, ref.fused, f"image {b}: fused masses")
            cmp = compare_sets(keep_all[im.keep_offset:im.keep_offset + K], ref)
            log(f"  {mode} image {b} {gh}x{gw} N_T={nt} K={K}: {cmp.verdict} swaps={cmp.swaps} "
                f"max|d fused|={err:.2e}")
            counts[cmp.verdict] = counts.get(cmp.verdict, 0) + 1
            assert cmp.verdict != "fail"
        log(f"  {mode}: {len(dims)} images, sets {counts}")


def test_ragged_validation_on_device_pointers():
    """Invalid records are refused before anything is enqueued."""
    cfg, dims, cells = CASES["gqa16_bf16_d64"]
    L, H, Hkv, D = cfg.num_layers, cfg.num_heads, cfg.num_kv_heads, cfg.head_dim
    arr, qtot, ktot = _layout(cfg, dims)
    q = torch.zeros(qtot, device="cuda", dtype=torch.bfloat16)
    k = torch.zeros(ktot, device="cuda", dtype=torch.bfloat16)
    bad = (E.Image * len(dims))()
    ctypes.memmove(bad, arr, ctypes.sizeof(arr))
    bad[1].token_offset = bad[0].token_offset + 1            # overlaps image 0's tokens
    with pytest.raises(E.E2SError):
        E.prune_ragged(q, k, bad, L, H, Hkv, D, cells)
    ctypes.memmove(bad, arr, ctypes.sizeof(arr))
    bad[2].q_offset += 4                                      # not 16-byte aligned (bf16)
    with pytest.raises(E.E2SError):
        E.prune_ragged(q, k, bad, L, H, Hkv, D, cells)
    with pytest.raises(E.E2SError):                           # G above the 6x6 image's side
        E.prune_ragged(q, k, arr, L, H, Hkv, D, 7)


@pytest.mark.parametrize("heavy", [False, True], ids=["near_uniform", "peaked"])
def test_mean_prob_group_size_does_not_change_bits(heavy):
    """The mean-of-probabilities kernel takes 4 key tiles at a time when a query chunk
    holds 128 queries, else 1 when four workgroups' LDS fits a CU and 2 when it does
    not; an image's bits must not depend on which.  40 images with N_T <= 64 alone
    run with 1 (34 KiB per workgroup); one more image with N_T = 96 (51 KiB) makes
    the same images run with 2, one with N_T = 130 (two query chunks) with 4."""
    extra = dict(value_std=2.0, shift_sigmas=4.0) if heavy else {}
    cfg = _base("mp_group_size", config_id=79 + int(heavy), num_layers=2, num_heads=8,
                num_kv_heads=2, head_dim=128, salient_count=5, **extra)
    rng = np.random.default_rng(79)
    dims = [(int(rng.integers(2, 25)), int(rng.integers(2, 25)), int(rng.integers(1, 65)), 0)
            for _ in range(40)]
    dims = [(gh, gw, nt, int(rng.integers(0, gh * gw + 1))) for gh, gw, nt, _ in dims]
    dims[0] = (24, 24, 64, 100)
    log(f"[case] mean_prob group size heavy={heavy}")
    imgs, arr_a, keep_a, fused_a, prio_a = _run(cfg, dims, 2, "mean_prob")
    keep_a, fused_a, prio_a = keep_a.cpu().numpy(), fused_a.cpu().numpy(), prio_a.cpu().numpy()
    for extra_nt in (96, 130):
        _, arr_b, keep_b, fused_b, prio_b = _run(cfg, dims + [(6, 6, extra_nt, 5)], 2,
                                                 "mean_prob")
        keep_b, fused_b = keep_b.cpu().numpy(), fused_b.cpu().numpy()
        prio_b = prio_b.cpu().numpy()
        for b, (gh, gw, nt, K) in enumerate(dims):
            a, c = arr_a[b], arr_b[b]
            n = gh * gw
            np.testing.assert_array_equal(fused_a[a.token_offset:a.token_offset + n],
                                          fused_b[c.token_offset:c.token_offset + n])
            np.testing.assert_array_equal(prio_a[a.token_offset:a.token_offset + n],
                                          prio_b[c.token_offset:c.token_offset + n])
            assert keep_a[a.keep_offset:a.keep_offset + K].tolist() == \
                keep_b[c.keep_offset:c.keep_offset + K].tolist()
    for b in (0, 17, 33):
        gh, gw, nt, K = dims[b]
        qb, kb = imgs[b]
        a = arr_a[b]
        ref = O.prune_image(qb, kb, gh, gw, K, 2, 0.1, "mean_prob")
        got = fused_a[a.token_offset:a.token_offset + gh * gw].astype(np.float64)
        err = np.abs(got - ref.fused)
        assert_mass_bar(got, ref.fused, f"image {b}: fused masses")
        cmp = compare_sets(keep_a[a.keep_offset:a.keep_offset + K], ref)
        log(f"  image {b} {gh}x{gw} N_T={nt} K={K}: set {cmp.verdict} "
            f"max|d fused|={err.max():.2e}")
        assert cmp.verdict != "fail"
