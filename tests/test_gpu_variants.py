"""GPU parity of the ablation variants (Sec. 5, Table 2) against the oracle.

Each variant runs through e2s_prune (and, except attention top-K, through
e2s_fuse_select on the staged reliability outputs, which must give the same bits)
on seeded cases covering one query head per key head (the on-chip layer path at
full size, the staged path at small batch), grouped-query heads, fp32 and bf16,
an image of 20000 tokens (selection in segments), both score readings.  Kept sets: exact or tie-excused (R-A16's rule on the
variant's ranking score)."""
import numpy as np
import pytest

import oracle as O
import synth
from _helpers import check_keep_wellformed, compare_sets, log, to_device

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
E = pytest.importorskip("paper_2608_23253_amd")


def _small(name, **kw):
    base = dict(name=name, config_id=60, batch=2, num_layers=3, num_heads=4, num_kv_heads=4,
                head_dim=64, num_text=8, grid_h=8, grid_w=8, keep=16, lambdas=(0.3,),
                dtype="bf16", salient_count=4, clusters=0, shift_sigmas=2.0)
    base.update(kw)
    return synth.Config(**base)


CASES = [
    synth.config_by_name("tiny"),
    _small("gqa_d128", config_id=61, num_heads=6, num_kv_heads=2, head_dim=128, grid_h=7,
           grid_w=9, keep=20, cells=3),
    synth.config_by_name("llava").replace(batch=2),
    # 20000 visual tokens: the selections stream the image in segments
    _small("large_20000", config_id=62, batch=1, num_layers=2, num_heads=2, num_kv_heads=2,
           grid_h=100, grid_w=200, keep=2500, cells=4, salient_count=40, clusters=3),
]
VARIANTS = [v for v in O.VARIANTS]


@pytest.mark.parametrize("mode", ["mean_logit", "mean_prob"])
@pytest.mark.parametrize("variant", VARIANTS)
@pytest.mark.parametrize("cfg", CASES, ids=[c.name for c in CASES])
def test_variant_parity(cfg, variant, mode):
    log(f"[case] {cfg.name} variant={variant} mode={mode}")
    gh, gw, K, G, lam = cfg.grid_h, cfg.grid_w, cfg.keep, cfg.cells, cfg.lam
    q, k, _ = synth.gen_batch(cfg)
    qd, kd = to_device(q, cfg.dtype), to_device(k, cfg.dtype)
    keep, _, _ = E.prune(qd, kd, gh, gw, K, G, lam, mode, variant=variant)
    if variant != "a1_attention_topk":
        e, _ = E.score_heads(qd, kd, gh, gw, mode)
        rho, pbar = E.head_reliability(e, gh, gw)
        keep_f, _, _ = E.fuse_select(rho, pbar, gh, gw, K, G, lam, variant=variant)
        torch.cuda.synchronize()
        assert torch.equal(keep, keep_f)
    keep = keep.cpu().numpy()
    check_keep_wellformed(keep, gh * gw, K)
    lam32 = float(np.float32(lam))
    for b in range(cfg.batch):
        ref = O.prune_image(q[b], k[b], gh, gw, K, G, lam32, mode, variant=variant)
        cmp = compare_sets(keep[b], ref)
        log(f"  image {b}: {cmp.verdict} swaps={cmp.swaps} near-boundary={cmp.near_boundary}")
        assert cmp.verdict != "fail"


def _conflicting_keys(q, k, tokens, amp):
    """Keys with chosen tokens pushed toward the mean query in even layers and away
    from it in odd layers: their layers disagree, so their conflict K is large."""
    k = k.copy()
    for l in range(k.shape[1]):
        u = q[:, l].mean(axis=(1, 2))
        u = u / np.linalg.norm(u, axis=-1, keepdims=True)
        sign = 1.0 if l % 2 == 0 else -1.0
        for t in tokens:
            k[:, l, :, t, :] += sign * amp * u[:, None, :]
    return synth.bf16_bits_to_f32(synth.to_bf16_bits(k.astype(np.float32)))


def test_variants_change_the_selection():
    """Each variant keeps a different set from the full method on some image.  On
    the LLaVA-shaped case with a budget of 24 (fewer than three tokens per cell on
    average, so the novelty bonus competes with the salient clusters) for A1, A2,
    A3 and A5.  There the layer masses are ~1e-4, so K ~ 1e-8 and dropping the
    conflict factor (A4) reorders nothing; A4 is checked on high-contrast inputs
    whose tokens 3, 14, 25, ... have conflicting layers (K up to ~0.13), where
    conflict protection keeps tokens the plausibility alone drops.  The A4 sets
    there are also checked against the oracle."""
    cfg = synth.config_by_name("llava").replace(batch=2)
    q, k, _ = synth.gen_batch(cfg)
    qd, kd = to_device(q, "bf16"), to_device(k, "bf16")
    full, _, _ = E.prune(qd, kd, 24, 24, 24, 4, cfg.lam)
    for v in VARIANTS[1:]:
        if v == "a4_no_conflict_protection":
            continue
        other, _, _ = E.prune(qd, kd, 24, 24, 24, 4, cfg.lam, variant=v)
        assert not torch.equal(full, other), v
    hc = synth.heavy_tailed(cfg, name="heavy_llava")
    q, k, _ = synth.gen_batch(hc)
    k = _conflicting_keys(q, k, list(range(3, 576, 11)), 2.0)
    qd, kd = to_device(q, "bf16"), to_device(k, "bf16")
    full, _, _ = E.prune(qd, kd, 24, 24, hc.keep, 4, hc.lam)
    a4, _, _ = E.prune(qd, kd, 24, 24, hc.keep, 4, hc.lam, variant="a4_no_conflict_protection")
    assert not torch.equal(full, a4)
    a4 = a4.cpu().numpy()
    lam32 = float(np.float32(hc.lam))
    for b in range(hc.batch):
        ref = O.prune_image(q[b], k[b], 24, 24, hc.keep, 4, lam32,
                            variant="a4_no_conflict_protection")
        assert compare_sets(a4[b], ref).verdict != "fail"
