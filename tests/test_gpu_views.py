"""GPU checks of e2s_prune_views: the source layers' queries and keys read in place.

Each case builds, per source layer, the storage a model holds: a key/value cache
[B, Hkv, S, d] whose visual tokens start at token 7, and token-major query
projections [B, T, H, d] whose text tokens start at token 4, every other row
filled with unrelated values.  The views of those tensors must give exactly the
bits e2s_prune gives on packed copies (the kernels change only how they find a
head's rows), on the on-chip layer path, the staged path, grouped-query heads,
fp32 storage, both score readings, an ablation variant and an image whose logits
do not fit in LDS.
"""
import pytest

import synth
from _helpers import log, to_device

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
E = pytest.importorskip("paper_2608_23253_amd")


def _cfg(name, **kw):
    base = dict(name=name, config_id=90, batch=2, num_layers=3, num_heads=4, num_kv_heads=4,
                head_dim=64, num_text=8, grid_h=8, grid_w=9, keep=16, lambdas=(0.1,),
                dtype="bf16", salient_count=4, clusters=0, shift_sigmas=2.0)
    base.update(kw)
    return synth.Config(**base)


CASES = [
    _cfg("staged_mha_d64"),
    # batch x layers >= the CU count: the on-chip layer path
    _cfg("layer_path_d128", config_id=91, batch=64, num_layers=4, num_heads=6, num_kv_heads=6,
         head_dim=128, num_text=12, grid_h=9, grid_w=10, keep=25),
    # grouped-query heads over many workgroups
    _cfg("gqa4_batch32", config_id=99, batch=32, num_layers=4, num_heads=8, num_kv_heads=2,
         head_dim=128, num_text=10, grid_h=8, grid_w=12, keep=20),
    _cfg("gqa7_d128", config_id=92, num_heads=14, num_kv_heads=2, head_dim=128, grid_h=11,
         grid_w=7, keep=20),
    _cfg("f16_gqa2", config_id=43, dtype="f16", num_heads=6, num_kv_heads=3, head_dim=128,
         num_text=9, keep=12),
    _cfg("gqa4_f32", config_id=93, dtype="f32", num_layers=2, num_heads=8, num_kv_heads=2,
         num_text=5, keep=9),
    # 462 tokens, 40 queries: the register-resident mean-of-probabilities kernel
    _cfg("resident_gqa2_d128", config_id=95, num_heads=6, num_kv_heads=3, head_dim=128,
         num_text=40, grid_h=21, grid_w=22, keep=50, salient_count=8, clusters=2),
    # 25600 tokens: logits in the output rows, selection in segments
    _cfg("large_mha", config_id=94, batch=1, num_layers=1, num_heads=2, num_kv_heads=2,
         num_text=3, grid_h=160, grid_w=160, keep=3000, salient_count=30, clusters=3),
]


def _in_model_storage(qd, kd, v0=7, t0=4):
    """Per layer: (query view [B, H, N_T, d] of token-major projections, key view
    [B, Hkv, N, d] of a key/value cache), holding the values of qd and kd."""
    B, L, H, NT, D = qd.shape
    Hkv, N = kd.shape[2], kd.shape[3]
    qv, kv = [], []
    for l in range(L):
        proj = torch.randn((B, NT + t0 + 5, H, D), device=qd.device).to(qd.dtype)
        proj[:, t0:t0 + NT] = qd[:, l].transpose(1, 2)
        cache = torch.randn((B, Hkv, N + v0 + 3, D), device=kd.device).to(kd.dtype)
        cache[:, :, v0:v0 + N] = kd[:, l]
        qv.append(proj[:, t0:t0 + NT].transpose(1, 2))
        kv.append(cache[:, :, v0:v0 + N])
    return qv, kv


@pytest.mark.parametrize("mode", ["mean_logit", "mean_prob"])
@pytest.mark.parametrize("cfg", CASES, ids=[c.name for c in CASES])
def test_views_equal_packed(cfg, mode):
    log(f"[case] views {cfg.name} mode={mode} B={cfg.batch} L={cfg.num_layers} "
        f"H={cfg.num_heads}/{cfg.num_kv_heads} d={cfg.head_dim} grid={cfg.grid_h}x{cfg.grid_w}")
    gh, gw, K, G, lam = cfg.grid_h, cfg.grid_w, cfg.keep, cfg.cells, cfg.lam
    q, k, _ = synth.gen_batch(cfg)
    qd, kd = to_device(q, cfg.dtype), to_device(k, cfg.dtype)
    qv, kv = _in_model_storage(qd, kd)
    assert not qv[0].is_contiguous() and not kv[0].is_contiguous()
    variants = ["full", "a1_attention_topk"] if cfg.name == "staged_mha_d64" else ["full"]
    for variant in variants:
        a = E.prune(qd, kd, gh, gw, K, G, lam, mode, want_fused=True, want_prio=True,
                    variant=variant)
        b = E.prune_views(qv, kv, gh, gw, K, G, lam, mode, want_fused=True, want_prio=True,
                          variant=variant)
        torch.cuda.synchronize()
        assert torch.equal(a[0], b[0]), f"{variant}: kept indices"
        if variant == "full":
            assert torch.equal(a[1], b[1]) and torch.equal(a[2], b[2]), f"{variant}: masses"
