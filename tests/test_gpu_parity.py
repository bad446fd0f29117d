"""GPU parity of every stage against the CPU oracle on small seeded cases.

Shapes span several tiles and ragged tails (token counts that are not multiples
of 16 or 64, query-head groups of 1, 2, 4, 7, 8, 12 and 16, head_dim 64 and 128,
fp32, bf16 and fp16 storage, one to eight source layers) and include the largest grid whose
selection stays in registers (128 x 128 = 16384 tokens), larger grids up to 40000
tokens (selection in segments, logits or column sums in the output rows), and
batches with at least one (image, layer) per compute unit, where the whole path
keeps each layer's supports on chip.  Each stage is checked twice: fed the GPU's own
upstream output (isolates that stage's arithmetic) and end to end from Q and K.

Tolerances, all float32 arithmetic on exact inputs (err <= atol + rtol |ref|
unless stated otherwise):
  r (Eq. 8), e = p - 1/2 (Eq. 9)      atol 1e-6 / rtol 2e-4 of the logit-scale error
  evidence stages on equal inputs      atol 1e-7 / rtol 2e-5
  fused masses end to end              two gates, both enforced: max |d| <= 1e-4 (the
                                       stated bar), and |d| <= 1e-7 + 2e-3 |ref| per
                                       element
  kept sets                            exact, or differing only by tokens whose
                                       oracle score is within 1e-5 of the K-th
  selection on equal inputs            bit-exact sets and representatives
"""
import numpy as np
import pytest

import oracle as O
import synth
from _helpers import (TIE_GAP, SelectGeom, assert_mass_bar, check_keep_wellformed,
                      compare_sets, log, oracle_images, to_device)

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
E = pytest.importorskip("paper_2608_23253_amd")

MODES = ["mean_logit", "mean_prob"]


def F32(x):
    """The value a float parameter has after crossing the C ABI."""
    return float(np.float32(x))


def _small(name, **kw):
    base = dict(name=name, config_id=50, batch=2, num_layers=2, num_heads=4, num_kv_heads=4,
                head_dim=64, num_text=8, grid_h=8, grid_w=8, keep=16, lambdas=(0.1,),
                dtype="bf16", salient_count=4, clusters=0, shift_sigmas=2.0)
    base.update(kw)
    return synth.Config(**base)


CASES = [
    synth.config_by_name("tiny"),
    _small("ragged_bf16_d128", config_id=51, num_layers=3, num_heads=6, num_kv_heads=3,
           head_dim=128, num_text=5, grid_h=7, grid_w=9, keep=20),
    _small("ragged_f32_gqa8", config_id=52, dtype="f32", num_layers=1, num_heads=8,
           num_kv_heads=1, num_text=3, grid_h=5, grid_w=13, keep=7, lambdas=(0.25,), cells=3),
    _small("group7_d128", config_id=53, num_heads=14, num_kv_heads=2, head_dim=128, num_text=9,
           grid_h=11, grid_w=11, keep=30, salient_count=6, clusters=2),
    _small("group12_chunks", config_id=54, num_heads=12, num_kv_heads=1, num_text=4,
           grid_h=6, grid_w=6, keep=9, cells=2, lambdas=(0.5,)),
    # a full 16-head matrix-core tile, 4 | N (vector stores), several tiles per wave
    _small("group16_d128", config_id=59, num_heads=32, num_kv_heads=2, head_dim=128,
           num_text=7, grid_h=16, grid_w=20, keep=40, salient_count=12, clusters=3),
    synth.config_by_name("llava").replace(batch=2),
    # more text queries than one LDS chunk of the mean-of-probabilities kernel (128),
    # ragged in both queries and tokens
    _small("query_chunks_150", config_id=60, num_heads=4, num_kv_heads=2, head_dim=128,
           num_text=150, grid_h=9, grid_w=11, keep=20),
    synth.heavy_tailed(_small("heavy_d128", config_id=55, num_layers=4, num_heads=8,
                              num_kv_heads=8, head_dim=128, num_text=16, grid_h=12, grid_w=12,
                              keep=24, salient_count=8, clusters=2)),
    synth.heavy_tailed(synth.config_by_name("llava").replace(batch=1), name="heavy_llava"),
    # peaked attention with d = 128 and 100 queries: the mean-of-probabilities
    # kernel's online statistics with a query chunk of 112 rows
    synth.heavy_tailed(_small("heavy_text100_d128", config_id=63, num_layers=2, num_heads=4,
                              num_kv_heads=4, head_dim=128, num_text=100, grid_h=12,
                              grid_w=12, keep=24, salient_count=8), name="heavy_text100"),
    # the register-resident mean-of-probabilities kernel (bf16, at most 64 text
    # queries, 385 to 576 tokens): 1 to 4 query blocks, d = 64 and 128, waves with
    # unequal tile counts, grouped-query heads, and peaked attention, which leaves the
    # tight range and takes the two-pass fallback
    _small("resident_q37_d128", config_id=70, num_heads=4, num_kv_heads=2, head_dim=128,
           num_text=37, grid_h=23, grid_w=19, keep=60, salient_count=10, clusters=2),
    _small("resident_q20_d64", config_id=71, num_text=20, grid_h=24, grid_w=24, keep=100,
           salient_count=12, clusters=3),
    _small("resident_q5", config_id=72, num_text=5, grid_h=20, grid_w=25, keep=50),
    # the resident kernel's boundaries: 385 tokens (7 tiles for the first wave, 6 for
    # the others) with 16 and 17 queries (one and two query blocks), a single query
    # over 576 tokens; 384 tokens and 65 queries take the two-pass kernel
    _small("resident_n385_q16", config_id=74, num_text=16, grid_h=5, grid_w=77, keep=40),
    _small("resident_n385_q17", config_id=75, head_dim=128, num_text=17, grid_h=11,
           grid_w=35, keep=40),
    _small("resident_q1_n576", config_id=76, num_text=1, grid_h=24, grid_w=24, keep=64),
    _small("two_pass_n384", config_id=77, num_text=64, grid_h=16, grid_w=24, keep=40),
    _small("two_pass_q65", config_id=78, head_dim=128, num_text=65, grid_h=24, grid_w=24,
           keep=64),
    synth.heavy_tailed(_small("resident_heavy_q48", config_id=73, head_dim=128, num_text=48,
                              grid_h=22, grid_w=22, keep=40, salient_count=12, clusters=2),
                       name="resident_heavy_q48"),
    _small("max_grid_16384", config_id=56, batch=1, num_layers=1, num_heads=2, num_kv_heads=1,
           num_text=2, grid_h=128, grid_w=128, keep=1000, salient_count=40, clusters=4),
    # more than 16384 visual tokens: the selection streams the image in segments;
    # above 24576 the logits of the one-head-per-key-head and grouped-query kernels
    # go to the output rows, and above 16384 the mean-of-probabilities column sums
    _small("large_grid_22500", config_id=64, batch=1, num_layers=2, num_heads=4, num_kv_heads=4,
           head_dim=128, num_text=6, grid_h=150, grid_w=150, keep=3000, salient_count=60,
           clusters=4),
    _small("large_mha_33000", config_id=65, batch=2, num_layers=1, num_heads=2, num_kv_heads=2,
           num_text=4, grid_h=150, grid_w=220, keep=4000, salient_count=50, clusters=3),
    _small("large_gqa_27200", config_id=66, batch=1, num_layers=1, num_heads=8, num_kv_heads=2,
           head_dim=128, num_text=5, grid_h=160, grid_w=170, keep=5000, salient_count=80,
           clusters=5),
    _small("large_f32_gqa_40000", config_id=67, dtype="f32", batch=1, num_layers=1,
           num_heads=4, num_kv_heads=1, num_text=3, grid_h=200, grid_w=200, keep=20000,
           cells=8, salient_count=100, clusters=6),
    # fp16 storage: per-head kernel, grouped-query vector kernel, the layer path, and
    # the mean-of-probabilities kernel on v_mfma_f32_16x16x32_f16
    _small("f16_mha_d128", config_id=40, dtype="f16", num_heads=4, num_kv_heads=4,
           head_dim=128, num_text=10, grid_h=9, grid_w=11, keep=20),
    _small("f16_gqa4_d64", config_id=41, dtype="f16", num_heads=12, num_kv_heads=3,
           num_text=6, grid_h=7, grid_w=10, keep=15, cells=3),
    _small("f16_layer_path_d64", config_id=42, dtype="f16", batch=64, num_layers=4,
           num_heads=6, num_kv_heads=6, num_text=5, grid_h=7, grid_w=9, keep=13, cells=3),
    # batch x layers >= the CU count: e2s_prune / e2s_layer_reliability take the
    # on-chip layer path (one workgroup per image and layer)
    _small("layer_path_ragged", config_id=57, batch=64, num_layers=4, num_heads=6,
           num_kv_heads=6, num_text=5, grid_h=7, grid_w=9, keep=13, cells=3),
    _small("layer_path_f32_d128", config_id=58, batch=32, num_layers=8, num_heads=20,
           num_kv_heads=20, head_dim=128, num_text=3, grid_h=9, grid_w=10, keep=25,
           dtype="f32", lambdas=(0.2,)),
]


def _errs(name, got, ref, atol, rtol):
    got = np.asarray(got, dtype=np.float64)
    err = np.abs(got - ref)
    bound = atol + rtol * np.abs(ref)
    worst = float((err / bound).max()) if err.size else 0.0
    log(f"    {name:10s} max|d|={err.max():.3e} max|d|/bound={worst:.3f}")
    assert (err <= bound).all(), f"{name}: {int((err > bound).sum())} elements out of tolerance"


def _run_case(cfg, mode):
    log(f"[case] {cfg.name} mode={mode} B={cfg.batch} L={cfg.num_layers} H={cfg.num_heads}/"
        f"{cfg.num_kv_heads} d={cfg.head_dim} NT={cfg.num_text} grid={cfg.grid_h}x{cfg.grid_w} "
        f"K={cfg.keep} G={cfg.cells} lam={cfg.lam} {cfg.dtype}")
    gh, gw, K, G, lam = cfg.grid_h, cfg.grid_w, cfg.keep, cfg.cells, cfg.lam
    q, k, _ = synth.gen_batch(cfg)
    qd, kd = to_device(q, cfg.dtype), to_device(k, cfg.dtype)
    e, r = E.score_heads(qd, kd, gh, gw, mode, want_r=True)
    rho, pbar = E.head_reliability(e, gh, gw)
    mass = E.head_masses(rho, pbar, gh, gw)
    fused, conflict, prio = E.ds_combine_layers(mass, gh, gw)
    f2, c2, p2 = E.fuse_evidence(e, gh, gw)
    keep, adj, rep = E.spatial_select(prio, gh, gw, K, G, lam, want_adj=True, want_rep=True)
    keep_p, fused_p, prio_p = E.prune(qd, kd, gh, gw, K, G, lam, mode, want_fused=True,
                                      want_prio=True)
    rho_l, pbar_l = E.layer_reliability(qd, kd, gh, gw, mode)
    keep_f, fused_f, prio_f = E.fuse_select(rho, pbar, gh, gw, K, G, lam, want_fused=True,
                                            want_prio=True)
    torch.cuda.synchronize()

    # fused / end-to-end entry points return exactly the staged bits (the on-chip
    # layer path for one query head per key head in the mean-of-logits reading, the
    # staged kernels otherwise)
    assert torch.equal(fused, f2) and torch.equal(conflict, c2) and torch.equal(prio, p2)
    assert torch.equal(rho, rho_l) and torch.equal(pbar, pbar_l)
    assert torch.equal(keep, keep_f) and torch.equal(fused, fused_f) and torch.equal(prio, prio_f)
    assert torch.equal(fused, fused_p) and torch.equal(prio, prio_p)
    assert torch.equal(keep, keep_p)

    e, r, rho, pbar, mass = (x.cpu().numpy() for x in (e, r, rho, pbar, mass))
    fused, conflict, prio = (x.cpu().numpy() for x in (fused, conflict, prio))
    keep, adj, rep = keep.cpu().numpy(), adj.cpu().numpy(), rep.cpu().numpy()
    check_keep_wellformed(keep, gh * gw, K)
    refs = oracle_images(cfg, q, k, range(cfg.batch), mode)
    for b, ref in enumerate(refs):
        log(f"  image {b}")
        # score stage vs oracle from Q, K
        _errs("r", r[b], ref.r, 1e-9, 2e-4)
        _errs("e", e[b], ref.p - 0.5, 1e-6, 2e-4)
        # evidence stages on the GPU's own supports
        p_gpu = 0.5 + e[b].astype(np.float64)
        rho_o, pbar_o = O.head_reliability(p_gpu)
        _errs("rho", rho[b], rho_o, 1e-7, 2e-5)
        _errs("pbar_c", pbar[b], pbar_o - 0.5, 1e-7, 2e-5)
        m_o = O.head_masses(rho_o, pbar_o)
        _errs("mass", mass[b], m_o, 1e-7, 2e-5)
        f_o, k_o, pl_o, q_o, _ = O.ds_combine_layers(mass[b].astype(np.float64))
        _errs("fused", fused[b], f_o, 1e-7, 2e-5)
        _errs("conflict", conflict[b], k_o, 1e-7, 2e-5)
        # float32 masses sum to 1 only within rounding, so on these inputs the two
        # forms of Eq. 18 differ by that rounding; compare with 1 - Pl = m~(U)
        _errs("prio_c", prio[b], f_o[:, 1] * (1.0 - k_o[-1]), 1e-9, 2e-5)
        # selection on the GPU's own priorities with the float32 lambda the kernel
        # received: bit-exact decisions
        sel_keep, sel_qt, sel_b = O.spatial_select(1.0 - prio[b].astype(np.float64), gh, gw, G,
                                                   F32(lam), K)
        np.testing.assert_array_equal(rep[b], sel_b)
        assert keep[b].tolist() == sel_keep.tolist()
        _errs("adj_c", adj[b], 1.0 - sel_qt, 1e-15, 1e-12)
        # end to end
        err = assert_mass_bar(fused[b], ref.fused, "fused e2e")
        log(f"    fused e2e  max|d|={err:.3e}")
        _errs("c e2e", prio[b], 1.0 - ref.q, 1e-7, 2e-3)
        cmp = compare_sets(keep[b], ref, geom=SelectGeom(gh, gw, G, lam))
        log(f"    set: {cmp.verdict} swaps={cmp.swaps} near-boundary={cmp.near_boundary}")
        assert cmp.verdict != "fail"


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("cfg", CASES, ids=[c.name for c in CASES])
def test_stage_parity(cfg, mode):
    _run_case(cfg, mode)


def test_heavy_tailed_salient_tokens_surface():
    """With high-contrast inputs the salient keys are the ones kept."""
    cfg = synth.heavy_tailed(synth.config_by_name("llava").replace(batch=2))
    q, k, sal = synth.gen_batch(cfg)
    idx, _, _ = E.prune(to_device(q, "bf16"), to_device(k, "bf16"), 24, 24, cfg.keep, 4, 0.1)
    idx = idx.cpu().numpy()
    for b in range(cfg.batch):
        frac = np.isin(sal[b], idx[b]).mean()
        log(f"  image {b}: {frac:.2%} of salient tokens kept")
        assert frac >= 0.9


def test_identical_keys_closed_form():
    """All keys identical: e = 0 exactly, rho = 0, m = (0, 0, 1), c = 0; the kept set is
    each cell's lowest-index token, then the lowest remaining indices."""
    cfg = _small("identical", config_id=57, batch=1, grid_h=8, grid_w=8, keep=20)
    q, k, _ = synth.gen_batch(cfg)
    k[:] = k[:, :, :, :1, :]
    for mode in MODES:
        idx, fused, prio = E.prune(to_device(q, "bf16"), to_device(k, "bf16"), 8, 8, 20, 4, 0.3,
                                   mode, want_fused=True, want_prio=True)
        e, _ = E.score_heads(to_device(q, "bf16"), to_device(k, "bf16"), 8, 8, mode)
        assert (e == 0).all()
        assert (prio == 0).all()
        assert torch.equal(fused.cpu(), torch.tensor([0.0, 0.0, 1.0]).expand(1, 64, 3))
        reps = sorted(16 * i + 2 * j for i in range(4) for j in range(4))
        rest = [n for n in range(64) if n not in reps][:4]
        assert idx[0].cpu().tolist() == sorted(reps + rest)


def test_total_conflict_through_ds_stage():
    """(1,0,0) then (0,1,0): K = 1, the fused mass is vacuous and c = 0 (q = 1)."""
    m = torch.tensor([[[[1.0, 0.0, 0.0]], [[0.0, 1.0, 0.0]], [[0.2, 0.3, 0.5]]]],
                     device="cuda")                              # [B=1, L=3, N=1, 3]
    fused, conflict, prio = E.ds_combine_layers(m.contiguous(), 1, 1)
    torch.cuda.synchronize()
    assert conflict[0, :, 0].cpu().tolist() == [0.0, 1.0, 0.0]
    np.testing.assert_allclose(fused[0, 0].cpu().numpy(), [0.2, 0.3, 0.5], rtol=1e-7)
    f_o, k_o, _, q_o, _ = O.ds_combine_layers(m[0].double().cpu().numpy())
    np.testing.assert_allclose(prio[0].cpu().numpy(), 1 - q_o, atol=1e-7)
    m2 = m[:, :2].contiguous()
    fused2, _, prio2 = E.ds_combine_layers(m2, 1, 1)
    assert fused2[0, 0].cpu().tolist() == [0.0, 0.0, 1.0] and prio2.item() == 0.0


@pytest.mark.parametrize("keep", [0, 1, 64])
@pytest.mark.parametrize("cells", [1, 8])
@pytest.mark.parametrize("lam", [0.0, 1.0])
def test_selection_edges(keep, cells, lam):
    """K = 0 and K = N, one cell and one token per cell, lambda at both ends;
    exact ties in c."""
    rng = np.random.default_rng(keep * 31 + cells)
    c = (rng.integers(0, 6, size=(3, 64)) / 8.0).astype(np.float32)
    cd = torch.from_numpy(c).cuda()
    idx, adj, rep = E.spatial_select(cd, 8, 8, keep, cells, lam, want_adj=True, want_rep=True)
    torch.cuda.synchronize()
    for b in range(3):
        ok, qt, bb = O.spatial_select(1.0 - c[b].astype(np.float64), 8, 8, cells, F32(lam), keep)
        assert idx[b].cpu().tolist() == ok.tolist()
        np.testing.assert_array_equal(rep[b].cpu().numpy(), bb)


@pytest.mark.parametrize("grid", [(1, 1), (7, 9), (8, 8), (5, 13), (31, 33), (32, 32), (25, 41)])
def test_selection_workgroup_sizes(grid):
    """1, 63, 64, 65, 1023, 1024 and 1025 tokens: the selection kernels run with one
    thread per token in whole waves up to 1024 tokens and with 1024 threads (two
    tokens per thread) above; kept sets and representatives equal the oracle's,
    with exact ties in c."""
    gh, gw = grid
    n = gh * gw
    rng = np.random.default_rng(n)
    c = (rng.integers(0, 9, size=(2, n)) / 16.0).astype(np.float32)
    cd = torch.from_numpy(c).cuda()
    cells = min(4, gh, gw)
    for keep in sorted({0, 1, n // 3, n}):
        idx, _, rep = E.spatial_select(cd, gh, gw, keep, cells, 0.25, want_rep=True)
        torch.cuda.synchronize()
        for b in range(2):
            ok, _, bb = O.spatial_select(1.0 - c[b].astype(np.float64), gh, gw, cells,
                                         F32(0.25), keep)
            assert idx[b].cpu().tolist() == ok.tolist(), (grid, keep, b)
            np.testing.assert_array_equal(rep[b].cpu().numpy(), bb)


def test_determinism_and_stream():
    """Two runs give identical bits; a call on a side stream matches the default stream."""
    cfg = synth.config_by_name("llava").replace(batch=3)
    q, k, _ = synth.gen_batch(cfg)
    qd, kd = to_device(q, "bf16"), to_device(k, "bf16")
    a = E.prune(qd, kd, 24, 24, 128, want_fused=True, want_prio=True)
    b = E.prune(qd, kd, 24, 24, 128, want_fused=True, want_prio=True)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        c = E.prune(qd, kd, 24, 24, 128, want_fused=True, want_prio=True)
    s.synchronize()
    torch.cuda.synchronize()
    for x, y, z in zip(a, b, c):
        assert torch.equal(x, y) and torch.equal(x, z)


def test_binding_errors_on_gpu_tensors():
    q = torch.zeros((1, 1, 2, 3, 96), device="cuda", dtype=torch.bfloat16)
    k = torch.zeros((1, 1, 2, 4, 96), device="cuda", dtype=torch.bfloat16)
    with pytest.raises(E.E2SError) as ei:
        E.score_heads(q, k, 2, 2)
    assert ei.value.status == 4            # head_dim 96 unsupported
    with pytest.raises(TypeError):
        E.score_heads(q, k.float(), 2, 2)
