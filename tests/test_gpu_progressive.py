"""GPU parity of the progressive schedule (Algorithm 1 with shrinking candidate
sets; Sec. 5.1 schedules) through e2s_prune_stage.

Operation s uses source layer s of a seeded batch; its candidates' keys are the
rows of that layer's keys at the survivors' positions (what the model would
compute for the pruned sequence).  Each operation is checked against the oracle's
prune_stage fed the GPU's own candidates and carried masses (isolating the
operation), with the kept set exact or tie-excused and the carried masses within
the fused-mass bar; the no-early-pruning schedule must equal e2s_prune bit for
bit."""
import numpy as np
import pytest

import oracle as O
import synth
from _helpers import compare_sets, log, to_device

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
E = pytest.importorskip("paper_2608_23253_amd")


def _cfg(name, **kw):
    base = dict(name=name, config_id=70, batch=2, num_layers=3, num_heads=4, num_kv_heads=4,
                head_dim=64, num_text=8, grid_h=8, grid_w=8, keep=5, lambdas=(0.1,),
                dtype="bf16", salient_count=6, clusters=2, shift_sigmas=2.0)
    base.update(kw)
    return synth.Config(**base)


CASES = [
    (_cfg("small_3ops"), [30, 12, 5]),
    (_cfg("gqa_d128", config_id=71, num_heads=8, num_kv_heads=2, head_dim=128, grid_h=9,
          grid_w=11, num_text=6), [40, 17, 9]),
    (synth.config_by_name("llava").replace(batch=2, num_layers=3), [122, 48, 42]),
    (synth.config_by_name("llava").replace(batch=2, num_layers=3), [20, 8, 0]),
    # 24000 tokens, then 18000 candidates: selections in segments, with candidate
    # positions and carried masses
    (_cfg("large_grid", config_id=72, batch=1, num_heads=2, num_kv_heads=2, grid_h=150,
          grid_w=160, num_text=4, salient_count=50, clusters=3), [18000, 5000, 900]),
]


def _gather_keys(k_layer, pos):
    """Rows of k_layer [B, Hkv, N, d] at the candidate positions pos [B, N_l]."""
    return torch.stack([k_layer[b][:, pos[b].long(), :] for b in range(k_layer.shape[0])])


def _run(cfg, budgets, mode):
    gh, gw, G, lam = cfg.grid_h, cfg.grid_w, cfg.cells, cfg.lam
    q, k, _ = synth.gen_batch(cfg)
    qd, kd = to_device(q, cfg.dtype), to_device(k, cfg.dtype)
    B, N = cfg.batch, gh * gw
    pos = None
    m_prev = None
    results = []
    for s, budget in enumerate(budgets):
        k_c = (kd[:, s] if pos is None else _gather_keys(kd[:, s], pos)).unsqueeze(1).contiguous()
        q_s = qd[:, s:s + 1].contiguous()
        sp = E.StagePruner(q_s, k_c, gh, gw, budget, G, lam, mode)
        idx, kpos, m_out = sp(q_s, k_c, pos, m_prev)
        torch.cuda.synchronize()
        results.append((None if pos is None else pos.cpu().numpy(),
                        None if m_prev is None else m_prev.cpu().numpy(),
                        idx.cpu().numpy().copy(), kpos.cpu().numpy().copy(),
                        m_out.cpu().numpy().copy()))
        pos = kpos.clone()
        m_prev = m_out.clone()
    return q, k, results


@pytest.mark.parametrize("mode", ["mean_logit", "mean_prob"])
@pytest.mark.parametrize("case", CASES, ids=[f"{c.name}-{'-'.join(map(str, b))}" for c, b in CASES])
def test_progressive_operations(case, mode):
    cfg, budgets = case
    log(f"[case] {cfg.name} budgets={budgets} mode={mode}")
    gh, gw, G = cfg.grid_h, cfg.grid_w, cfg.cells
    lam32 = float(np.float32(cfg.lam))
    q, k, results = _run(cfg, budgets, mode)
    N = gh * gw
    for s, (pos, m_prev, idx, kpos, m_out) in enumerate(results):
        K = budgets[s]
        for b in range(cfg.batch):
            cand = np.arange(N) if pos is None else pos[b].astype(np.int64)
            assert (np.diff(cand) > 0).all()
            ref = O.prune_stage(q[b, s:s + 1], k[b, s:s + 1][:, :, cand, :], cand, gh, gw, K, G,
                                lam32, mode, None,
                                None if m_prev is None else m_prev[b].astype(np.float64))
            cmp = compare_sets(idx[b], ref)
            log(f"  op {s} image {b}: N_l={cand.size} K={K} {cmp.verdict} swaps={cmp.swaps} "
                f"near={cmp.near_boundary}")
            assert cmp.verdict != "fail"
            np.testing.assert_array_equal(kpos[b], cand[idx[b]])
            if cmp.verdict == "exact" and K:
                err = np.abs(m_out[b] - ref.m_out)
                assert (err <= 1e-4).all() and (err <= 1e-7 + 2e-3 * np.abs(ref.m_out)).all()


def test_no_early_pruning_equals_one_shot():
    """Budgets N, N, K reproduce e2s_prune over the three layers bit for bit."""
    cfg = _cfg("one_shot_equiv", config_id=72)
    gh, gw, N = cfg.grid_h, cfg.grid_w, cfg.grid_h * cfg.grid_w
    q, k, results = _run(cfg, [N, N, 9], "mean_logit")
    qd, kd = to_device(q, cfg.dtype), to_device(k, cfg.dtype)
    keep, fused, _ = E.prune(qd, kd, gh, gw, 9, cfg.cells, cfg.lam, want_fused=True)
    torch.cuda.synchronize()
    assert np.array_equal(results[-1][2], keep.cpu().numpy())
    f = fused.cpu().numpy()
    for b in range(cfg.batch):
        np.testing.assert_array_equal(results[-1][4][b], f[b][keep.cpu().numpy()[b]])


def test_first_operation_equals_prune_on_one_layer():
    cfg = _cfg("first_op", config_id=73)
    gh, gw = cfg.grid_h, cfg.grid_w
    q, k, _ = synth.gen_batch(cfg)
    qd, kd = to_device(q, cfg.dtype), to_device(k, cfg.dtype)
    idx, _, _ = E.prune_stage(qd[:, :1].contiguous(), kd[:, :1].contiguous(), gh, gw, 11,
                              cells=cfg.cells, lam=cfg.lam)
    keep, _, _ = E.prune(qd[:, :1].contiguous(), kd[:, :1].contiguous(), gh, gw, 11, cfg.cells,
                         cfg.lam)
    torch.cuda.synchronize()
    assert torch.equal(idx, keep)


def test_positions_outside_the_grid_get_no_cell():
    """A candidate position outside the grid is ranked without a cell (no bonus)
    and never indexes out of bounds; the rest of the selection is unaffected."""
    cfg = _cfg("bad_pos", config_id=74, batch=1)
    gh, gw = cfg.grid_h, cfg.grid_w
    q, k, _ = synth.gen_batch(cfg)
    qd, kd = to_device(q, cfg.dtype), to_device(k, cfg.dtype)
    pos = torch.arange(0, 64, 2, device="cuda", dtype=torch.int32)[None]     # 32 candidates
    k_c = _gather_keys(kd[:, 0], pos).unsqueeze(1).contiguous()
    q0 = qd[:, :1].contiguous()
    good, _, _ = E.prune_stage(q0, k_c, gh, gw, 8, cand_pos=pos, cells=4, lam=0.0)
    bad = pos.clone()
    bad[0, 5] = 10_000
    bad[0, 6] = -3
    worse, wpos, _ = E.prune_stage(q0, k_c, gh, gw, 8, cand_pos=bad, cells=4, lam=0.0)
    torch.cuda.synchronize()
    # lambda = 0: cells do not enter the ranking, so the kept indices agree
    assert torch.equal(good, worse)
