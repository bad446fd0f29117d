"""e2s_prune captured in a HIP graph (torch.cuda.CUDAGraph) and replayed.

Serving loops capture their launch-bound steps.  The library launches only
kernels on the caller's stream (no allocation, no memset, no host synchronisation),
so a captured e2s_prune must replay with the eager call's exact results.  Each
case replays the graph several times with eager work and synchronisations in
between, on fresh inputs copied into the captured buffers, and checks every replay
against an eager call on the same inputs.
"""
import pytest

import synth
from _helpers import log, to_device

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
E = pytest.importorskip("paper_2608_23253_amd")


def _cfg(name, **kw):
    base = dict(name=name, config_id=95, batch=3, num_layers=2, num_heads=4, num_kv_heads=2,
                head_dim=128, num_text=7, grid_h=9, grid_w=10, keep=20, lambdas=(0.1,),
                dtype="bf16", salient_count=4, clusters=0, shift_sigmas=2.0)
    base.update(kw)
    return synth.Config(**base)


CASES = [
    (_cfg("gqa_d128"), "mean_logit"),
    (_cfg("mha_layer_path", config_id=96, batch=64, num_layers=4, num_heads=6, num_kv_heads=6,
          num_text=12), "mean_logit"),
    (_cfg("gqa_prob", config_id=97), "mean_prob"),
    # 456 tokens, 40 queries: the register-resident mean-of-probabilities kernel
    (_cfg("resident_prob", config_id=98, num_text=40, grid_h=19, grid_w=24, keep=60),
     "mean_prob"),
]


@pytest.mark.parametrize("cfg,mode", CASES, ids=[c.name for c, _ in CASES])
def test_captured_prune_replays_exactly(cfg, mode):
    log(f"[case] graph {cfg.name} mode={mode}")
    gh, gw, K, G, lam = cfg.grid_h, cfg.grid_w, cfg.keep, cfg.cells, cfg.lam
    inputs = []
    for s in range(3):
        q, k, _ = synth.gen_batch(cfg.replace(config_id=cfg.config_id * 10 + s))
        inputs.append((to_device(q, cfg.dtype), to_device(k, cfg.dtype)))
    q_buf, k_buf = inputs[0][0].clone(), inputs[0][1].clone()
    pr = E.Pruner(q_buf, k_buf, gh, gw, K, G, lam, mode)
    fused = torch.empty((cfg.batch, gh * gw, 3), device="cuda", dtype=torch.float32)
    prio = torch.empty((cfg.batch, gh * gw), device="cuda", dtype=torch.float32)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):          # warm-up (kernel attributes) off the capture
        pr(q_buf, k_buf, fused, prio)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()

    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        pr(q_buf, k_buf, fused, prio)
    torch.cuda.synchronize()

    for rep in range(6):
        qd, kd = inputs[rep % 3]
        q_buf.copy_(qd)
        k_buf.copy_(kd)
        graph.replay()
        torch.cuda.synchronize()
        got = (pr.keep_idx.clone(), fused.clone(), prio.clone())
        ref_keep, ref_fused, ref_prio = E.prune(qd, kd, gh, gw, K, G, lam, mode, want_fused=True,
                                                want_prio=True)
        torch.cuda.synchronize()
        assert torch.equal(got[0], ref_keep), f"replay {rep}: kept indices"
        assert torch.equal(got[1], ref_fused) and torch.equal(got[2], ref_prio), \
            f"replay {rep}: masses"
