"""Concurrent e2s_prune calls on two streams.

The C ABI lets calls run concurrently when they share no workspace and no output
(every call only enqueues kernels on its own stream).  Two Pruners, each with its
own workspace and outputs, alternate steps over different batches on two side
streams (as a serving loop with two batches in flight does), so the kernels of
neighbouring steps overlap on the device; every step's kept indices, fused masses
and priorities must equal those of the same batch run alone.
"""
import pytest

import synth
from _helpers import log, to_device

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
E = pytest.importorskip("paper_2608_23253_amd")


def _cfg(name, **kw):
    base = dict(name=name, config_id=110, batch=16, num_layers=4, num_heads=8, num_kv_heads=8,
                head_dim=128, num_text=24, grid_h=12, grid_w=12, keep=30, lambdas=(0.1,),
                dtype="bf16", salient_count=6, clusters=2, shift_sigmas=1.5)
    base.update(kw)
    return synth.Config(**base)


CASES = [
    (_cfg("mha_layer_path", batch=64), "mean_logit"),
    (_cfg("gqa_staged", config_id=111, num_heads=12, num_kv_heads=3), "mean_logit"),
    (_cfg("mha_prob", config_id=112), "mean_prob"),
    # 24 x 24 tokens, 64 queries: the register-resident mean-of-probabilities kernel
    (_cfg("resident_prob", config_id=113, num_text=64, grid_h=24, grid_w=24, keep=100),
     "mean_prob"),
]


@pytest.mark.parametrize("cfg,mode", CASES, ids=[c.name for c, _ in CASES])
def test_two_streams_match_sequential(cfg, mode):
    log(f"[case] two streams {cfg.name} mode={mode}")
    gh, gw, K, G, lam = cfg.grid_h, cfg.grid_w, cfg.keep, cfg.cells, cfg.lam
    B, N = cfg.batch, gh * gw
    batches = []
    for s in range(4):
        q, k, _ = synth.gen_batch(cfg.replace(config_id=cfg.config_id * 10 + s))
        batches.append((to_device(q, cfg.dtype), to_device(k, cfg.dtype)))
    # each batch alone, on the current stream
    ref = []
    for q, k in batches:
        idx, fused, prio = E.prune(q, k, gh, gw, K, G, lam, mode, want_fused=True,
                                   want_prio=True)
        ref.append((idx.clone(), fused, prio))
    torch.cuda.synchronize()

    prs = [E.Pruner(batches[0][0], batches[0][1], gh, gw, K, G, lam, mode) for _ in range(2)]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    outs = [(torch.empty((B, K), device="cuda", dtype=torch.int32),
             torch.empty((B, N, 3), device="cuda"), torch.empty((B, N), device="cuda"))
            for _ in batches]
    for s in streams:
        s.wait_stream(torch.cuda.current_stream())
    for rnd in range(3):
        for i, (q, k) in enumerate(batches):
            st = streams[i % 2]
            pr = prs[i % 2]
            with torch.cuda.stream(st):
                idx = pr(q, k, outs[i][1], outs[i][2], stream=st.cuda_stream)
                outs[i][0].copy_(idx)
        torch.cuda.synchronize()
        for i in range(len(batches)):
            assert torch.equal(outs[i][0], ref[i][0]), f"round {rnd} batch {i}: kept indices"
            assert torch.equal(outs[i][1], ref[i][1]), f"round {rnd} batch {i}: fused masses"
            assert torch.equal(outs[i][2], ref[i][2]), f"round {rnd} batch {i}: priorities"
    log(f"  {len(batches)} batches x 3 rounds on 2 streams: identical to sequential")
