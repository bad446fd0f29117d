"""e2s_prune_noalloc (the workspace in the library's static scratch) through the C
ABI: the same bits as e2s_prune with a caller workspace, and the oracle's results
under the parity rule (fused masses within 1e-4 absolute and 1e-7 + 2e-3 |ref|,
kept sets exact or tie-excused), on calls in a row that shrink:
  1. 64 LLaVA-1.5-7B-shaped images (one workgroup per image and layer, 20 MB of
     scratch), mean-of-logits reading;
  2. one 64 x 64 high-resolution image (supports in the scratch, and the fusion
     run device-wide in its support region), mean-of-logits reading;
  3. two Qwen2-VL-7B-shaped images (grouped-query heads), mean-of-probabilities
     reading.
The scratch keeps each call's contents, so a kernel that read a stale byte of the
previous, larger call would show here as a difference from e2s_prune.
"""
import ctypes

import pytest

import oracle as O
import synth
from _helpers import assert_mass_bar, compare_sets, log, to_device

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
E = pytest.importorskip("paper_2608_23253_amd")
from paper_2608_23253_amd import _lib as L  # noqa: E402

CALLS = [("llava", 64, "mean_logit"), ("hires", 1, "mean_logit"), ("qwen2vl_gqa", 2, "mean_prob"),
         ("llava", 2, "mean_prob")]


def _noalloc_raw(qd, kd, cfg, mode):
    """One e2s_prune_noalloc call on the raw C symbol; outputs allocated by the caller."""
    B, N = cfg.batch, cfg.num_visual
    sh = L.shape_from(qd, kd, cfg.grid_h, cfg.grid_w)
    pa = L.make_params(L._dtype_code(qd), mode, 0.0, cfg.cells, cfg.lam, cfg.keep)
    keep = torch.full((B, cfg.keep), -1, device="cuda", dtype=torch.int32)
    fused = torch.full((B, N, 3), float("nan"), device="cuda")
    prio = torch.full((B, N), float("nan"), device="cuda")
    st = torch.cuda.current_stream().cuda_stream
    rc = L.lib().e2s_prune_noalloc(ctypes.byref(sh), ctypes.byref(pa), qd.data_ptr(),
                                   kd.data_ptr(), keep.data_ptr(), fused.data_ptr(),
                                   prio.data_ptr(), st)
    assert rc == L.OK, L.lib().e2s_status_string(rc).decode()
    return keep, fused, prio


def test_noalloc_matches_prune_and_oracle_on_shrinking_calls():
    for name, batch, mode in CALLS:
        cfg = synth.config_by_name(name).replace(batch=batch)
        q, k, _ = synth.gen_batch(cfg)
        qd, kd = to_device(q, cfg.dtype), to_device(k, cfg.dtype)
        ws = L.workspace_size(L.shape_from(qd, kd, cfg.grid_h, cfg.grid_w), L.make_params())
        log(f"[noalloc] {name} B={batch} mode={mode} workspace {ws / 2**20:.1f} MiB")
        keep, fused, prio = _noalloc_raw(qd, kd, cfg, mode)
        r_keep, r_fused, r_prio = E.prune(qd, kd, cfg.grid_h, cfg.grid_w, cfg.keep, cfg.cells,
                                          cfg.lam, mode, want_fused=True, want_prio=True)
        torch.cuda.synchronize()
        assert torch.equal(keep, r_keep), f"{name}: kept sets differ from e2s_prune"
        assert torch.equal(fused, r_fused), f"{name}: fused masses differ from e2s_prune"
        assert torch.equal(prio, r_prio), f"{name}: priorities differ from e2s_prune"
        keep_h, fused_h = keep.cpu().numpy(), fused.cpu().numpy()
        counts = {}
        worst = 0.0
        for b in range(batch):
            ref = O.prune_image(q[b], k[b], cfg.grid_h, cfg.grid_w, cfg.keep, cfg.cells,
                                cfg.lam, mode)
            worst = max(worst, assert_mass_bar(fused_h[b], ref.fused, f"{name} image {b}"))
            cmp = compare_sets(keep_h[b], ref)
            counts[cmp.verdict] = counts.get(cmp.verdict, 0) + 1
            assert cmp.verdict != "fail", f"{name} image {b}: kept set"
        log(f"  equal to e2s_prune; oracle: max|d fused|={worst:.2e}, sets {counts}")


def test_noalloc_rejects_oversize_before_launch():
    """256 LLaVA-shaped images need 80 MB of workspace: refused, nothing enqueued."""
    cfg = synth.config_by_name("llava").replace(batch=2)
    q, k, _ = synth.gen_batch(cfg)
    qd, kd = to_device(q, cfg.dtype), to_device(k, cfg.dtype)
    sh = L.make_shape(256, cfg.num_layers, cfg.num_heads, cfg.num_kv_heads, cfg.head_dim,
                      cfg.num_text, cfg.grid_h, cfg.grid_w)
    pa = L.make_params(L.DTYPE_BF16, "mean_logit", 0.0, cfg.cells, cfg.lam, cfg.keep)
    keep = torch.empty((2, cfg.keep), device="cuda", dtype=torch.int32)
    rc = L.lib().e2s_prune_noalloc(ctypes.byref(sh), ctypes.byref(pa), qd.data_ptr(),
                                   kd.data_ptr(), keep.data_ptr(), None, None,
                                   torch.cuda.current_stream().cuda_stream)
    assert rc == L.ERR_SCRATCH_TOO_SMALL
