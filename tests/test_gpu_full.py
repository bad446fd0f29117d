"""Full-size workloads through e2s_prune in the launch configuration the benchmark
times (whole batch, one call), every image compared with the CPU oracle.

For every image of every workload, in both readings:
  * fused masses: max |d m~| <= 1e-4 absolute AND |d| <= 1e-7 + 2e-3 |ref| per
    element (Eq. 12-16);
  * c = 1 - q within 2e-3 relative (Eq. 19);
  * the kept set exact, tie-excused (every differing token's oracle q~ within 1e-5
    of the oracle's K-th kept score) or a representative flip (a cell whose two
    best tokens' oracle q lie within 1e-5: the novelty bonus of Eq. 20-22 may sit
    on either); no failure (Eq. 23);
  * the staged selection on the GPU's own priorities equals the oracle's
    selection of the same float32 values bit for bit (Eq. 20-23 decided in the
    same precision on both sides).
The novelty-weight sweep of the aggressive workload reruns the selection on the
fused priorities for every lambda, against the oracle's selection of its own q.
Per workload, reading and lambda, one `[parity]` JSON line records the image
count, max |d m~| and the exact / tie / rep_flip / fail counts with the swaps.

Workloads: LLaVA-1.5-7B-shaped (64 images, K = 128), the aggressive variant
(256 images, K = 64, lambda in {0, 0.25, 0.5, 1}), Qwen2-VL-7B-shaped GQA
(28 query heads over 4 key heads, 32 x 32 grid, 32 images, K = 256) and the
64 x 64 high-resolution stress case with near-duplicate keys (16 images, K = 512).
"""
import dataclasses
import json
import time

import numpy as np
import pytest

import oracle as O
import synth
from _helpers import (SelectGeom, check_keep_wellformed, compare_sets, log, mass_errors,
                      MASS_ATOL, to_device)

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
E = pytest.importorskip("paper_2608_23253_amd")

MODES = ["mean_logit", "mean_prob"]
WORKLOADS = ["llava", "llava_aggressive", "qwen2vl_gqa", "hires"]

_cache = {}


def F32(x):
    """The value a float parameter has after crossing the C ABI."""
    return float(np.float32(x))


def _batch(name):
    if name not in _cache:
        _cache.clear()
        cfg = synth.config_by_name(name)
        t = time.time()
        q, k, sal = synth.gen_batch(cfg)
        log(f"[gen] {name}: {cfg.batch} images in {time.time() - t:.1f}s")
        _cache[name] = (cfg, q, k, to_device(q, cfg.dtype), to_device(k, cfg.dtype))
    return _cache[name]


class Tally:
    def __init__(self, name, mode, lam, n_images):
        self.rec = {"workload": name, "mode": mode, "lambda": lam, "images": n_images,
                    "max_abs_dfused": 0.0, "exact": 0, "tie": 0, "rep_flip": 0, "fail": 0,
                    "swaps": 0, "near_boundary_max": 0}

    def add(self, cmp, abs_err=None):
        self.rec[cmp.verdict] += 1
        self.rec["swaps"] += cmp.swaps
        self.rec["near_boundary_max"] = max(self.rec["near_boundary_max"], cmp.near_boundary)
        if abs_err is not None:
            self.rec["max_abs_dfused"] = max(self.rec["max_abs_dfused"], abs_err)

    def emit(self):
        log("[parity] " + json.dumps(self.rec))
        return self.rec


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("name", WORKLOADS)
def test_full_size(name, mode):
    cfg, q, k, qd, kd = _batch(name)
    B, N, gh, gw, G, K = cfg.batch, cfg.num_visual, cfg.grid_h, cfg.grid_w, cfg.cells, cfg.keep
    log(f"[full] {name} mode={mode} B={B} N={N} K={K} lambdas={cfg.lambdas}")
    pr = E.Pruner(qd, kd, gh, gw, K, G, cfg.lam, mode)
    fused = torch.empty((B, N, 3), device="cuda")
    prio = torch.empty((B, N), device="cuda")
    idx = pr(qd, kd, fused, prio).clone()
    torch.cuda.synchronize()
    f = fused.cpu().numpy()
    c = prio.cpu().numpy()
    kept = idx.cpu().numpy()
    # properties on every image
    check_keep_wellformed(kept, N, K)
    assert (f >= -1e-7).all() and np.abs(f.sum(-1) - 1).max() < 1e-5
    assert (c >= 0).all() and (c <= 1).all()
    # the staged selection agrees with the fused call on every image
    sel, _, _ = E.spatial_select(prio, gh, gw, K, G, cfg.lam)
    assert torch.equal(sel, idx)

    # every image against the oracle
    t0 = time.time()
    tally = Tally(name, mode, cfg.lam, B)
    refs = []
    for b in range(B):
        ref = O.prune_image(q[b], k[b], gh, gw, K, G, cfg.lam, mode)
        refs.append(ref)
        abs_err, rel_worst = mass_errors(f[b], ref.fused)
        cerr = np.abs(c[b] - (1 - ref.q)) / np.maximum(1 - ref.q, 1e-30)
        cmp = compare_sets(kept[b], ref, geom=SelectGeom(gh, gw, G, cfg.lam))
        tally.add(cmp, abs_err)
        if cmp.verdict != "exact" or b in (0, B - 1):
            log(f"  image {b}: max|d fused|={abs_err:.2e} (rel/bound {rel_worst:.3f}), "
                f"max rel d c={cerr.max():.2e}, set {cmp.verdict} swaps={cmp.swaps} "
                f"near-boundary={cmp.near_boundary}")
        assert abs_err <= MASS_ATOL, f"image {b}: max |d fused| {abs_err:.3e}"
        assert rel_worst <= 1.0, f"image {b}: fused masses outside the relative bound"
        assert cerr.max() <= 2e-3, f"image {b}: c"
        # selection of the GPU's own priorities: the same decisions bit for bit
        ok, _, _ = O.spatial_select(1.0 - c[b].astype(np.float64), gh, gw, G, F32(cfg.lam), K)
        assert kept[b].tolist() == ok.tolist(), f"image {b}: selection of equal priorities"
    rec = tally.emit()
    log(f"  oracle over {B} images in {time.time() - t0:.1f}s")
    assert rec["fail"] == 0

    # the novelty-weight sweep reuses the fused priorities
    for lam in cfg.lambdas[1:]:
        sel, _, _ = E.spatial_select(prio, gh, gw, K, G, lam)
        sel = sel.cpu().numpy()
        check_keep_wellformed(sel, N, K)
        tally = Tally(name, mode, lam, B)
        for b in range(B):
            ok, _, _ = O.spatial_select(1.0 - c[b].astype(np.float64), gh, gw, G, F32(lam), K)
            assert sel[b].tolist() == ok.tolist(), f"lambda={lam} image {b}: equal priorities"
            o_keep, o_qt, o_b = O.spatial_select(refs[b].q, gh, gw, G, lam, K)
            ref_l = dataclasses.replace(refs[b], keep=o_keep, qt=o_qt, is_rep=o_b)
            cmp = compare_sets(sel[b], ref_l, geom=SelectGeom(gh, gw, G, lam))
            tally.add(cmp)
            if cmp.verdict != "exact":
                log(f"  lambda={lam} image {b}: set {cmp.verdict} swaps={cmp.swaps}")
        assert tally.emit()["fail"] == 0
