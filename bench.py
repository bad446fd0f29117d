#!/usr/bin/env python3
"""Throughput of the E2S-Pruner scoring path (score + fuse + select) on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload llava] [--mode mean_logit]

One step is one e2s_prune call over the whole batch with Q and K already resident
in HBM: e2s_layer_reliability (score and head reliability, Eq. 1, 8-10) then
e2s_fuse_select (masses, fusion and selection, Eq. 11-23).  Prints ONE JSON line
with images/s, a roofline object for the dominant kernel (the score and
reliability stage, timed alone with HIP events on the launch stream), per-stage
times of the staged entry points, the ablation variants, the progressive
schedule, a ragged batch (e2s_prune_ragged on seeded dynamic-resolution images),
token compaction of the kept tokens (e2s_compact_tokens), the step rate with two
batches in flight on two streams (`pipelined`: a serving loop's rate; `value`
stays the one-stream rate) and the CPU oracle's throughput on a bounded sample,
with a parity summary of the step's results on the images the oracle processed.
`device` records the GPU and its achievable streaming-read bandwidth (e2s_read_probe
over the batch's keys), and `roofline.frac_of_measured_read` the dominant kernel's
rate against it as well as against the nominal 8 TB/s.

`configs` repeats the measurement for the other workloads and readings at their
full batches (the aggressive LLaVA workload for each lambda of its sweep): step
time and images/s, the two kernels of e2s_prune timed alone, the fraction of the
binding roofline (bf16 MFMA for the mean-of-probabilities reading where the
contraction outweighs the bytes), the selection tail's bytes and HBM fraction, and
the oracle on a few images of each, timed, with the parity summary of those images.

Other modes (used by the profiling commands kept with the results):
    --kernel-only   run only the timed e2s_prune steps (no CPU baseline)
    --copy-calibrate N_MIB   time a plain device copy of N MiB (counter calibration)
"""
from __future__ import annotations

import argparse
import ctypes
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "images pruned/sec (score+fuse+select) at LLaVA shape; % MFMA / % HBM peak"
HBM_PEAK_GBS = 8000.0
MFMA_BF16_PEAK_TFLOPS = 2500.0
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "layer_evidence_llava_traffic.txt")
# the sources of the score and reliability stage: a counter summary taken on other
# versions of them is not used
# The sources compiled into the kernel whose counters the traffic summary holds
# (layer_evidence_kernel: the score and reliability stage of the mean-of-logits
# reading at the LLaVA shape); the summary is used only while they are unchanged.
STAGE_SOURCES = ("layer.hip", "score_common.h", "batch_geom.h", "e2s_device.h", "e2s_kernels.h")
TRAFFIC_WORKLOAD = "llava"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawTextHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="llava")
    ap.add_argument("--mode", default="mean_logit", choices=["mean_logit", "mean_prob"])
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="minimum CPU time spent timing the oracle")
    ap.add_argument("--kernel-only", action="store_true")
    ap.add_argument("--no-extras", action="store_true",
                    help="skip the ablation-variant and progressive-schedule timings")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the other workloads and readings (the configs object)")
    ap.add_argument("--copy-calibrate", type=int, default=0, metavar="N_MIB")
    ap.add_argument("--hbm-probe", type=int, default=0, metavar="N_MIB",
                    help="time a streaming read (torch sum) of N MiB: a practical read ceiling")
    return ap.parse_args()


def source_digest() -> str:
    import hashlib
    h = hashlib.sha256()
    for name in STAGE_SOURCES:
        with open(os.path.join(ROOT, "paper_2608_23253_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def read_traffic(mode: str, workload: str):
    """HBM bytes per launch of the score and reliability stage from the committed
    counter summary, or None when it is missing, covers another workload or reading,
    or was taken on other sources."""
    if workload != TRAFFIC_WORKLOAD or not os.path.exists(TRAFFIC_FILE):
        return None
    vals = {}
    with open(TRAFFIC_FILE) as f:
        for line in f:
            if ":" in line and not line.startswith("#"):
                key, val = line.split(":", 1)
                vals[key.strip()] = val.strip()
    if vals.get("stage_source_sha256_16") != source_digest() or vals.get("mode") != mode:
        return None
    try:
        return float(vals["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def cpu_model() -> str:
    """The host CPU's model name (from /proc/cpuinfo), or "unknown"."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def copy_calibrate(mib: int):
    import torch
    n = mib * (1 << 20) // 4
    src = torch.ones(n, device="cuda", dtype=torch.float32)
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s.record()
    for _ in range(10):
        dst.copy_(src)
    e.record()
    torch.cuda.synchronize()
    ms = s.elapsed_time(e) / 10
    moved = 2 * n * 4
    print(json.dumps({"copy_mib": mib, "bytes_read": n * 4, "bytes_written": n * 4,
                      "ms": ms, "GBps": moved / ms / 1e6}))


def hbm_probe(mib: int):
    import torch
    n = mib * (1 << 20) // 4
    x = torch.ones(n, device="cuda", dtype=torch.float32)
    for _ in range(3):
        x.sum()
    torch.cuda.synchronize()
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s.record()
    for _ in range(10):
        x.sum()
    e.record()
    torch.cuda.synchronize()
    ms = s.elapsed_time(e) / 10
    print(json.dumps({"read_mib": mib, "ms": ms, "GBps": n * 4 / ms / 1e6}))


def avg_tokens(num_layers, n_visual, prune_after, kept):
    """Eq. 24: mean over the LLM layers of the visual tokens each layer processes."""
    total = 0
    for i in range(1, num_layers + 1):
        t = n_visual
        for a, k in zip(prune_after, kept):
            if i > a:
                t = k
        total += t
    return total / num_layers


# The paper's default LLaVA-1.5-7B schedule (Sec. 5.1): pruning after LLM layers 3,
# 17 and 22 of 32 keeps 122, 48 and 42 of the 576 visual tokens (AvgTokens 128).
SCHEDULE = (122, 48, 42)
PRUNE_AFTER = (3, 17, 22)


# the model whose attention shapes each workload has
SHAPES = {"tiny": "small fp32 test shape", "llava": "LLaVA-1.5-7B-shaped",
          "llava_aggressive": "LLaVA-1.5-7B-shaped", "qwen2vl_gqa": "Qwen2-VL-7B-shaped",
          "hires": "LLaVA-shaped at high resolution"}

# Inputs are cycled through copies totalling more than twice the 256 MiB Infinity
# Cache, so that no timed call finds its Q and K there from an earlier call.
CACHE_DEFEAT_BYTES = 2 * 256 * 2**20 + 1


def cache_sets(*tensors):
    """[tensors, copy 1, ...]: as many copies as needed to exceed CACHE_DEFEAT_BYTES."""
    nbytes = sum(t.numel() * t.element_size() for t in tensors)
    n = max(1, -(-CACHE_DEFEAT_BYTES // max(nbytes, 1)))
    return [tuple(tensors)] + [tuple(t.clone() for t in tensors) for _ in range(n - 1)]


class Cycle:
    """Round-robin over input sets; each call of next() gives the following set."""

    def __init__(self, sets):
        self.sets, self.i = sets, 0

    def next(self):
        s = self.sets[self.i % len(self.sets)]
        self.i += 1
        return s


def bench_variants_and_schedule(args, cfg, qd, kd, stream, timed):
    """Per-step time of every ablation variant through e2s_prune, and the
    progressive schedule as three e2s_prune_stage calls (operation s on source
    layer s of the batch; its candidates' keys gathered beforehand from that
    layer's keys, as the model would compute them for the pruned sequence)."""
    import numpy as np
    import torch
    import paper_2608_23253_amd as E

    B, gh, gw, N = cfg.batch, cfg.grid_h, cfg.grid_w, cfg.num_visual
    n_rep = max(20, args.steps // 4)
    variants = {}
    sets = Cycle(cache_sets(qd, kd))
    for v in E.VARIANTS:
        pr = E.Pruner(qd, kd, gh, gw, cfg.keep, cfg.cells, cfg.lam, args.mode, variant=v)
        for _ in range(args.warmup):
            pr(*sets.next())
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(n_rep):
            pr(*sets.next())
        torch.cuda.synchronize()
        ms = (time.perf_counter() - t0) * 1e3 / n_rep
        variants[v] = {"ms_per_step": round(ms, 4), "images_per_s": round(B / ms * 1e3, 1)}
    log("[bench] variants: " + ", ".join(f"{k} {v['ms_per_step']:.3f} ms"
                                         for k, v in variants.items()))

    # progressive schedule: prepare each operation's inputs with one untimed pass
    ops = []
    pos, m_prev = None, None
    for s, budget in enumerate(SCHEDULE):
        q_s = qd[:, s:s + 1].contiguous()
        if pos is None:
            k_s = kd[:, s:s + 1].contiguous()
        else:
            idx = pos.long()[:, None, :, None].expand(B, kd.shape[2], pos.shape[1], kd.shape[4])
            k_s = torch.gather(kd[:, s], 2, idx).unsqueeze(1).contiguous()
        sp = E.StagePruner(q_s, k_s, gh, gw, budget, cfg.cells, cfg.lam, args.mode)
        _, kpos, m_out = sp(q_s, k_s, pos, m_prev)
        torch.cuda.synchronize()
        ops.append((sp, Cycle(cache_sets(q_s, k_s)), None if pos is None else pos.clone(),
                    None if m_prev is None else m_prev.clone()))
        pos, m_prev = kpos.clone(), m_out.clone()
    calls = [(lambda o=o: (o[0](*o[1].next(), o[2], o[3]), 0)[1]) for o in ops]
    times = timed(calls, n_rep)
    op_us = [float(t.mean()) * 1e3 for t in times]
    total_us = sum(op_us)
    qk_bytes = sum(t.numel() * t.element_size() for o in ops for t in o[1].sets[0])
    prog = {
        "schedule": "->".join(str(x) for x in (N,) + SCHEDULE),
        "avg_tokens_eq24": avg_tokens(32, N, PRUNE_AFTER, SCHEDULE),
        "operation_us": [round(x, 2) for x in op_us],
        "images_per_s": round(B / (total_us * 1e-6), 1),
        "qk_bytes_per_batch": int(qk_bytes),
        "hbm_frac": round(qk_bytes / (total_us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
    }
    log(f"[bench] progressive {prog['schedule']}: {', '.join(f'{x:.1f}' for x in op_us)} us "
        f"-> {prog['images_per_s']:.0f} images/s")
    return {"variants": variants, "progressive": prog}


def bench_ragged(args, timed, name="qwen2vl_dynamic"):
    """e2s_prune_ragged over a seeded ragged batch (every image its own grid, text
    length and budget): images/s and the Q + K bytes read per second."""
    import numpy as np
    import torch
    import synth
    import paper_2608_23253_amd as E

    rc = synth.ragged_by_name(name)
    qs, ks, _, dims = synth.gen_ragged(rc)
    cfg = rc.base
    L_, H_, Hkv, D = cfg.num_layers, cfg.num_heads, cfg.num_kv_heads, cfg.head_dim
    arr, qtot, ktot, _, _ = E.packed_images(dims, L_, H_, Hkv, D)
    q = np.concatenate([x.reshape(-1) for x in qs])
    k = np.concatenate([x.reshape(-1) for x in ks])
    qd = torch.from_numpy(synth.to_bf16_bits(q).view(np.int16)).cuda().view(torch.bfloat16)
    kd = torch.from_numpy(synth.to_bf16_bits(k).view(np.int16)).cuda().view(torch.bfloat16)
    rp = E.RaggedPruner(arr, L_, H_, Hkv, D, qd.device, mode=args.mode, cells=cfg.cells,
                        lam=cfg.lam)
    n_rep = max(20, args.steps // 4)
    sets = Cycle(cache_sets(qd, kd))
    t = timed([lambda: (rp(*sets.next()), 0)[1]], n_rep)[0]
    us = float(t.mean()) * 1e3
    qk_bytes = (qtot + ktot) * 2
    n_tok = [gh * gw for gh, gw, _, _ in dims]
    out = {
        "workload": (f"{name}: {rc.batch} images, Qwen2-VL-7B-shaped heads ({H_} over {Hkv}, "
                     f"d {D}, {L_} layers), grids {rc.grid_sides[0]}..{rc.grid_sides[1]} per "
                     f"side ({min(n_tok)}..{max(n_tok)} tokens), {rc.num_text[0]}..."
                     f"{rc.num_text[1]} text queries, keep {rc.keep_frac:.1%}"),
        "us_per_batch": round(us, 2),
        "images_per_s": round(rc.batch / (us * 1e-6), 1),
        "qk_bytes_per_batch": int(qk_bytes),
        "hbm_frac": round(qk_bytes / (us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
    }
    log(f"[bench] ragged {name}: {us:.1f} us per batch -> {out['images_per_s']:.0f} images/s")
    return out


def bench_compaction(args, timed, kd, keep_idx):
    """e2s_compact_tokens after the step: the kept tokens' hidden states (LLaVA-1.5-7B
    width 4096, bf16) and the kept tokens' keys of the source layers (kd), with the
    kept indices of the step.  Bytes moved = 2 x the kept vectors (read + write)."""
    import torch
    import paper_2608_23253_amd as E

    B, L_, Hkv, N, D = kd.shape
    K = keep_idx.shape[1]
    hidden = torch.empty((B, 1, N, 4096), device=kd.device, dtype=torch.bfloat16).normal_()
    h_out = torch.empty((B, 1, K, 4096), device=kd.device, dtype=torch.bfloat16)
    kk = kd.reshape(B, L_ * Hkv, N, D)
    k_out = torch.empty((B, L_ * Hkv, K, D), device=kd.device, dtype=kd.dtype)
    n_rep = max(20, args.steps // 4)
    th, tk = timed([lambda: (E.compact_tokens(hidden, keep_idx, h_out), 0)[1],
                    lambda: (E.compact_tokens(kk, keep_idx, k_out), 0)[1]], n_rep)
    out = {}
    for name, t, o in (("hidden_states", th, h_out), ("source_layer_keys", tk, k_out)):
        us = float(t.mean()) * 1e3
        moved = 2 * o.numel() * o.element_size()
        out[name] = {"shape": list(o.shape), "us": round(us, 2), "bytes_moved": int(moved),
                     "GBps": round(moved / (us * 1e-6) / 1e9, 1),
                     "hbm_frac": round(moved / (us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4)}
    log("[bench] compaction: " + ", ".join(f"{k} {v['us']:.1f} us ({v['GBps']:.0f} GB/s)"
                                             for k, v in out.items()))
    return out


# The workloads and readings reported beside the headline one, each at its full
# batch, and how many images of each are compared with the oracle.
CONFIG_RUNS = (("llava", ("mean_prob",)),
               ("llava_aggressive", ("mean_logit", "mean_prob")),
               ("qwen2vl_gqa", ("mean_logit", "mean_prob")),
               ("hires", ("mean_logit", "mean_prob")))
PARITY_SAMPLE = {"llava": 8, "llava_aggressive": 8, "qwen2vl_gqa": 8, "hires": 2}


def roofline_floor_us(cfg, mode, batch):
    """Roofline time of one step: max(Q + K bytes / 8 TB/s, Eq. 1 flops / bf16 MFMA
    peak), the flops only for the mean-of-probabilities reading (the mean-of-logits
    reading hoists the query mean and streams the keys against one vector)."""
    hbm_us = batch * cfg.bytes_per_image() / (HBM_PEAK_GBS * 1e9) * 1e6
    if mode != "mean_prob":
        return hbm_us, "hbm", None
    flops = 2.0 * batch * cfg.num_layers * cfg.num_heads * cfg.num_text * cfg.num_visual \
        * cfg.head_dim
    mfma_us = flops / (MFMA_BF16_PEAK_TFLOPS * 1e12) * 1e6
    return max(hbm_us, mfma_us), ("mfma" if mfma_us > hbm_us else "hbm"), flops


def cpu_baseline_leg(cfg, mode, q_np, k_np, sample):
    """The CPU oracle on the sampled images: (images/s, threads used, its results)."""
    import oracle as O
    from threadpoolctl import threadpool_info, threadpool_limits
    threadpool_limits(len(os.sched_getaffinity(0)))
    used = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    t0 = time.perf_counter()
    refs = [O.prune_image(q_np[j], k_np[j], cfg.grid_h, cfg.grid_w, cfg.keep, cfg.cells,
                          cfg.lam, mode) for j in range(len(sample))]
    dt = time.perf_counter() - t0
    return len(sample) / dt, used, refs


def parity_summary(cfg, refs, sample, kept_by_lam, fused):
    """GPU results of the sampled images against the oracle's results `refs` (from the
    CPU-baseline leg): max |d m~| (first lambda's fused masses) and the exact / tie /
    rep_flip / fail counts of every lambda's kept sets, by the test suite's rule
    (tests/_helpers.compare_sets)."""
    import dataclasses
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    from _helpers import SelectGeom, compare_sets, mass_errors
    import oracle as O

    out = {"images": [int(b) for b in sample], "max_abs_dfused": 0.0, "by_lambda": {}}
    gh, gw, G, K = cfg.grid_h, cfg.grid_w, cfg.cells, cfg.keep
    for j, b in enumerate(sample):
        a, _ = mass_errors(fused[b], refs[j].fused)
        out["max_abs_dfused"] = max(out["max_abs_dfused"], a)
    for lam, kept in kept_by_lam.items():
        counts = {"exact": 0, "tie": 0, "rep_flip": 0, "fail": 0, "swaps": 0}
        for j, b in enumerate(sample):
            ref = refs[j]
            if lam != cfg.lam:
                o_keep, o_qt, o_b = O.spatial_select(ref.q, gh, gw, G, lam, K)
                ref = dataclasses.replace(ref, keep=o_keep, qt=o_qt, is_rep=o_b)
            cmp = compare_sets(kept[b], ref, geom=SelectGeom(gh, gw, G, lam))
            counts[cmp.verdict] += 1
            counts["swaps"] += cmp.swaps
        out["by_lambda"][str(lam)] = counts
    out["max_abs_dfused"] = float(f"{out['max_abs_dfused']:.3e}")
    return out


def make_timed(args):
    """timed(calls, n) on a given stream: per-call durations (ms) of each function in
    `calls`, run in order n times, from HIP events recorded on the launch stream
    between the calls (after args.warmup untimed rounds)."""
    import numpy as np
    import torch

    def on_stream(stream):
        def timed(calls, n):
            for _ in range(args.warmup):
                for c in calls:
                    c()
            torch.cuda.synchronize()
            ev = [[torch.cuda.Event(enable_timing=True) for _ in range(len(calls) + 1)]
                  for _ in range(n)]
            for i in range(n):
                ev[i][0].record(stream)
                for j, c in enumerate(calls):
                    rc = c()
                    if rc:
                        raise RuntimeError(f"{c.__name__} failed with status {rc}")
                    ev[i][j + 1].record(stream)
            torch.cuda.synchronize()
            return [np.array([ev[i][j].elapsed_time(ev[i][j + 1]) for i in range(n)])
                    for j in range(len(calls))]
        return timed
    return on_stream


def bench_configs(args, make_timed):
    """Every other workload at its full batch, both readings: wall-clock step time
    and images/s per lambda, the rate with two batches in flight (bench_pipelined,
    first lambda), the two kernels of e2s_prune timed alone with HIP events,
    the fraction of the binding roofline, the selection tail's bytes and HBM fraction,
    and a sampled parity summary against the oracle."""
    import numpy as np
    import torch
    import synth
    import paper_2608_23253_amd as E
    from paper_2608_23253_amd import _lib as L

    lib = L.lib()
    out = {}
    n_rep = max(20, args.steps // 4)
    for name, modes in CONFIG_RUNS:
        cfg = synth.config_by_name(name)
        B, N, L_, gh, gw = cfg.batch, cfg.num_visual, cfg.num_layers, cfg.grid_h, cfg.grid_w
        t0 = time.time()
        q_np, k_np, _ = synth.gen_batch(cfg)
        qd = torch.from_numpy(synth.to_bf16_bits(q_np).view(np.int16)).cuda().view(torch.bfloat16)
        kd = torch.from_numpy(synth.to_bf16_bits(k_np).view(np.int16)).cuda().view(torch.bfloat16)
        sample = sorted(set(np.linspace(0, B - 1, PARITY_SAMPLE[name]).round().astype(int)))
        q_s, k_s = q_np[sample].copy(), k_np[sample].copy()
        del q_np, k_np
        sets = Cycle(cache_sets(qd, kd))
        log(f"[bench] {name}: batch {B} generated and uploaded in {time.time() - t0:.1f}s, "
            f"{len(sets.sets)} input set(s) in rotation")
        stream = torch.cuda.current_stream()
        timed = make_timed(stream)
        for mode in modes:
            rec = {"batch": B, "lambdas": {}}
            kept_by_lam = {}
            for lam in cfg.lambdas:
                pr = E.Pruner(qd, kd, gh, gw, cfg.keep, cfg.cells, lam, mode)
                for _ in range(args.warmup):
                    pr(*sets.next())
                torch.cuda.synchronize()
                t_a = time.perf_counter()
                for _ in range(n_rep):
                    pr(*sets.next())
                torch.cuda.synchronize()
                us = (time.perf_counter() - t_a) * 1e6 / n_rep
                rec["lambdas"][str(lam)] = {"us_per_step": round(us, 2),
                                            "images_per_s": round(B / (us * 1e-6), 1)}
                kept_by_lam[lam] = pr(qd, kd).cpu().numpy()
            rec["pipelined"] = bench_pipelined(
                cfg, mode, cfg.lam, qd, kd, sets, n_rep, args.warmup,
                torch.from_numpy(kept_by_lam[cfg.lam]).cuda())
            # the two kernels of e2s_prune at the first lambda, each timed alone
            pr = E.Pruner(qd, kd, gh, gw, cfg.keep, cfg.cells, cfg.lam, mode)
            fused = torch.empty((B, N, 3), device="cuda")
            pr(qd, kd, fused)
            fused_h = fused.cpu().numpy()
            del fused
            sh, pa = pr.shape, pr.params
            rho = torch.empty((B, L_, N), device="cuda")
            pbar = torch.empty_like(rho)
            keep_buf = torch.empty((B, cfg.keep), device="cuda", dtype=torch.int32)
            st = stream.cuda_stream
            ws, ws_n = pr.workspace.data_ptr(), pr.workspace.numel()

            def layer_rel():
                qx, kx = sets.next()
                return lib.e2s_layer_reliability(ctypes.byref(sh), ctypes.byref(pa),
                                                 qx.data_ptr(), kx.data_ptr(), ws, ws_n,
                                                 rho.data_ptr(), pbar.data_ptr(), st)

            def fuse_sel():
                return lib.e2s_fuse_select(ctypes.byref(sh), ctypes.byref(pa), rho.data_ptr(),
                                           pbar.data_ptr(), keep_buf.data_ptr(), None, None, st)

            t_lr, t_fs = timed([layer_rel, fuse_sel], n_rep)
            stage_us, tail_us = float(t_lr.mean()) * 1e3, float(t_fs.mean()) * 1e3
            step_us = rec["lambdas"][str(cfg.lam)]["us_per_step"]
            floor_us, bound, flops = roofline_floor_us(cfg, mode, B)
            tail_bytes = B * (2 * 4 * L_ * N + 4 * cfg.keep)
            rec.update({
                "us_per_step": step_us,
                "images_per_s": round(B / (step_us * 1e-6), 1),
                "stage_us": round(stage_us, 2),
                "tail_us": round(tail_us, 2),
                "roofline": {"bound": bound, "floor_us": round(floor_us, 2),
                             "path_frac": round(floor_us / step_us, 4),
                             "stage_frac": round(floor_us / stage_us, 4),
                             "stage_hbm_GBps": round(B * cfg.bytes_per_image()
                                                     / (stage_us * 1e-6) / 1e9, 1)},
                "tail": {"algorithmic_bytes": int(tail_bytes),
                         "hbm_frac": round(tail_bytes / (tail_us * 1e-6) / 1e9 / HBM_PEAK_GBS, 5),
                         "share_of_step": round(tail_us / step_us, 4)},
            })
            if flops is not None:
                rec["roofline"]["stage_mfma_frac"] = round(
                    flops / (stage_us * 1e-6) / 1e12 / MFMA_BF16_PEAK_TFLOPS, 4)
            if mode == "mean_logit":
                # the staged fusion kernel (Eq. 10-19, e2s_fuse_evidence) alone on the
                # batch's supports: it reads e and writes the fused masses, every
                # layer's conflict and c
                H_ = cfg.num_heads
                e_buf = torch.empty((B, L_, H_, N), device="cuda")
                assert lib.e2s_score_heads(ctypes.byref(sh), ctypes.byref(pa), qd.data_ptr(),
                                           kd.data_ptr(), e_buf.data_ptr(), None, st) == 0
                f_buf = torch.empty((B, N, 3), device="cuda")
                k_buf = torch.empty((B, L_, N), device="cuda")
                c_buf = torch.empty((B, N), device="cuda")

                def fuse():
                    return lib.e2s_fuse_evidence(ctypes.byref(sh), e_buf.data_ptr(),
                                                 f_buf.data_ptr(), k_buf.data_ptr(),
                                                 c_buf.data_ptr(), st)

                (t_fu,) = timed([fuse], n_rep)
                fu_us = float(t_fu.mean()) * 1e3
                fu_bytes = B * (4 * L_ * H_ * N + (16 + 4 * L_) * N)
                rec["staged_fuse"] = {
                    "us": round(fu_us, 2), "algorithmic_bytes": int(fu_bytes),
                    "hbm_frac": round(fu_bytes / (fu_us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4)}
                log(f"[bench] {name}: staged fusion kernel {fu_us:.1f} us, "
                    f"{fu_bytes / 1e6:.1f} MB, {rec['staged_fuse']['hbm_frac']:.1%} of 8 TB/s")
                del e_buf, f_buf, k_buf, c_buf
            t_p = time.time()
            ips, used, refs = cpu_baseline_leg(cfg, mode, q_s, k_s, sample)
            rec["cpu_baseline"] = {"value": round(ips, 2), "unit": "images/s", "cores": used,
                                   "kind": "oracle",
                                   "sample": f"images {[int(i) for i in sample]} of the batch, "
                                             f"mode {mode}"}
            rec["parity"] = parity_summary(cfg, refs, sample, kept_by_lam, fused_h)
            log(f"[bench] {name}/{mode}: {step_us:.1f} us/step ({rec['images_per_s']:.0f} "
                f"images/s; 2 streams {rec['pipelined']['us_per_step']:.1f} us/step), "
                f"stage {stage_us:.1f} us, tail {tail_us:.1f} us, "
                f"{rec['roofline']['path_frac']:.1%} of the {bound} roofline; parity "
                f"max|d m~| {rec['parity']['max_abs_dfused']:.1e} "
                f"{rec['parity']['by_lambda']} ({time.time() - t_p:.1f}s)")
            out[f"{name}/{mode}"] = rec
            del pr, rho, pbar, keep_buf
        del qd, kd, sets
        torch.cuda.empty_cache()
    return out


def read_probe_GBps(buf):
    """Achievable streaming-read bandwidth of the device: e2s_read_probe over `buf`
    (the batch's keys, larger than the Infinity Cache), timed with events on the
    current stream; the best of two launch widths, median of 10 launches each."""
    import torch
    from paper_2608_23253_amd import _lib as L
    sink = torch.zeros(1, device=buf.device, dtype=torch.int32)
    nbytes = buf.numel() * buf.element_size()
    best = None
    for wgs in (512, 1024):
        for _ in range(3):
            L.read_probe(buf, wgs, sink)
        ts = []
        for _ in range(10):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            L.read_probe(buf, wgs, sink)
            b.record()
            b.synchronize()
            ts.append(a.elapsed_time(b) * 1e-3)
        gbps = nbytes / sorted(ts)[len(ts) // 2] / 1e9
        if best is None or gbps > best[0]:
            best = (gbps, wgs)
    return {"GBps": round(best[0], 1), "bytes": int(nbytes), "workgroups": best[1],
            "frac_of_nominal": round(best[0] / HBM_PEAK_GBS, 4)}


def bench_pipelined(cfg, mode, lam, qd, kd, sets, steps, warmup, ref_keep):
    """Two batches in flight: the steps alternate between two streams (default
    priority), each with its own Pruner (workspace and outputs), so that a step's
    selection tail can run beside the next step's score stage, as in a serving loop
    that prunes batch after batch.  Wall clock over as many steps as the metric;
    every step's kept indices are those of the one-stream step (same inputs)."""
    import torch
    import paper_2608_23253_amd as E
    prs = [E.Pruner(qd, kd, cfg.grid_h, cfg.grid_w, cfg.keep, cfg.cells, lam, mode)
           for _ in range(2)]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    cur = torch.cuda.current_stream()
    for s in streams:
        s.wait_stream(cur)

    def run(n):
        for i in range(n):
            qx, kx = sets.next()
            prs[i % 2](qx, kx, stream=streams[i % 2].cuda_stream)

    run(max(warmup, 2))
    torch.cuda.synchronize()
    t = time.perf_counter()
    run(steps)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t
    for p in prs:
        assert torch.equal(p.keep_idx, ref_keep), "pipelined steps changed the kept sets"
    us = wall * 1e6 / steps
    B = cfg.batch
    return {"streams": 2, "steps": steps, "us_per_step": round(us, 2),
            "images_per_s": round(B / (us * 1e-6), 1),
            "path_hbm_frac": round(B * cfg.bytes_per_image() / (us * 1e-6) / 1e9 / HBM_PEAK_GBS,
                                   4)}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the path is data-parallel over images and needs no collective; see the "
              "design notes for how it would shard)", file=sys.stderr)
        sys.exit(2)
    if args.copy_calibrate:
        copy_calibrate(args.copy_calibrate)
        return
    if args.hbm_probe:
        hbm_probe(args.hbm_probe)
        return

    import numpy as np
    import torch

    import synth
    import paper_2608_23253_amd as E
    from paper_2608_23253_amd import _lib as L

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    cfg = synth.config_by_name(args.workload)
    B, N = cfg.batch, cfg.num_visual
    t0 = time.time()
    q_np, k_np, _ = synth.gen_batch(cfg)
    log(f"[bench] generated {cfg.name} batch {B} in {time.time() - t0:.1f}s")

    def upload(x):
        if cfg.dtype == "bf16":
            bits = synth.to_bf16_bits(x).view(np.int16)
            return torch.from_numpy(bits).cuda().view(torch.bfloat16)
        return torch.from_numpy(synth.storage_view(x, cfg.dtype)).cuda()

    qd, kd = upload(q_np), upload(k_np)
    torch.cuda.synchronize()
    log(f"[bench] uploaded Q {tuple(qd.shape)} K {tuple(kd.shape)} {qd.dtype}")

    pr = E.Pruner(qd, kd, cfg.grid_h, cfg.grid_w, cfg.keep, cfg.cells, cfg.lam, args.mode)
    stream = torch.cuda.current_stream()
    sets = Cycle(cache_sets(qd, kd))
    log(f"[bench] {len(sets.sets)} input set(s) in rotation")

    # ---- region A: the metric -------------------------------------------------
    for _ in range(args.warmup):
        pr(*sets.next())
    torch.cuda.synchronize()
    t_a = time.perf_counter()
    for _ in range(args.steps):
        pr(*sets.next())
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_a
    ms_step = wall * 1e3 / args.steps
    value = B / (wall / args.steps)
    log(f"[bench] e2s_prune: {ms_step:.4f} ms/step, {value:.1f} images/s")
    if args.kernel_only:
        print(json.dumps({"ms_per_step": ms_step, "value": value}))
        return

    # ---- region B: the two kernels of e2s_prune, each timed alone ---------------
    lib = L.lib()
    sh = pr.shape
    pa = L.make_params(pr.params.dtype, args.mode, 0.0, cfg.cells, cfg.lam, cfg.keep)
    L_, H_ = cfg.num_layers, cfg.num_heads
    rho = torch.empty((B, L_, N), device="cuda", dtype=torch.float32)
    pbar = torch.empty_like(rho)
    keep_buf = torch.empty((B, cfg.keep), device="cuda", dtype=torch.int32)
    st = stream.cuda_stream
    shp, pap = ctypes.byref(sh), ctypes.byref(pa)
    ws, ws_n = pr.workspace.data_ptr(), pr.workspace.numel()
    n_ev = args.steps

    def layer_rel():
        qx, kx = sets.next()
        return lib.e2s_layer_reliability(shp, pap, qx.data_ptr(), kx.data_ptr(), ws, ws_n,
                                         rho.data_ptr(), pbar.data_ptr(), st)

    def fuse_sel():
        return lib.e2s_fuse_select(shp, pap, rho.data_ptr(), pbar.data_ptr(), keep_buf.data_ptr(),
                                   None, None, st)

    timed = make_timed(args)(stream)

    t_lr, t_fs = timed([layer_rel, fuse_sel], n_ev)
    assert torch.equal(keep_buf, pr.keep_idx), "two-call and e2s_prune results differ"

    # ---- region C: the staged entry points (score, fused evidence, select) -----
    e_buf = torch.empty((B, L_, H_, N), device="cuda", dtype=torch.float32)
    c_buf = torch.empty((B, N), device="cuda", dtype=torch.float32)

    def score():
        qx, kx = sets.next()
        return lib.e2s_score_heads(shp, pap, qx.data_ptr(), kx.data_ptr(), e_buf.data_ptr(),
                                   None, st)

    def fuse():
        return lib.e2s_fuse_evidence(shp, e_buf.data_ptr(), None, None, c_buf.data_ptr(), st)

    def select():
        return lib.e2s_spatial_select(shp, pap, c_buf.data_ptr(), keep_buf.data_ptr(), None,
                                      None, st)

    t_score, t_fuse, t_sel = timed([score, fuse, select], n_ev)
    assert torch.equal(keep_buf, pr.keep_idx), "staged and fused paths disagree"

    per_img_qk = cfg.bytes_per_image()
    # algorithmic bytes of the score and reliability stage: Q and K read once,
    # rho and pbar_c [B, L, N] f32 written
    algo_bytes = B * per_img_qk + 2 * 4 * B * L_ * N
    lr_ms = float(t_lr.mean())
    achieved = algo_bytes / (lr_ms * 1e-3) / 1e9
    traffic = read_traffic(args.mode, args.workload)
    flops_eq1 = 2.0 * B * L_ * H_ * cfg.num_text * N * cfg.head_dim
    log(f"[bench] layer_reliability {lr_ms * 1e3:.1f} us (p10 {np.percentile(t_lr, 10) * 1e3:.1f},"
        f" p90 {np.percentile(t_lr, 90) * 1e3:.1f}) {achieved:.0f} GB/s; fuse_select "
        f"{t_fs.mean() * 1e3:.1f} us | staged: score {t_score.mean() * 1e3:.1f} us, fuse "
        f"{t_fuse.mean() * 1e3:.1f} us, select {t_sel.mean() * 1e3:.1f} us")

    probe = read_probe_GBps(kd)
    log(f"[bench] streaming read of the keys ({probe['bytes'] / 1e9:.2f} GB): "
        f"{probe['GBps']:.0f} GB/s ({probe['frac_of_nominal']:.1%} of 8 TB/s)")
    props = torch.cuda.get_device_properties(qd.device)
    device = {"name": props.name, "gcn_arch": getattr(props, "gcnArchName", ""),
              "compute_units": props.multi_processor_count, "read_probe": probe}

    extras = {}
    if not args.no_extras:
        extras = bench_variants_and_schedule(args, cfg, qd, kd, stream, timed)
        extras["ragged"] = bench_ragged(args, timed)
        extras["compaction"] = bench_compaction(args, timed, kd, pr.keep_idx)
        extras["pipelined"] = bench_pipelined(cfg, args.mode, cfg.lam, qd, kd, sets,
                                              args.steps, args.warmup, pr.keep_idx)
        log(f"[bench] two batches in flight (2 streams): "
            f"{extras['pipelined']['us_per_step']:.1f} us/step, "
            f"{extras['pipelined']['images_per_s']:.0f} images/s")

    # ---- CPU oracle baseline ----------------------------------------------------
    import oracle as O
    from threadpoolctl import threadpool_info, threadpool_limits
    cores = len(os.sched_getaffinity(0))
    threadpool_limits(cores)
    used = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    t_c = time.perf_counter()
    done = 0
    passes = 0
    first_pass = []
    while True:
        for b in range(B):
            ref = O.prune_image(q_np[b], k_np[b], cfg.grid_h, cfg.grid_w, cfg.keep, cfg.cells,
                                cfg.lam, args.mode)
            if passes == 0:
                first_pass.append(ref)
            done += 1
            if time.perf_counter() - t_c >= args.cpu_seconds and done >= 8:
                break
        passes += 1
        if time.perf_counter() - t_c >= args.cpu_seconds:
            break
    cpu_s = time.perf_counter() - t_c
    cpu_value = done / cpu_s
    log(f"[bench] oracle: {done} images in {cpu_s:.1f}s on {used} threads ({cores} cores, "
        f"{cpu_model()})")
    # the step's results on the images the oracle processed, against its results
    fused_full = torch.empty((B, N, 3), device="cuda")
    kept_full = pr(qd, kd, fused_full).cpu().numpy()
    head_sample = list(range(len(first_pass)))
    parity = parity_summary(cfg, first_pass, head_sample, {cfg.lam: kept_full},
                            fused_full.cpu().numpy())
    parity["images"] = f"0..{len(first_pass) - 1}"
    log(f"[bench] parity on {len(first_pass)} images: {parity}")
    if not args.no_configs:
        extras["configs"] = bench_configs(args, make_timed(args))

    out = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "images/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic",
        "config": {
            "workload": (f"{cfg.name}: {SHAPES.get(cfg.name, 'synthetic')}, batch {B} images, "
                         f"{cfg.num_layers} "
                         f"source layers, {cfg.num_heads} heads ({cfg.num_kv_heads} key heads) "
                         f"x {cfg.head_dim}, "
                         f"{cfg.num_text} text queries, {cfg.grid_h}x{cfg.grid_w}={N} visual "
                         f"tokens, keep {cfg.keep}, G={cfg.cells}, lambda={cfg.lam}"),
            "score_mode": args.mode,
            "input_dtype": cfg.dtype,
            "batch": B,
        },
        "roofline": {
            "bound": "hbm",
            "kernel": "score + head reliability (e2s_layer_reliability)",
            "achieved": round(achieved, 1),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": traffic,
            "algorithmic_bytes_per_launch": algo_bytes,
            "launch_us": round(lr_ms * 1e3, 2),
            "launch_us_p10_p50_p90": [round(float(np.percentile(t_lr, x)) * 1e3, 2)
                                      for x in (10, 50, 90)],
            "mfma_frac_if_eq1_flops": round(flops_eq1 / (lr_ms * 1e-3) / 1e12
                                            / MFMA_BF16_PEAK_TFLOPS, 4),
            "frac_of_measured_read": round(achieved / probe["GBps"], 4),
        },
        "device": device,
        "stages_us": {"layer_reliability": round(lr_ms * 1e3, 2),
                      "fuse_select": round(float(t_fs.mean()) * 1e3, 2),
                      "staged_score": round(float(t_score.mean()) * 1e3, 2),
                      "staged_fuse": round(float(t_fuse.mean()) * 1e3, 2),
                      "staged_select": round(float(t_sel.mean()) * 1e3, 2)},
        "path_hbm_frac": round(B * per_img_qk / (ms_step * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        "parity": parity,
        "cpu_baseline": {
            "value": round(cpu_value, 2),
            "unit": "images/s",
            "cores": used,
            "cpu_model": cpu_model(),
            "kind": "oracle",
            "sample": (f"{done} images of the same {cfg.name} batch ({passes} pass(es) over "
                       f"images 0..{B - 1}), NumPy float64 oracle, mode {args.mode}"),
        },
    }
    out.update(extras)
    print(json.dumps(out))


if __name__ == "__main__":
    main()
