"""Shared helpers of the GPU parity tests: device upload, oracle runs and the
set-comparison rule with its tie excuse."""
from __future__ import annotations

import dataclasses
import sys

import numpy as np

import oracle as O
import synth

# Tie excuse of the set comparison: a GPU kept set may differ from the oracle's
# only by tokens whose oracle score q~ lies within this distance of the oracle's
# K-th kept score.
TIE_GAP = 1e-5


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def to_device(x: np.ndarray, dtype: str):
    """Upload float32 values holding exactly representable storage values, bit-exact."""
    import torch
    if dtype == "bf16":
        bits = synth.to_bf16_bits(x).view(np.int16)
        return torch.from_numpy(bits).cuda().view(torch.bfloat16)
    if dtype == "f16":
        return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float16)).cuda()
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).cuda()


@dataclasses.dataclass
class SetCompare:
    verdict: str          # "exact", "tie", "fail"
    swaps: int
    near_boundary: int    # oracle tokens within TIE_GAP of the K-th kept score


def compare_sets(gpu_keep: np.ndarray, ref: O.ImageResult, gap: float = TIE_GAP) -> SetCompare:
    """Tie rule on the oracle's ranking score: q~ with an absolute window, or, for
    the attention top-K variant, the mean attention with a window relative to the
    K-th kept value (attention averages 1/N, so an absolute window would not
    scale)."""
    ok = list(ref.keep)
    K = len(ok)
    if K == 0:
        return SetCompare("exact" if len(gpu_keep) == 0 else "fail", 0, 0)
    score = ref.qt if ref.score is None else ref.score
    s_k = score[ok].min()
    if ref.score is not None:
        gap = gap * abs(s_k)
    near = int((np.abs(score - s_k) < gap).sum())
    g, o = set(int(x) for x in gpu_keep), set(int(x) for x in ok)
    if g == o:
        return SetCompare("exact", 0, near)
    sym = g ^ o
    if len(g) == K and all(abs(score[n] - s_k) < gap for n in sym):
        return SetCompare("tie", len(sym) // 2, near)
    return SetCompare("fail", len(sym) // 2, near)


def check_keep_wellformed(keep: np.ndarray, N: int, K: int):
    assert keep.shape[-1] == K
    if K == 0:
        return
    for row in keep.reshape(-1, K):
        assert (np.diff(row) > 0).all(), "keep_idx must be strictly ascending"
        if K:
            assert row[0] >= 0 and row[-1] < N


def oracle_images(cfg: synth.Config, q: np.ndarray, k: np.ndarray, images, mode: str,
                  lam: float | None = None, keep: int | None = None):
    lam = cfg.lam if lam is None else lam
    keep = cfg.keep if keep is None else keep
    return [O.prune_image(q[i], k[i], cfg.grid_h, cfg.grid_w, keep, cfg.cells, lam, mode)
            for i in images]
