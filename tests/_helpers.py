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


# Mass bar of the fused masses end to end: 1e-4 absolute (the stated bar) AND a
# relative bound, since at the workloads' scale m~(I) and m~(U) are ~1e-4 themselves.
MASS_ATOL = 1e-4
MASS_RTOL = 2e-3
MASS_FLOOR = 1e-7


def mass_errors(got, ref):
    """(max absolute error, max error / (MASS_FLOOR + MASS_RTOL |ref|)) of fused masses."""
    got = np.asarray(got, dtype=np.float64)
    err = np.abs(got - ref)
    if err.size == 0:
        return 0.0, 0.0
    return float(err.max()), float((err / (MASS_FLOOR + MASS_RTOL * np.abs(ref))).max())


def assert_mass_bar(got, ref, what="fused masses"):
    """Both gates: max |d m~| <= 1e-4, and every element within the relative bound."""
    abs_err, rel_worst = mass_errors(got, ref)
    assert abs_err <= MASS_ATOL, f"{what}: max |d| = {abs_err:.3e} > {MASS_ATOL}"
    assert rel_worst <= 1.0, (f"{what}: relative error {rel_worst:.3f} x the bound "
                              f"{MASS_FLOOR} + {MASS_RTOL} |ref|")
    return abs_err


@dataclasses.dataclass
class SetCompare:
    verdict: str          # "exact", "tie", "rep_flip", "fail"
    swaps: int
    near_boundary: int    # oracle tokens within TIE_GAP of the K-th kept score


@dataclasses.dataclass
class SelectGeom:
    """What the representative-flip excuse needs to recompute the oracle's ranking:
    the grid, G, the novelty weight and the candidates' raster positions."""
    grid_h: int
    grid_w: int
    cells: int
    lam: float
    pos: np.ndarray | None = None


def _tie_verdict(gpu_keep, keep, score, gap):
    """exact / tie / fail of one GPU set against one ranking (see compare_sets)."""
    K = len(keep)
    s_k = score[list(keep)].min()
    near = int((np.abs(score - s_k) < gap).sum())
    g, o = set(int(x) for x in gpu_keep), set(int(x) for x in keep)
    if g == o:
        return "exact", 0, near
    sym = g ^ o
    if len(g) == K and all(abs(score[n] - s_k) < gap for n in sym):
        return "tie", len(sym) // 2, near
    return "fail", len(sym) // 2, near


def _flip_rankings(ref: O.ImageResult, geom: SelectGeom, gap: float, limit: int = 256):
    """Kept sets and q~ of the oracle ranking redone with another representative in
    cells whose best tokens' oracle q lie within `gap` of each other (Eq. 20 on
    numerical ties: the GPU decides from float32 c, the oracle from float64 q)."""
    q = ref.q
    cell = O.cell_of_token(geom.grid_h, geom.grid_w, geom.cells, geom.pos)
    choices = []
    for g in np.unique(cell):
        members = np.nonzero(cell == g)[0]
        best = q[members].max()
        alt = members[np.abs(q[members] - best) < gap]
        rep = members[int(np.argmax(q[members]))]
        if alt.size > 1:
            choices.append((rep, [int(a) for a in alt if a != rep]))
    if not choices:
        return []
    combos = [[]]
    for rep, alts in choices:
        combos = [c + [(rep, a)] for c in combos for a in [None] + alts]
        if len(combos) > limit:
            return []
    out = []
    idx = np.arange(q.shape[0])
    for c in combos:
        if all(a is None for _, a in c):
            continue
        b = ref.is_rep.astype(np.float64).copy()
        for rep, a in c:
            if a is not None:
                b[rep], b[a] = 0.0, 1.0
        qt = (1.0 - geom.lam) * q + geom.lam * b
        kept = np.sort(np.lexsort((idx, -qt))[:len(ref.keep)])
        out.append((kept, qt))
    return out


def compare_sets(gpu_keep: np.ndarray, ref: O.ImageResult, gap: float = TIE_GAP,
                 geom: SelectGeom | None = None) -> SetCompare:
    """Tie rule on the oracle's ranking score: q~ with an absolute window, or, for
    the attention top-K variant, the mean attention with a window relative to the
    K-th kept value (attention averages 1/N, so an absolute window would not
    scale).

    With `geom`, a set that would fail is checked once more for a representative
    flip: a cell whose two best tokens have oracle q within `gap` may have its
    novelty bonus on either; if the GPU set matches (exactly or by the tie rule)
    the ranking redone with the other representative, the verdict is "rep_flip"."""
    ok = list(ref.keep)
    K = len(ok)
    if K == 0:
        return SetCompare("exact" if len(gpu_keep) == 0 else "fail", 0, 0)
    score = ref.qt if ref.score is None else ref.score
    if ref.score is not None:
        gap_s = gap * abs(score[ok].min())
    else:
        gap_s = gap
    verdict, swaps, near = _tie_verdict(gpu_keep, ok, score, gap_s)
    if verdict != "fail" or geom is None or ref.score is not None or geom.lam == 0.0:
        return SetCompare(verdict, swaps, near)
    for kept, qt in _flip_rankings(ref, geom, gap):
        v, s, _ = _tie_verdict(gpu_keep, kept, qt, gap)
        if v != "fail":
            return SetCompare("rep_flip", s, near)
    return SetCompare(verdict, swaps, near)


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
