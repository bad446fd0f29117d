"""CPU oracle for the E2S-Pruner token-scoring path (arXiv 2608.23253).

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute this module: only the test suite, the smoke check and the benchmark's
CPU-baseline leg use it.  It shares no code with the HIP library.

Plain, slow, obviously-correct NumPy in float64.  Inputs are converted exactly
from their stored float32 / bfloat16 values.  Each function follows one passage
of the paper, in the paper's order and notation; there is no blocking, fusion
or reordering beyond what the definitions state.  A matrix product and a sort
are used as library steps.

Readings taken where the paper is silent or ambiguous (the project's design
notes list them in full):
  * score mode "mean_logit" (default): Eq. (1) averages the scaled logits over
    the text queries, then Eq. (8) takes a softmax over the visual tokens.
    Score mode "mean_prob": a softmax over the visual tokens per text query,
    then the mean over queries.
  * the softmax of Eq. (8) runs over the N_V visual tokens only; N_l of Eq. (9)
    is N_V (all visual tokens are candidates).
  * query head h reads key head floor(h * Hkv / H) (grouped-query attention).
  * K^(1) = 0, so with one source layer q = Pl(I).
  * total conflict (1 - K <= 0): the fused mass becomes vacuous (0, 0, 1) and
    K is recorded as 1, so q = 1 by Eq. (19).
  * cells: cell(n) = floor(row*G/grid_h)*G + floor(col*G/grid_w), row-major.
  * ties (cell argmax and the global top-K) go to the lowest token index; the
    kept set is returned in ascending index order.
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np

SCORE_MODES = ("mean_logit", "mean_prob")

# The full method and the ablation variants of Sec. 5 (ablation study, Table 2);
# each removes or replaces one component, as read in prune_stage.
VARIANTS = ("full", "a1_attention_topk", "a2_no_head_reliability", "a3_no_layer_fusion",
            "a4_no_conflict_protection", "a5_no_spatial_novelty")


# ---------------------------------------------------------------------------
# Stage 1 inputs: text-to-visual attention (Sec. 3.1 and 4.1)
# ---------------------------------------------------------------------------

def text_visual_logits(q_lh: np.ndarray, k_lg: np.ndarray, scale: float) -> np.ndarray:
    """z[t, n] = Q_t K_n^T / sqrt(d) for one head (the summand of Eq. (1), Sec. 3.1).

    q_lh: [N_T, d] text queries of head h; k_lg: [N_V, d] keys of the KV head h reads.
    """
    q = np.asarray(q_lh, dtype=np.float64)
    k = np.asarray(k_lg, dtype=np.float64)
    return (q @ k.T) * float(scale)


def softmax_over_visual(x: np.ndarray) -> np.ndarray:
    """Eq. (8): r_n = exp(x_n) / sum_j exp(x_j) along the last axis (visual tokens).

    The maximum is subtracted first; this leaves the quotient unchanged."""
    x = np.asarray(x, dtype=np.float64)
    e = np.exp(x - x.max(axis=-1, keepdims=True))
    return e / e.sum(axis=-1, keepdims=True)


def normalized_attention(z: np.ndarray, mode: str = "mean_logit") -> np.ndarray:
    """r over the visual tokens for one head from its logits z [N_T, N_V].

    mean_logit: a = mean_t z (Eq. (1)), r = softmax_n(a) (Eq. (8)).
    mean_prob:  r = mean_t softmax_n(z[t, :]).
    """
    if mode == "mean_logit":
        a = z.mean(axis=0)
        return softmax_over_visual(a)
    if mode == "mean_prob":
        return softmax_over_visual(z).mean(axis=0)
    raise ValueError(f"unknown score mode {mode!r}")


def support_from_attention(r: np.ndarray, n_l: int) -> np.ndarray:
    """Eq. (9): p = N_l r / (1 + N_l r), in [0, 1); r = 1/N_l gives exactly 0.5."""
    x = float(n_l) * np.asarray(r, dtype=np.float64)
    return x / (1.0 + x)


def score_heads(q: np.ndarray, k: np.ndarray, mode: str = "mean_logit",
                scale: float | None = None):
    """Per-head normalized attention r and support p for one image.

    q: [L, H, N_T, d]; k: [L, Hkv, N_V, d].  Returns (r, p), each [L, H, N_V].
    Query head h reads KV head floor(h*Hkv/H).  scale defaults to 1/sqrt(d) (Eq. (1)).
    """
    L, H, _, d = q.shape
    Hkv, n = k.shape[1], k.shape[2]
    if k.shape[0] != L or H % Hkv != 0:
        raise ValueError("shape mismatch between Q and K")
    s = 1.0 / math.sqrt(d) if scale is None else float(scale)
    r = np.empty((L, H, n), dtype=np.float64)
    for l in range(L):
        for h in range(H):
            g = (h * Hkv) // H
            z = text_visual_logits(q[l, h], k[l, g], s)
            r[l, h] = normalized_attention(z, mode)
    return r, support_from_attention(r, n)


# ---------------------------------------------------------------------------
# Stage 1: multi-head evidence fusion (Sec. 4.1)
# ---------------------------------------------------------------------------

def head_reliability(p: np.ndarray):
    """Eq. (10): rho = clarity * consistency over the H heads (axis -2 of p).

    p: [..., H, N].  clarity = (2/H)|sum_h (p_h - 0.5)|;
    consistency = 1 - (2/H) sum_h |p_h - pbar|, pbar = mean_h p_h.
    Returns (rho, pbar), each [..., N].
    """
    p = np.asarray(p, dtype=np.float64)
    H = p.shape[-2]
    pbar = p.mean(axis=-2)
    clarity = (2.0 / H) * np.abs((p - 0.5).sum(axis=-2))
    consistency = 1.0 - (2.0 / H) * np.abs(p - pbar[..., None, :]).sum(axis=-2)
    return clarity * consistency, pbar


def head_masses(rho: np.ndarray, pbar: np.ndarray) -> np.ndarray:
    """Eq. (11): (m(I), m(U), m(Theta)) = (rho pbar, rho (1 - pbar), 1 - rho); [..., N, 3]."""
    rho = np.asarray(rho, dtype=np.float64)
    pbar = np.asarray(pbar, dtype=np.float64)
    return np.stack([rho * pbar, rho * (1.0 - pbar), 1.0 - rho], axis=-1)


# ---------------------------------------------------------------------------
# Stage 2: layer-wise evidence fusion with explicit conflict (Sec. 4.2)
# ---------------------------------------------------------------------------

def dempster_step(acc: np.ndarray, m: np.ndarray):
    """One recursion step of Eq. (13)-(16): fuse the cumulative mass acc with layer mass m.

    acc, m: [..., 3] over (I, U, Theta).  Returns (fused, K).  Where 1 - K is not
    positive (total conflict) the fused mass is vacuous (0, 0, 1) and K is 1.
    """
    aI, aU, aT = acc[..., 0], acc[..., 1], acc[..., 2]
    mI, mU, mT = m[..., 0], m[..., 1], m[..., 2]
    K = aI * mU + aU * mI                                     # Eq. (13)
    denom = 1.0 - K
    ok = denom > 0.0
    safe = np.where(ok, denom, 1.0)
    fI = (aI * mI + aI * mT + aT * mI) / safe                 # Eq. (14)
    fU = (aU * mU + aU * mT + aT * mU) / safe                 # Eq. (15)
    fT = (aT * mT) / safe                                     # Eq. (16)
    fused = np.stack([np.where(ok, fI, 0.0), np.where(ok, fU, 0.0),
                      np.where(ok, fT, 1.0)], axis=-1)
    return fused, np.where(ok, K, 1.0)


def ds_combine_layers(masses: np.ndarray, init: np.ndarray | None = None):
    """Eq. (12)-(19) over the source layers in order (axis 0 of masses [L, N, 3]).

    Without `init` the recursion starts from the first layer (Eq. 12) and
    conflict row 0 is 0.  With `init` [N, 3], the cumulative mass carried from
    earlier pruning operations, every layer is combined onto it and row l holds
    the conflict of that layer's step.
    Returns (fused [N,3], conflict [L,N], Pl [N], q [N], Bel [N]).
    """
    masses = np.asarray(masses, dtype=np.float64)
    L = masses.shape[0]
    conflict = np.zeros(masses.shape[:2], dtype=np.float64)
    if init is None:
        acc, first = masses[0].copy(), 1                      # Eq. (12)
    else:
        acc, first = np.asarray(init, dtype=np.float64).copy(), 0
    for l in range(first, L):
        acc, conflict[l] = dempster_step(acc, masses[l])
    bel = acc[..., 0]                                         # Eq. (17)
    pl = acc[..., 0] + acc[..., 2]                            # Eq. (18)
    q = 1.0 - (1.0 - pl) * (1.0 - conflict[L - 1])            # Eq. (19)
    return acc, conflict, pl, q, bel


# ---------------------------------------------------------------------------
# Spatial novelty and top-K (Sec. 4.3)
# ---------------------------------------------------------------------------

def cell_of_token(grid_h: int, grid_w: int, cells: int, pos: np.ndarray | None = None) -> np.ndarray:
    """Cell id of every token of a grid_h x grid_w raster under a G x G partition
    (of the tokens at raster positions `pos`, default all of them in order)."""
    n = np.arange(grid_h * grid_w) if pos is None else np.asarray(pos, dtype=np.int64)
    row, col = n // grid_w, n % grid_w
    return (row * cells // grid_h) * cells + (col * cells // grid_w)


def cell_representatives(q: np.ndarray, grid_h: int, grid_w: int, cells: int,
                         pos: np.ndarray | None = None) -> np.ndarray:
    """Eq. (20)-(21): b_n = 1 for the highest-q token of each occupied cell.

    q[i] belongs to the token at raster position pos[i] (default i; positions
    ascending).  A cell is occupied when it holds at least one of these tokens.
    Ties go to the lowest index (np.argmax returns the first maximum)."""
    q = np.asarray(q, dtype=np.float64)
    cell = cell_of_token(grid_h, grid_w, cells, pos)
    b = np.zeros(q.shape[0], dtype=np.int64)
    for g in range(cells * cells):
        members = np.nonzero(cell == g)[0]          # ascending indices
        if members.size:
            b[members[int(np.argmax(q[members]))]] = 1
    return b


def spatial_select(q: np.ndarray, grid_h: int, grid_w: int, cells: int, lam: float,
                   keep: int, pos: np.ndarray | None = None):
    """Eq. (20)-(23): representatives, q~ = (1-lam) q + lam b, keep the K largest q~.

    Ties in q~ go to the lowest index.  Returns (kept ascending [K], q~ [N], b [N]),
    indices into q."""
    q = np.asarray(q, dtype=np.float64)
    b = cell_representatives(q, grid_h, grid_w, cells, pos)
    qt = (1.0 - lam) * q + lam * b                            # Eq. (22)
    idx = np.arange(q.shape[0])
    order = np.lexsort((idx, -qt))                            # by -q~, then index
    kept = np.sort(order[:keep])                              # Eq. (23)
    return kept.astype(np.int64), qt, b


# ---------------------------------------------------------------------------
# The whole path for one image / a batch
# ---------------------------------------------------------------------------

@dataclasses.dataclass
class ImageResult:
    r: np.ndarray          # [L, H, N]  normalized attention (Eq. 8)
    p: np.ndarray          # [L, H, N]  support (Eq. 9)
    rho: np.ndarray        # [L, N]     reliability (Eq. 10)
    pbar: np.ndarray       # [L, N]     mean support
    masses: np.ndarray     # [L, N, 3]  layer masses (Eq. 11)
    fused: np.ndarray      # [N, 3]     cumulative fused mass after the last layer
    conflict: np.ndarray   # [L, N]     K^(l) of each step (Eq. 13)
    pl: np.ndarray         # [N]        plausibility of I (Eq. 18)
    q: np.ndarray          # [N]        retention priority (Eq. 19)
    qt: np.ndarray         # [N]        spatially adjusted score (Eq. 22)
    is_rep: np.ndarray     # [N]        representative indicator b (Eq. 21)
    keep: np.ndarray       # [K]        kept entries, ascending (Eq. 23)
    score: np.ndarray | None = None   # [N] ranking score of the A1 variant
    keep_pos: np.ndarray | None = None   # [K] raster positions of the kept entries
    m_out: np.ndarray | None = None      # [K, 3] fused mass of the kept entries


def prune_stage(q: np.ndarray, k: np.ndarray, cand_pos: np.ndarray, grid_h: int, grid_w: int,
                keep: int, cells: int = 4, lam: float = 0.1, mode: str = "mean_logit",
                scale: float | None = None, m_prev: np.ndarray | None = None,
                variant: str = "full") -> ImageResult:
    """One pruning operation of Algorithm 1 for one image.

    q: [L, H, N_T, d] text queries of the operation's L evidence layers;
    k: [L, Hkv, N_l, d] keys of the N_l current candidates, in candidate order;
    cand_pos: [N_l] the candidates' raster positions on the grid_h x grid_w grid,
    ascending; m_prev: [N_l, 3] their cumulative fused mass from the earlier
    operations (None for the first).  N_l is the N_l of Eq. (9) and the softmax of
    Eq. (8) runs over the candidates.  Returns indices into the candidate list, the
    kept positions and the kept tokens' fused masses (carried to the next
    operation).

    Ablation variants (Sec. 5, Table 2), each changing one component:
      a1_attention_topk          top-K of the attention r averaged over the
                                 operation's layers and heads; no evidence, no
                                 carried mass, no spatial term
      a2_no_head_reliability     rho = 1 in Eq. (11): Bayesian layer masses
      a3_no_layer_fusion         only the operation's last layer's masses; no
                                 Dempster combination with earlier layers or
                                 operations, so K = 0 and q = Pl
      a4_no_conflict_protection  q = Pl(I) instead of Eq. (19)
      a5_no_spatial_novelty      lambda = 0 in Eq. (22)
    """
    if variant not in VARIANTS:
        raise ValueError(f"unknown variant {variant!r}")
    cand_pos = np.asarray(cand_pos, dtype=np.int64)
    n_l = k.shape[2]
    if cand_pos.shape != (n_l,):
        raise ValueError("cand_pos must list the raster position of every candidate")
    r, p = score_heads(q, k, mode, scale)
    if variant == "a1_attention_topk":
        score = r.mean(axis=(0, 1))                           # [N_l]
        idx = np.arange(n_l)
        kept = np.sort(np.lexsort((idx, -score))[:keep]).astype(np.int64)
        nan = np.full(n_l, np.nan)
        return ImageResult(r, p, nan, nan, np.full((1, n_l, 3), np.nan), np.full((n_l, 3), np.nan),
                           np.zeros((1, n_l)), nan, nan, nan, np.zeros(n_l, np.int64), kept,
                           score=score, keep_pos=cand_pos[kept], m_out=None)
    rho, pbar = head_reliability(p)
    if variant == "a2_no_head_reliability":
        rho = np.ones_like(rho)
    masses = head_masses(rho, pbar)
    if variant == "a3_no_layer_fusion":
        fused, conflict, pl, prio, _ = ds_combine_layers(masses[-1:])
    else:
        fused, conflict, pl, prio, _ = ds_combine_layers(masses, m_prev)
    if variant == "a4_no_conflict_protection":
        prio = pl
    if variant == "a5_no_spatial_novelty":
        lam = 0.0
    kept, qt, b = spatial_select(prio, grid_h, grid_w, cells, lam, keep, cand_pos)
    return ImageResult(r, p, rho, pbar, masses, fused, conflict, pl, prio, qt, b, kept,
                       keep_pos=cand_pos[kept], m_out=fused[kept])


def prune_image(q: np.ndarray, k: np.ndarray, grid_h: int, grid_w: int, keep: int,
                cells: int = 4, lam: float = 0.1, mode: str = "mean_logit",
                scale: float | None = None, variant: str = "full") -> ImageResult:
    """Algorithm 1 for one image with all evidence layers fused before one top-K
    (one pruning operation over every visual token).

    q: [L, H, N_T, d]; k: [L, Hkv, N_V, d] with N_V = grid_h * grid_w."""
    if k.shape[2] != grid_h * grid_w:
        raise ValueError("N_V must equal grid_h * grid_w")
    return prune_stage(q, k, np.arange(grid_h * grid_w), grid_h, grid_w, keep, cells, lam, mode,
                       scale, None, variant)


def prune(q: np.ndarray, k: np.ndarray, grid_h: int, grid_w: int, keep: int,
          cells: int = 4, lam: float = 0.1, mode: str = "mean_logit",
          scale: float | None = None, variant: str = "full"):
    """prune_image over a batch: q [B, L, H, N_T, d], k [B, L, Hkv, N_V, d]."""
    return [prune_image(q[b], k[b], grid_h, grid_w, keep, cells, lam, mode, scale, variant)
            for b in range(q.shape[0])]


# ---------------------------------------------------------------------------
# Progressive schedule (Algorithm 1 with shrinking candidate sets; Sec. 5.1)
# ---------------------------------------------------------------------------

def prune_progressive(q_ops, k_ops, grid_h: int, grid_w: int, budgets, cells: int = 4,
                      lam: float = 0.1, mode: str = "mean_logit", scale: float | None = None,
                      variant: str = "full"):
    """Algorithm 1 for one image over a sequence of pruning operations.

    q_ops[s]: [L_s, H, N_T, d] text queries of operation s; k_ops[s]: [L_s, Hkv,
    N_V, d] keys of every visual token at operation s's layers (the operation sees
    only the rows of its current candidates); budgets[s]: K_s, non-increasing.
    Operation s keeps budgets[s] of its candidates and hands them, with their
    fused masses, to operation s + 1.  Returns the list of per-operation results;
    result.keep_pos of the last is the retained set V."""
    cand = np.arange(grid_h * grid_w)
    m_prev = None
    out = []
    for s, keep in enumerate(budgets):
        if keep > cand.size:
            raise ValueError("a budget exceeds the candidates left")
        res = prune_stage(q_ops[s], k_ops[s][:, :, cand, :], cand, grid_h, grid_w, keep, cells,
                          lam, mode, scale, m_prev, variant)
        out.append(res)
        cand = res.keep_pos
        m_prev = res.m_out
    return out


def compact_tokens(x: np.ndarray, keep: np.ndarray) -> np.ndarray:
    """The retained tokens of a pruning operation (Algorithm 1's output V_keep; the
    layers after a pruning layer see only them, Sec. 5.1): x[..., keep[j], :] for
    j = 0..K-1 in order, from per-token vectors x [..., N, C].  A gather, no
    arithmetic."""
    keep = np.asarray(keep, dtype=np.int64)
    return np.take(x, keep, axis=-2)


def avg_tokens(num_layers: int, n_visual: int, prune_after, kept) -> float:
    """Eq. (24): mean over the num_layers LLM layers of the visual tokens each
    layer processes, when pruning after layers prune_after[j] (1-based) leaves
    kept[j] tokens for the layers that follow."""
    counts = []
    for i in range(1, num_layers + 1):
        t = n_visual
        for a, kj in zip(prune_after, kept):
            if i > a:
                t = kj
        counts.append(t)
    return sum(counts) / num_layers
