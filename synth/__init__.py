"""Seeded synthetic inputs for the E2S-Pruner token-scoring path.

This module produces the text-query tensor Q [B, L, H, N_T, d] and the visual-key
tensor K [B, L, Hkv, N_V, d] that both the HIP path and the CPU oracle consume.
It holds none of the pruning method's arithmetic: it draws Gaussian tensors,
places a spatially clustered set of "salient" visual tokens, shifts their keys
toward the mean text query, optionally plants near-duplicate keys, and rounds to
bfloat16 once.  Both sides see exactly the same bits.

Workload shapes follow the two vision-language models the paper evaluates
(LLaVA-1.5-7B: 576 visual tokens on a 24x24 grid, 32 heads of dim 128;
Qwen2-VL-7B: grouped-query attention with 28 query heads over 4 KV heads), see
the paper's experimental settings (Sec. 5.1) and the 24x24 grid of Sec. 4.3.
The paper's benchmarks (GQA, SQA, TextVQA, POPE, MME, MMBench, AI2D) and model
weights are not used: these seeded tensors stand in for them.

Random streams: every image draws from its own NumPy ``Philox`` generator seeded
by ``SeedSequence([2608, config_id, image_index])``, so any image of any batch can
be regenerated on its own (used to sample full-size batches in tests).
"""
from __future__ import annotations

import dataclasses
import math
import os
from concurrent.futures import ThreadPoolExecutor
from typing import Iterable, Sequence

import numpy as np

__all__ = [
    "Config", "CONFIGS", "config_by_name", "gen_image", "gen_batch",
    "to_bf16_bits", "bf16_bits_to_f32", "salient_set", "heavy_tailed",
    "RaggedConfig", "RAGGED", "ragged_by_name", "ragged_dims", "gen_ragged",
]

SEED_ROOT = 2608


@dataclasses.dataclass(frozen=True)
class Config:
    """One synthetic workload: tensor shapes, value recipe and selection params."""
    name: str
    config_id: int
    batch: int
    num_layers: int          # L: source (pruning) layers whose evidence is fused
    num_heads: int           # H: query heads
    num_kv_heads: int        # Hkv: key/value heads (H % Hkv == 0)
    head_dim: int            # d
    num_text: int            # N_T: text queries
    grid_h: int
    grid_w: int
    keep: int                # K of the final top-K
    lambdas: tuple           # novelty weights run on this workload (first = default)
    cells: int = 4           # G: cells per side of the spatial partition
    dtype: str = "bf16"      # storage type of Q and K: "bf16", "f16" or "f32"
    salient_frac: float = 0.05
    salient_count: int = -1  # explicit count (overrides salient_frac when >= 0)
    clusters: int = 3        # 0 = uniformly scattered salient tokens
    shift_sigmas: float = 1.5
    neardup_frac: float = 0.0
    value_std: float = -1.0  # element std of Q/K; <0 means 1/sqrt(d)

    @property
    def num_visual(self) -> int:
        return self.grid_h * self.grid_w

    @property
    def lam(self) -> float:
        return float(self.lambdas[0])

    @property
    def sigma(self) -> float:
        return self.value_std if self.value_std > 0 else 1.0 / math.sqrt(self.head_dim)

    @property
    def num_salient(self) -> int:
        if self.salient_count >= 0:
            return self.salient_count
        return int(round(self.salient_frac * self.num_visual))

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2

    def q_shape(self, batch: int | None = None):
        b = self.batch if batch is None else batch
        return (b, self.num_layers, self.num_heads, self.num_text, self.head_dim)

    def k_shape(self, batch: int | None = None):
        b = self.batch if batch is None else batch
        return (b, self.num_layers, self.num_kv_heads, self.num_visual, self.head_dim)

    def bytes_per_image(self) -> int:
        q = self.num_layers * self.num_heads * self.num_text * self.head_dim
        k = self.num_layers * self.num_kv_heads * self.num_visual * self.head_dim
        return (q + k) * self.elem_bytes

    def replace(self, **kw) -> "Config":
        return dataclasses.replace(self, **kw)


# The five workloads.  Shapes: LLaVA-1.5-7B (32 heads x 128, 24x24 = 576 visual
# tokens); Qwen2-VL-7B (28 query heads over 4 KV heads, 32x32 grid); a 64x64
# high-resolution stress case.  G = 4 and lambda = 0.1 are the paper's defaults
# (Algorithm 1 inputs, Eq. 22 text).
CONFIGS: tuple = (
    Config("tiny", 0, batch=1, num_layers=2, num_heads=4, num_kv_heads=4, head_dim=64,
           num_text=16, grid_h=8, grid_w=8, keep=16, lambdas=(0.5,), dtype="f32",
           salient_count=4, clusters=0, shift_sigmas=2.0),
    Config("llava", 1, batch=64, num_layers=4, num_heads=32, num_kv_heads=32, head_dim=128,
           num_text=64, grid_h=24, grid_w=24, keep=128, lambdas=(0.1,)),
    Config("llava_aggressive", 2, batch=256, num_layers=4, num_heads=32, num_kv_heads=32,
           head_dim=128, num_text=64, grid_h=24, grid_w=24, keep=64,
           lambdas=(0.0, 0.25, 0.5, 1.0)),
    Config("qwen2vl_gqa", 3, batch=32, num_layers=4, num_heads=28, num_kv_heads=4, head_dim=128,
           num_text=96, grid_h=32, grid_w=32, keep=256, lambdas=(0.1,)),
    Config("hires", 4, batch=16, num_layers=6, num_heads=32, num_kv_heads=32, head_dim=128,
           num_text=128, grid_h=64, grid_w=64, keep=512, lambdas=(0.1,),
           salient_frac=0.02, clusters=8, neardup_frac=0.10),
)


def config_by_name(name: str) -> Config:
    for c in CONFIGS:
        if c.name == name:
            return c
    raise KeyError(f"unknown workload {name!r}; known: {[c.name for c in CONFIGS]}")


def heavy_tailed(base: Config, name: str = "heavy") -> Config:
    """A high-contrast variant: elements N(0, 2^2), salient keys shifted 4 sigma.

    At the 1/sqrt(d) scale of the standard workloads every token is nearly
    vacuous; this variant gives logits of O(1) spread so that tests can check the
    semantics (salient tokens surfacing) and exercise non-trivial masses.
    """
    return base.replace(name=name, config_id=100 + base.config_id, value_std=2.0,
                        shift_sigmas=4.0)


# ---------------------------------------------------------------------------
# bfloat16 storage
# ---------------------------------------------------------------------------

def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (round to nearest, ties to even); uint16 bits."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    bias = ((u >> 16) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + bias) >> 16).astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << 16).view(np.float32)


def _round_storage(x: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "bf16":
        return bf16_bits_to_f32(to_bf16_bits(x))
    if dtype == "f16":
        return x.astype(np.float16).astype(np.float32)
    return x


# ---------------------------------------------------------------------------
# salient tokens
# ---------------------------------------------------------------------------

def _cluster_tokens(rng: np.random.Generator, cfg: Config) -> np.ndarray:
    """|S| tokens in `clusters` clusters: centres are distinct uniform grid cells;
    cluster c takes floor(|S|/n_c) tokens (+1 for the first |S| mod n_c), the ones
    nearest to its centre by squared grid distance (ties by token index), skipping
    tokens another cluster already took."""
    n = cfg.num_visual
    total, nc = cfg.num_salient, cfg.clusters
    centres = rng.choice(n, size=nc, replace=False)
    rows, cols = np.divmod(np.arange(n), cfg.grid_w)
    taken = np.zeros(n, dtype=bool)
    out = []
    for c in range(nc):
        want = total // nc + (1 if c < total % nc else 0)
        cr, cc = divmod(int(centres[c]), cfg.grid_w)
        d2 = (rows - cr) ** 2 + (cols - cc) ** 2
        order = np.lexsort((np.arange(n), d2))
        got = 0
        for t in order:
            if got == want:
                break
            if not taken[t]:
                taken[t] = True
                out.append(int(t))
                got += 1
    return np.sort(np.array(out, dtype=np.int64))


def salient_set(rng: np.random.Generator, cfg: Config) -> np.ndarray:
    if cfg.num_salient == 0:
        return np.zeros(0, dtype=np.int64)
    if cfg.clusters <= 0:
        return np.sort(rng.choice(cfg.num_visual, size=cfg.num_salient, replace=False))
    return _cluster_tokens(rng, cfg)


def _neardup_sources(rng: np.random.Generator, cfg: Config, salient: np.ndarray):
    """Pick near-duplicate tokens among the non-salient ones and, for each, a
    uniformly random other token within Chebyshev distance 2 on the grid."""
    n = cfg.num_visual
    count = int(round(cfg.neardup_frac * n))
    if count == 0:
        return np.zeros(0, np.int64), np.zeros(0, np.int64)
    pool = np.setdiff1d(np.arange(n), salient)
    dups = np.sort(rng.choice(pool, size=count, replace=False))
    srcs = np.empty(count, dtype=np.int64)
    for i, t in enumerate(dups):
        r, c = divmod(int(t), cfg.grid_w)
        cand = [rr * cfg.grid_w + cc
                for rr in range(max(0, r - 2), min(cfg.grid_h, r + 3))
                for cc in range(max(0, c - 2), min(cfg.grid_w, c + 3))
                if not (rr == r and cc == c)]
        srcs[i] = cand[int(rng.integers(len(cand)))]
    return dups, srcs


# ---------------------------------------------------------------------------
# one image
# ---------------------------------------------------------------------------

def gen_image(cfg: Config, image_index: int, q_out: np.ndarray | None = None,
              k_out: np.ndarray | None = None):
    """Generate image `image_index` of workload `cfg`.

    Returns (Q, K, salient) with Q float32 [L, H, N_T, d], K float32
    [L, Hkv, N_V, d] (values exactly representable in the storage dtype) and the
    sorted salient token indices.
    """
    L, H, Hkv, d, nt, n = (cfg.num_layers, cfg.num_heads, cfg.num_kv_heads, cfg.head_dim,
                           cfg.num_text, cfg.num_visual)
    rng = np.random.Generator(np.random.Philox(
        np.random.SeedSequence([SEED_ROOT, cfg.config_id, int(image_index)])))
    sig = np.float32(cfg.sigma)
    q = q_out if q_out is not None else np.empty((L, H, nt, d), np.float32)
    k = k_out if k_out is not None else np.empty((L, Hkv, n, d), np.float32)
    rng.standard_normal(out=q, dtype=np.float32)
    q *= sig
    q[...] = _round_storage(q, cfg.dtype)
    rng.standard_normal(out=k, dtype=np.float32)
    k *= sig
    sal = salient_set(rng, cfg)
    if sal.size and cfg.shift_sigmas != 0.0:
        grp = H // Hkv
        for l in range(L):
            for g in range(Hkv):
                u = q[l, g * grp:(g + 1) * grp].astype(np.float64).mean(axis=(0, 1))
                nrm = np.linalg.norm(u)
                if nrm == 0.0:
                    continue
                shift = (cfg.shift_sigmas * float(sig) / nrm) * u
                k[l, g, sal, :] = (k[l, g, sal, :].astype(np.float64) + shift).astype(np.float32)
    dups, srcs = _neardup_sources(rng, cfg, sal)
    if dups.size:
        snap = k[:, :, srcs, :].copy()
        noise = rng.standard_normal(size=snap.shape, dtype=np.float32) * np.float32(0.01 * sig)
        k[:, :, dups, :] = snap + noise
    k[...] = _round_storage(k, cfg.dtype)
    return q, k, sal


def gen_batch(cfg: Config, images: Iterable[int] | None = None, threads: int | None = None):
    """Generate a batch (default: all cfg.batch images) with a thread pool.

    Returns (Q [B,L,H,N_T,d] f32, K [B,L,Hkv,N_V,d] f32, salient list)."""
    idx = list(range(cfg.batch)) if images is None else [int(i) for i in images]
    b = len(idx)
    q = np.empty(cfg.q_shape(b), np.float32)
    k = np.empty(cfg.k_shape(b), np.float32)
    sal = [None] * b
    if threads is None:
        threads = min(16, len(os.sched_getaffinity(0)))

    def one(j):
        _, _, s = gen_image(cfg, idx[j], q_out=q[j], k_out=k[j])
        sal[j] = s

    if b == 1 or threads <= 1:
        for j in range(b):
            one(j)
    else:
        with ThreadPoolExecutor(max_workers=threads) as ex:
            list(ex.map(one, range(b)))
    return q, k, sal


def storage_view(x: np.ndarray, dtype: str) -> np.ndarray:
    """The bits a device buffer should hold: uint16 bf16 bits, the float16 array or
    the float32 array."""
    if dtype == "bf16":
        return to_bf16_bits(x)
    if dtype == "f16":
        return np.ascontiguousarray(x, dtype=np.float16)
    return np.ascontiguousarray(x, dtype=np.float32)


# ---------------------------------------------------------------------------
# ragged batches: every image its own grid, text length and budget
# ---------------------------------------------------------------------------

@dataclasses.dataclass(frozen=True)
class RaggedConfig:
    """A ragged workload.  Image b's grid sides are drawn uniformly from
    grid_sides (rows and columns independently), its text-query count from
    num_text, and it keeps round(keep_frac * N_b) tokens (at least 1).  The head
    geometry, storage type and value recipe (salient clusters, shift) come from
    `base`; image b's tensors are gen_image of base with image b's sizes and this
    workload's config_id, so every image is reproducible on its own."""
    name: str
    config_id: int
    batch: int
    base: Config
    grid_sides: tuple        # (smallest, largest) side
    num_text: tuple          # (smallest, largest) N_T
    keep_frac: float


# Qwen2-VL-7B with dynamic resolution (Sec. 5: Qwen2-VL-7B's visual tokens come from
# native-resolution images): 28 query heads over 4 KV heads, grids from 16x16 to
# 40x40 patches (256-1600 tokens), prompts of 32-160 text tokens, 22.2 % of the
# tokens kept (the paper's -77.8 % setting for Qwen2-VL, Table 5).
RAGGED: tuple = (
    RaggedConfig("qwen2vl_dynamic", 5, batch=32,
                 base=CONFIGS[3].replace(name="qwen2vl_dynamic", config_id=5),
                 grid_sides=(16, 40), num_text=(32, 160), keep_frac=0.222),
)


def ragged_by_name(name: str) -> RaggedConfig:
    for c in RAGGED:
        if c.name == name:
            return c
    raise KeyError(f"unknown ragged workload {name!r}; known: {[c.name for c in RAGGED]}")


def ragged_dims(rc: RaggedConfig) -> list:
    """[(grid_h, grid_w, num_text, keep)] of every image, from the workload's own
    seeded stream."""
    rng = np.random.Generator(np.random.Philox(
        np.random.SeedSequence([SEED_ROOT, rc.config_id, 1 << 30])))
    lo, hi = rc.grid_sides
    out = []
    for _ in range(rc.batch):
        gh = int(rng.integers(lo, hi + 1))
        gw = int(rng.integers(lo, hi + 1))
        nt = int(rng.integers(rc.num_text[0], rc.num_text[1] + 1))
        keep = max(1, int(round(rc.keep_frac * gh * gw)))
        out.append((gh, gw, nt, keep))
    return out


def image_config(rc: RaggedConfig, dims: tuple) -> Config:
    gh, gw, nt, keep = dims
    return rc.base.replace(config_id=rc.config_id, grid_h=gh, grid_w=gw, num_text=nt, keep=keep)


def gen_ragged(rc: RaggedConfig, dims: list | None = None, threads: int | None = None):
    """Every image of a ragged workload: (list of Q_b [L,H,N_T,b,d] f32, list of
    K_b [L,Hkv,N_b,d] f32, list of salient sets, dims)."""
    dims = ragged_dims(rc) if dims is None else list(dims)
    out = [None] * len(dims)
    if threads is None:
        threads = min(16, len(os.sched_getaffinity(0)))

    def one(b):
        out[b] = gen_image(image_config(rc, dims[b]), b)

    if threads <= 1 or len(dims) == 1:
        for b in range(len(dims)):
            one(b)
    else:
        with ThreadPoolExecutor(max_workers=threads) as ex:
            list(ex.map(one, range(len(dims))))
    return [o[0] for o in out], [o[1] for o in out], [o[2] for o in out], dims

