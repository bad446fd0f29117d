"""ctypes binding of libe2s.so (the C ABI declared in include/e2s.h).

Argument marshalling only: every step of the scoring path runs in the library's
HIP kernels.  Two layers are exposed:

  * ``lib()``: the loaded ``ctypes.CDLL`` with argument and result types set, so
    the C entry points can be called directly with raw pointers;
  * functions with the C names minus the ``e2s_`` prefix (``score_heads``,
    ``head_reliability``, ``head_masses``, ``ds_combine_layers``,
    ``fuse_evidence``, ``spatial_select``, ``layer_reliability``, ``fuse_select``,
    ``prune``, ``prune_stage``, ``prune_ragged``, ``compact_tokens``) that take torch tensors on
    the GPU, allocate the outputs with torch, pass raw device pointers and the
    current torch stream, and raise ``E2SError`` on a non-zero status.

There is no fallback: if the library has not been built, importing the binding
raises ``ImportError``.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
import re
from typing import Optional

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libe2s.so")
HEADER = os.path.join(os.path.dirname(PKG), "include", "e2s.h")

# status codes (e2s_status)
OK, ERR_NULL_POINTER, ERR_BAD_SHAPE, ERR_BAD_PARAM, ERR_UNSUPPORTED, ERR_MISALIGNED, \
    ERR_WORKSPACE_TOO_SMALL, ERR_LAUNCH, ERR_SCRATCH_TOO_SMALL = range(9)
# E2S_NOALLOC_SCRATCH_BYTES: the static scratch of e2s_prune_noalloc
NOALLOC_SCRATCH_BYTES = 64 << 20
DTYPE_F32, DTYPE_BF16, DTYPE_F16 = 0, 1, 2
MEAN_LOGIT, MEAN_PROB = 0, 1
MODES = {"mean_logit": MEAN_LOGIT, "mean_prob": MEAN_PROB}
# e2s_variant: the full method and the ablation variants A1-A5
VARIANTS = {"full": 0, "a1_attention_topk": 1, "a2_no_head_reliability": 2,
            "a3_no_layer_fusion": 3, "a4_no_conflict_protection": 4, "a5_no_spatial_novelty": 5}


class Shape(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("num_layers", ctypes.c_int32),
                ("num_heads", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("num_text", ctypes.c_int32),
                ("grid_h", ctypes.c_int32), ("grid_w", ctypes.c_int32)]


class Params(ctypes.Structure):
    _fields_ = [("dtype", ctypes.c_int32), ("mode", ctypes.c_int32), ("scale", ctypes.c_float),
                ("cells", ctypes.c_int32), ("lam", ctypes.c_float), ("keep", ctypes.c_int32),
                ("variant", ctypes.c_int32)]


class Image(ctypes.Structure):
    """e2s_image: one image of a ragged batch (sizes and element offsets)."""
    _fields_ = [("grid_h", ctypes.c_int32), ("grid_w", ctypes.c_int32),
                ("num_text", ctypes.c_int32), ("keep", ctypes.c_int32),
                ("q_offset", ctypes.c_int64), ("k_offset", ctypes.c_int64),
                ("token_offset", ctypes.c_int64), ("keep_offset", ctypes.c_int64)]


class RaggedShape(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("num_layers", ctypes.c_int32),
                ("num_heads", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32)]


class CompactShape(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("rows", ctypes.c_int32),
                ("num_tokens", ctypes.c_int32), ("keep", ctypes.c_int32),
                ("channels", ctypes.c_int32), ("elem_bytes", ctypes.c_int32),
                ("src_stride", ctypes.c_int64 * 3), ("dst_stride", ctypes.c_int64 * 3)]


MAX_VIEW_LAYERS = 16


class QKViews(ctypes.Structure):
    """e2s_qk_views: per-layer base pointers and element strides of Q and K."""
    _fields_ = [("q", ctypes.c_void_p * MAX_VIEW_LAYERS), ("k", ctypes.c_void_p * MAX_VIEW_LAYERS),
                ("q_stride_image", ctypes.c_int64), ("q_stride_head", ctypes.c_int64),
                ("q_stride_text", ctypes.c_int64), ("k_stride_image", ctypes.c_int64),
                ("k_stride_head", ctypes.c_int64), ("k_stride_token", ctypes.c_int64)]


class E2SError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        msg = _LIB.e2s_status_string(status).decode() if _LIB is not None else str(status)
        super().__init__(f"{where}: {msg}")


_P = ctypes.c_void_p
_SH = ctypes.POINTER(Shape)
_PA = ctypes.POINTER(Params)
_SIGNATURES = {
    "e2s_score_heads": [_SH, _PA, _P, _P, _P, _P, _P],
    "e2s_head_reliability": [_SH, _P, _P, _P, _P],
    "e2s_head_masses": [_SH, _P, _P, _P, _P],
    "e2s_ds_combine_layers": [_SH, _P, _P, _P, _P, _P],
    "e2s_fuse_evidence": [_SH, _P, _P, _P, _P, _P],
    "e2s_spatial_select": [_SH, _PA, _P, _P, _P, _P, _P],
    "e2s_layer_reliability": [_SH, _PA, _P, _P, _P, ctypes.c_size_t, _P, _P, _P],
    "e2s_fuse_select": [_SH, _PA, _P, _P, _P, _P, _P, _P],
    "e2s_prune_workspace_size": [_SH, _PA, ctypes.POINTER(ctypes.c_size_t)],
    "e2s_prune": [_SH, _PA, _P, _P, _P, ctypes.c_size_t, _P, _P, _P, _P],
    "e2s_prune_stage": [_SH, _PA, ctypes.c_int32, _P, _P, _P, _P, _P, ctypes.c_size_t, _P, _P,
                        _P, _P],
    "e2s_prune_ragged_workspace_size": [ctypes.POINTER(RaggedShape), _P,
                                        ctypes.POINTER(ctypes.c_size_t)],
    "e2s_prune_ragged": [ctypes.POINTER(RaggedShape), _PA, _P, _P, _P, _P, _P, ctypes.c_size_t,
                         _P, _P, _P, _P],
    "e2s_compact_tokens": [ctypes.POINTER(CompactShape), _P, _P, _P, _P],
    "e2s_prune_views": [_SH, _PA, ctypes.POINTER(QKViews), _P, ctypes.c_size_t, _P, _P, _P, _P],
    "e2s_prune_noalloc": [_SH, _PA, _P, _P, _P, _P, _P, _P],
    "e2s_read_probe": [_P, ctypes.c_size_t, ctypes.c_int32, _P, _P],
    "e2s_status_string": [ctypes.c_int],
    "e2s_abi_version": [],
}


def _load() -> ctypes.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with "
                          "`python paper_2608_23253_amd/build.py` (or __graft_entry__.build())")
    # Device memory and streams come from torch, whose wheel ships its own HIP
    # runtime (libamdhip64.so, libhsa-runtime64.so).  Load it before the library:
    # the library's libamdhip64.so.7 dependency then binds to that runtime.  Loaded
    # the other way round, the process would hold two HIP runtimes that do not
    # share device state (kernel attributes set through one fail on the other).
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    so = ctypes.CDLL(LIB_PATH)
    for name, args in _SIGNATURES.items():
        fn = getattr(so, name)
        fn.argtypes = args
        fn.restype = ctypes.c_int
    so.e2s_status_string.restype = ctypes.c_char_p
    so.e2s_abi_version.restype = ctypes.c_int32
    return so


_LIB: Optional[ctypes.CDLL] = _load()


def lib() -> ctypes.CDLL:
    return _LIB


def header_entry_points(path: str = HEADER) -> list:
    """Names of the functions include/e2s.h declares."""
    with open(path) as f:
        text = f.read()
    return sorted(set(re.findall(r"\b(e2s_[a-z_]+)\s*\(", text)))


# ---------------------------------------------------------------------------
# torch-facing wrappers
# ---------------------------------------------------------------------------

@dataclasses.dataclass
class Geometry:
    grid_h: int
    grid_w: int


def _torch():
    import torch
    return torch


def _check(t, name, dtype=None, ndim=None, contiguous=True):
    torch = _torch()
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be a GPU tensor (got {t.device})")
    if contiguous and not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype} (got {t.dtype})")
    if ndim is not None and t.dim() != ndim:
        raise ValueError(f"{name} must have {ndim} dimensions (got {t.dim()})")


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _device_of(*tensors):
    """The one device of the given tensors (None entries skipped)."""
    devs = {t.device for t in tensors if t is not None}
    if len(devs) != 1:
        raise ValueError(f"all tensors of a call must be on one GPU (got {sorted(map(str, devs))})")
    return devs.pop()


def _launch(where: str, tensors, fn, *args, stream=None):
    """fn(*args, stream) with the tensors' device current (kernels are launched on
    that device), on its current stream unless one is given; raises on a status."""
    torch = _torch()
    dev = _device_of(*tensors)
    with torch.cuda.device(dev):
        st = torch.cuda.current_stream(dev).cuda_stream if stream is None else stream
        _raise(fn(*args, st), where)


def _raise(status: int, where: str):
    if status != OK:
        raise E2SError(status, where)


def make_shape(batch, num_layers, num_heads, num_kv_heads, head_dim, num_text, grid_h,
               grid_w) -> Shape:
    return Shape(batch, num_layers, num_heads, num_kv_heads, head_dim, num_text, grid_h, grid_w)


def make_params(dtype=DTYPE_BF16, mode="mean_logit", scale=0.0, cells=4, lam=0.1,
                keep=0, variant="full") -> Params:
    m = MODES[mode] if isinstance(mode, str) else int(mode)
    v = VARIANTS[variant] if isinstance(variant, str) else int(variant)
    return Params(int(dtype), m, float(scale), int(cells), float(lam), int(keep), v)


def shape_from(q, k, grid_h: int, grid_w: int) -> Shape:
    """Shape of a call from Q [B,L,H,N_T,d] and K [B,L,Hkv,N,d]."""
    if q.dim() != 5 or k.dim() != 5:
        raise ValueError("q must be [B,L,H,N_T,d] and k [B,L,Hkv,N,d]")
    B, L, H, NT, D = q.shape
    if k.shape[0] != B or k.shape[1] != L or k.shape[4] != D:
        raise ValueError(f"q {tuple(q.shape)} and k {tuple(k.shape)} disagree")
    if k.shape[3] != grid_h * grid_w:
        raise ValueError(f"k has {k.shape[3]} visual tokens, grid {grid_h}x{grid_w}")
    return make_shape(B, L, H, k.shape[2], D, NT, grid_h, grid_w)


def _dtype_code(t) -> int:
    torch = _torch()
    if t.dtype == torch.bfloat16:
        return DTYPE_BF16
    if t.dtype == torch.float32:
        return DTYPE_F32
    if t.dtype == torch.float16:
        return DTYPE_F16
    raise TypeError(f"q/k must be bfloat16, float16 or float32 (got {t.dtype})")


def score_heads(q, k, grid_h: int, grid_w: int, mode="mean_logit", scale: float = 0.0,
                want_r: bool = False):
    """Eq. 1, 8, 9: returns (support_c [B,L,H,N] = p - 1/2, r or None)."""
    torch = _torch()
    _check(q, "q", ndim=5)
    _check(k, "k", dtype=q.dtype, ndim=5)
    sh = shape_from(q, k, grid_h, grid_w)
    pa = make_params(_dtype_code(q), mode, scale)
    n = grid_h * grid_w
    e = torch.empty((sh.batch, sh.num_layers, sh.num_heads, n), device=q.device,
                    dtype=torch.float32)
    r = torch.empty_like(e) if want_r else None
    _launch("e2s_score_heads", (q, k, e, r), _LIB.e2s_score_heads, ctypes.byref(sh),
            ctypes.byref(pa), q.data_ptr(), k.data_ptr(), e.data_ptr(), _ptr(r))
    return e, r


def _shape_from_support(e, grid_h, grid_w) -> Shape:
    B, L, H, N = e.shape
    if N != grid_h * grid_w:
        raise ValueError("support_c's last dimension must be grid_h*grid_w")
    # num_kv_heads, head_dim and num_text do not enter the evidence stages
    return make_shape(B, L, H, 1, 128, 1, grid_h, grid_w)


def head_reliability(support_c, grid_h: int, grid_w: int):
    """Eq. 10: (rho, pbar_c) each [B, L, N]."""
    torch = _torch()
    _check(support_c, "support_c", dtype=torch.float32, ndim=4)
    sh = _shape_from_support(support_c, grid_h, grid_w)
    B, L, H, N = support_c.shape
    rho = torch.empty((B, L, N), device=support_c.device, dtype=torch.float32)
    pbar = torch.empty_like(rho)
    _launch("e2s_head_reliability", (support_c,), _LIB.e2s_head_reliability, ctypes.byref(sh),
            support_c.data_ptr(), rho.data_ptr(), pbar.data_ptr())
    return rho, pbar


def head_masses(rho, pbar_c, grid_h: int, grid_w: int):
    """Eq. 11: mass [B, L, N, 3] (I, U, Theta)."""
    torch = _torch()
    _check(rho, "rho", dtype=torch.float32, ndim=3)
    _check(pbar_c, "pbar_c", dtype=torch.float32, ndim=3)
    B, L, N = rho.shape
    sh = make_shape(B, L, 1, 1, 128, 1, grid_h, grid_w)
    mass = torch.empty((B, L, N, 3), device=rho.device, dtype=torch.float32)
    _launch("e2s_head_masses", (rho, pbar_c), _LIB.e2s_head_masses, ctypes.byref(sh),
            rho.data_ptr(), pbar_c.data_ptr(), mass.data_ptr())
    return mass


def ds_combine_layers(mass, grid_h: int, grid_w: int, want_fused=True, want_conflict=True):
    """Eq. 12-19: (fused [B,N,3] or None, conflict [B,L,N] or None, prio_c [B,N])."""
    torch = _torch()
    _check(mass, "mass", dtype=torch.float32, ndim=4)
    B, L, N, _ = mass.shape
    sh = make_shape(B, L, 1, 1, 128, 1, grid_h, grid_w)
    dev = mass.device
    fused = torch.empty((B, N, 3), device=dev, dtype=torch.float32) if want_fused else None
    conflict = torch.empty((B, L, N), device=dev, dtype=torch.float32) if want_conflict else None
    prio = torch.empty((B, N), device=dev, dtype=torch.float32)
    _launch("e2s_ds_combine_layers", (mass,), _LIB.e2s_ds_combine_layers, ctypes.byref(sh),
            mass.data_ptr(), _ptr(fused), _ptr(conflict), prio.data_ptr())
    return fused, conflict, prio


def fuse_evidence(support_c, grid_h: int, grid_w: int, want_fused=True, want_conflict=True):
    """Eq. 10-19 in one pass: (fused or None, conflict or None, prio_c)."""
    torch = _torch()
    _check(support_c, "support_c", dtype=torch.float32, ndim=4)
    sh = _shape_from_support(support_c, grid_h, grid_w)
    B, L, H, N = support_c.shape
    dev = support_c.device
    fused = torch.empty((B, N, 3), device=dev, dtype=torch.float32) if want_fused else None
    conflict = torch.empty((B, L, N), device=dev, dtype=torch.float32) if want_conflict else None
    prio = torch.empty((B, N), device=dev, dtype=torch.float32)
    _launch("e2s_fuse_evidence", (support_c,), _LIB.e2s_fuse_evidence, ctypes.byref(sh),
            support_c.data_ptr(), _ptr(fused), _ptr(conflict), prio.data_ptr())
    return fused, conflict, prio


def spatial_select(prio_c, grid_h: int, grid_w: int, keep: int, cells: int = 4,
                   lam: float = 0.1, want_adj=False, want_rep=False):
    """Eq. 20-23: (keep_idx [B,K] int32 ascending, adj_c [B,N] f64 or None, is_rep or None)."""
    torch = _torch()
    _check(prio_c, "prio_c", dtype=torch.float32, ndim=2)
    B, N = prio_c.shape
    sh = make_shape(B, 1, 1, 1, 128, 1, grid_h, grid_w)
    pa = make_params(cells=cells, lam=lam, keep=keep)
    dev = prio_c.device
    out = torch.empty((B, keep), device=dev, dtype=torch.int32)
    adj = torch.empty((B, N), device=dev, dtype=torch.float64) if want_adj else None
    rep = torch.empty((B, N), device=dev, dtype=torch.uint8) if want_rep else None
    _launch("e2s_spatial_select", (prio_c,), _LIB.e2s_spatial_select, ctypes.byref(sh),
            ctypes.byref(pa), prio_c.data_ptr(), out.data_ptr() if keep > 0 else None,
            _ptr(adj), _ptr(rep))
    return out, adj, rep


def layer_reliability(q, k, grid_h: int, grid_w: int, mode="mean_logit", scale: float = 0.0,
                      workspace=None):
    """Eq. 1, 8-10 in one call: (rho, pbar_c) each [B, L, N].  workspace: a uint8
    device tensor of at least workspace_size() bytes (allocated here if None)."""
    torch = _torch()
    _check(q, "q", ndim=5)
    _check(k, "k", dtype=q.dtype, ndim=5)
    sh = shape_from(q, k, grid_h, grid_w)
    pa = make_params(_dtype_code(q), mode, scale)
    if workspace is None:
        workspace = torch.empty(workspace_size(sh, pa), device=q.device, dtype=torch.uint8)
    B, L, N = sh.batch, sh.num_layers, grid_h * grid_w
    rho = torch.empty((B, L, N), device=q.device, dtype=torch.float32)
    pbar = torch.empty_like(rho)
    _launch("e2s_layer_reliability", (q, k, workspace), _LIB.e2s_layer_reliability,
            ctypes.byref(sh), ctypes.byref(pa), q.data_ptr(), k.data_ptr(), workspace.data_ptr(),
            workspace.numel(), rho.data_ptr(), pbar.data_ptr())
    return rho, pbar


def fuse_select(rho, pbar_c, grid_h: int, grid_w: int, keep: int, cells: int = 4,
                lam: float = 0.1, want_fused=False, want_prio=False, variant="full"):
    """Eq. 11-23 in one call: (keep_idx [B,K], fused [B,N,3] or None, prio_c [B,N] or None)."""
    torch = _torch()
    _check(rho, "rho", dtype=torch.float32, ndim=3)
    _check(pbar_c, "pbar_c", dtype=torch.float32, ndim=3)
    B, L, N = rho.shape
    sh = make_shape(B, L, 1, 1, 128, 1, grid_h, grid_w)
    pa = make_params(cells=cells, lam=lam, keep=keep, variant=variant)
    dev = rho.device
    out = torch.empty((B, keep), device=dev, dtype=torch.int32)
    fused = torch.empty((B, N, 3), device=dev, dtype=torch.float32) if want_fused else None
    prio = torch.empty((B, N), device=dev, dtype=torch.float32) if want_prio else None
    _launch("e2s_fuse_select", (rho, pbar_c), _LIB.e2s_fuse_select, ctypes.byref(sh),
            ctypes.byref(pa), rho.data_ptr(), pbar_c.data_ptr(),
            out.data_ptr() if keep > 0 else None, _ptr(fused), _ptr(prio))
    return out, fused, prio


def workspace_size(shape: Shape, params: Params) -> int:
    n = ctypes.c_size_t(0)
    _raise(_LIB.e2s_prune_workspace_size(ctypes.byref(shape), ctypes.byref(params),
                                         ctypes.byref(n)), "e2s_prune_workspace_size")
    return int(n.value)


class Pruner:
    """Holds the shape, params and workspace of repeated e2s_prune calls."""

    def __init__(self, q, k, grid_h: int, grid_w: int, keep: int, cells: int = 4,
                 lam: float = 0.1, mode="mean_logit", scale: float = 0.0, variant="full"):
        torch = _torch()
        _check(q, "q", ndim=5)
        _check(k, "k", dtype=q.dtype, ndim=5)
        self.shape = shape_from(q, k, grid_h, grid_w)
        self.params = make_params(_dtype_code(q), mode, scale, cells, lam, keep, variant)
        self.device = q.device
        self.workspace = torch.empty(workspace_size(self.shape, self.params), device=q.device,
                                     dtype=torch.uint8)
        self.keep_idx = torch.empty((self.shape.batch, keep), device=q.device, dtype=torch.int32)

    def __call__(self, q, k, fused=None, prio_c=None, stream: Optional[int] = None):
        if tuple(q.shape) != (self.shape.batch, self.shape.num_layers, self.shape.num_heads,
                              self.shape.num_text, self.shape.head_dim):
            raise ValueError("q does not match the Pruner's shape")
        if tuple(k.shape) != (self.shape.batch, self.shape.num_layers, self.shape.num_kv_heads,
                              self.shape.grid_h * self.shape.grid_w, self.shape.head_dim):
            raise ValueError("k does not match the Pruner's shape")
        if q.dtype != k.dtype or _dtype_code(q) != self.params.dtype:
            raise TypeError("q/k dtype does not match the Pruner's")
        _launch("e2s_prune", (q, k, fused, prio_c, self.workspace), _LIB.e2s_prune,
                ctypes.byref(self.shape), ctypes.byref(self.params), q.data_ptr(), k.data_ptr(),
                self.workspace.data_ptr(), self.workspace.numel(),
                self.keep_idx.data_ptr() if self.params.keep > 0 else None, _ptr(fused),
                _ptr(prio_c), stream=stream)
        return self.keep_idx


def prune(q, k, grid_h: int, grid_w: int, keep: int, cells: int = 4, lam: float = 0.1,
          mode="mean_logit", scale: float = 0.0, want_fused=False, want_prio=False,
          variant="full"):
    """The whole path: (keep_idx [B,K], fused [B,N,3] or None, prio_c [B,N] or None)."""
    torch = _torch()
    p = Pruner(q, k, grid_h, grid_w, keep, cells, lam, mode, scale, variant)
    B, N = p.shape.batch, grid_h * grid_w
    fused = torch.empty((B, N, 3), device=q.device, dtype=torch.float32) if want_fused else None
    prio = torch.empty((B, N), device=q.device, dtype=torch.float32) if want_prio else None
    idx = p(q, k, fused, prio)
    return idx, fused, prio


def prune_noalloc(q, k, grid_h: int, grid_w: int, keep: int, cells: int = 4, lam: float = 0.1,
                  mode="mean_logit", scale: float = 0.0, keep_idx=None, fused=None, prio_c=None,
                  variant="full"):
    """e2s_prune with the library's static scratch as its workspace (e2s_prune_noalloc):
    (keep_idx [B,K], fused [B,N,3] or None, prio_c [B,N] or None).  Output tensors may
    be passed in; only those not given are allocated here, by torch."""
    torch = _torch()
    _check(q, "q", ndim=5)
    _check(k, "k", dtype=q.dtype, ndim=5)
    sh = shape_from(q, k, grid_h, grid_w)
    pa = make_params(_dtype_code(q), mode, scale, cells, lam, keep, variant)
    if keep_idx is None:
        keep_idx = torch.empty((sh.batch, keep), device=q.device, dtype=torch.int32)
    _launch("e2s_prune_noalloc", (q, k, keep_idx, fused, prio_c), _LIB.e2s_prune_noalloc,
            ctypes.byref(sh), ctypes.byref(pa), q.data_ptr(), k.data_ptr(),
            keep_idx.data_ptr() if keep > 0 else None, _ptr(fused), _ptr(prio_c))
    return keep_idx, fused, prio_c


def read_probe(buf, workgroups: int, sink, stream: Optional[int] = None):
    """e2s_read_probe over the bytes of the contiguous tensor `buf` (a measurement
    helper: a streaming read, timed by the caller); sink: a 4-byte device tensor."""
    _check(buf, "buf")
    _check(sink, "sink")
    nbytes = buf.numel() * buf.element_size()
    _launch("e2s_read_probe", (buf, sink), _LIB.e2s_read_probe, buf.data_ptr(), nbytes,
            int(workgroups), sink.data_ptr(), stream=stream)


def qk_views(q_layers, k_layers) -> QKViews:
    """e2s_qk_views of per-layer tensors q_layers[l] [B, H, N_T, d] and k_layers[l]
    [B, Hkv, N, d]: any views (slices of a key/value cache, token-major projection
    outputs) with the last dimension contiguous and the same strides in every
    layer.  The tensors must stay alive while the call's kernels run."""
    if len(q_layers) != len(k_layers) or not 1 <= len(q_layers) <= MAX_VIEW_LAYERS:
        raise ValueError(f"need 1..{MAX_VIEW_LAYERS} layers of q and of k")
    v = QKViews()
    for name, ts in (("q", q_layers), ("k", k_layers)):
        st = ts[0].stride()
        for t in ts:
            _check(t, name, dtype=q_layers[0].dtype, ndim=4, contiguous=False)
            if t.stride() != st or t.stride(3) != 1 or t.shape != ts[0].shape:
                raise ValueError(f"{name} views need one shape, one set of strides, and "
                                 "contiguous rows")
    for l, (tq, tk) in enumerate(zip(q_layers, k_layers)):
        v.q[l] = tq.data_ptr()
        v.k[l] = tk.data_ptr()
    v.q_stride_image, v.q_stride_head, v.q_stride_text = q_layers[0].stride()[:3]
    v.k_stride_image, v.k_stride_head, v.k_stride_token = k_layers[0].stride()[:3]
    return v


def prune_views(q_layers, k_layers, grid_h: int, grid_w: int, keep: int, cells: int = 4,
                lam: float = 0.1, mode="mean_logit", scale: float = 0.0, want_fused=False,
                want_prio=False, variant="full"):
    """e2s_prune_views on per-layer views (see qk_views): (keep_idx, fused, prio_c)
    as from prune() on packed copies."""
    torch = _torch()
    q0, k0 = q_layers[0], k_layers[0]
    B, H, NT, D = q0.shape
    Hkv, N = k0.shape[1], k0.shape[2]
    if k0.shape[0] != B or k0.shape[3] != D or N != grid_h * grid_w:
        raise ValueError("k views do not match q views and the grid")
    views = qk_views(q_layers, k_layers)
    shape = make_shape(B, len(q_layers), H, Hkv, D, NT, grid_h, grid_w)
    params = make_params(_dtype_code(q0), mode, scale, cells, lam, keep, variant)
    ws = torch.empty(workspace_size(shape, params), device=q0.device, dtype=torch.uint8)
    out = torch.empty((B, keep), device=q0.device, dtype=torch.int32)
    fused = torch.empty((B, N, 3), device=q0.device, dtype=torch.float32) if want_fused else None
    prio = torch.empty((B, N), device=q0.device, dtype=torch.float32) if want_prio else None
    _launch("e2s_prune_views", (*q_layers, *k_layers), _LIB.e2s_prune_views, ctypes.byref(shape),
            ctypes.byref(params), ctypes.byref(views), ws.data_ptr(), ws.numel(),
            out.data_ptr() if keep > 0 else None, _ptr(fused), _ptr(prio))
    return out, fused, prio


class StagePruner:
    """Repeated calls of one pruning operation of a progressive schedule
    (e2s_prune_stage): the original grid, the operation's layers and its budget."""

    def __init__(self, q, k, grid_h: int, grid_w: int, keep: int, cells: int = 4,
                 lam: float = 0.1, mode="mean_logit", scale: float = 0.0, variant="full"):
        torch = _torch()
        _check(q, "q", ndim=5)
        _check(k, "k", dtype=q.dtype, ndim=5)
        B, L, H, NT, D = q.shape
        self.num_cand = int(k.shape[3])
        if self.num_cand > grid_h * grid_w:
            raise ValueError("more candidates than grid positions")
        self.shape = make_shape(B, L, H, k.shape[2], D, NT, grid_h, grid_w)
        self.params = make_params(_dtype_code(q), mode, scale, cells, lam, keep, variant)
        self.device = q.device
        self.workspace = torch.empty(workspace_size(self.shape, self.params), device=q.device,
                                     dtype=torch.uint8)
        self.keep_idx = torch.empty((B, keep), device=q.device, dtype=torch.int32)
        self.keep_pos = torch.empty((B, keep), device=q.device, dtype=torch.int32)
        self.m_out = torch.empty((B, keep, 3), device=q.device, dtype=torch.float32)

    def __call__(self, q, k, cand_pos=None, m_prev=None, stream: Optional[int] = None):
        torch = _torch()
        _check(q, "q", ndim=5)
        _check(k, "k", dtype=q.dtype, ndim=5)
        B, N = self.shape.batch, self.num_cand
        sh = self.shape
        if tuple(q.shape) != (B, sh.num_layers, sh.num_heads, sh.num_text, sh.head_dim):
            raise ValueError("q does not match the StagePruner's shape")
        if tuple(k.shape) != (B, sh.num_layers, sh.num_kv_heads, N, sh.head_dim):
            raise ValueError("k does not match the StagePruner's candidates")
        if _dtype_code(q) != self.params.dtype:
            raise TypeError("q/k dtype does not match the StagePruner's")
        if cand_pos is not None:
            _check(cand_pos, "cand_pos", dtype=torch.int32, ndim=2)
            if tuple(cand_pos.shape) != (B, N):
                raise ValueError("cand_pos must be [B, num_cand]")
        if m_prev is not None:
            _check(m_prev, "m_prev", dtype=torch.float32, ndim=3)
            if tuple(m_prev.shape) != (B, N, 3):
                raise ValueError("m_prev must be [B, num_cand, 3]")
        K = self.params.keep
        _launch("e2s_prune_stage", (q, k, cand_pos, m_prev, self.workspace), _LIB.e2s_prune_stage,
                ctypes.byref(self.shape), ctypes.byref(self.params), N, q.data_ptr(), k.data_ptr(),
                _ptr(cand_pos), _ptr(m_prev), self.workspace.data_ptr(), self.workspace.numel(),
                self.keep_idx.data_ptr() if K > 0 else None,
                self.keep_pos.data_ptr() if K > 0 else None,
                self.m_out.data_ptr() if K > 0 else None, stream=stream)
        return self.keep_idx, self.keep_pos, self.m_out


def prune_stage(q, k, grid_h: int, grid_w: int, keep: int, cand_pos=None, m_prev=None,
                cells: int = 4, lam: float = 0.1, mode="mean_logit", scale: float = 0.0,
                variant="full"):
    """One pruning operation over the candidates whose keys k [B,L,Hkv,N_l,d] holds:
    (keep_idx [B,K] candidate indices, keep_pos [B,K] raster positions,
    m_out [B,K,3] fused masses for the next operation)."""
    sp = StagePruner(q, k, grid_h, grid_w, keep, cells, lam, mode, scale, variant)
    idx, pos, m = sp(q, k, cand_pos, m_prev)
    return idx, pos, m


# ---------------------------------------------------------------------------
# ragged batches (e2s_prune_ragged)
# ---------------------------------------------------------------------------

def packed_images(dims, num_layers: int, num_heads: int, num_kv_heads: int, head_dim: int):
    """e2s_image records of images packed one after the other: dims is a list of
    (grid_h, grid_w, num_text, keep).  Returns (ctypes array, total Q elements,
    total K elements, total tokens, total kept)."""
    arr = (Image * len(dims))()
    qo = ko = to = kk = 0
    for i, (gh, gw, nt, keep) in enumerate(dims):
        n = gh * gw
        arr[i] = Image(gh, gw, nt, keep, qo, ko, to, kk)
        qo += num_layers * num_heads * nt * head_dim
        ko += num_layers * num_kv_heads * n * head_dim
        to += n
        kk += keep
    return arr, qo, ko, to, kk


class RaggedPruner:
    """Repeated e2s_prune_ragged calls over one ragged batch layout.

    images: a ctypes array of Image records (see packed_images); the records are
    copied once to a device table.  q and k are flat device tensors holding every
    image's blocks at the records' offsets."""

    def __init__(self, images, num_layers: int, num_heads: int, num_kv_heads: int,
                 head_dim: int, device, dtype=DTYPE_BF16, mode="mean_logit", scale: float = 0.0,
                 cells: int = 4, lam: float = 0.1, variant="full"):
        torch = _torch()
        self.images = images
        self.shape = RaggedShape(len(images), num_layers, num_heads, num_kv_heads, head_dim)
        self.params = make_params(dtype, mode, scale, cells, lam, 0, variant)
        self.device = torch.device(device)
        raw = bytes(images)
        host = torch.frombuffer(bytearray(raw), dtype=torch.uint8)
        self.images_dev = host.to(self.device)
        n = ctypes.c_size_t(0)
        _raise(_LIB.e2s_prune_ragged_workspace_size(ctypes.byref(self.shape),
                                                    ctypes.addressof(images), ctypes.byref(n)),
               "e2s_prune_ragged_workspace_size")
        self.workspace = torch.empty(int(n.value), device=self.device, dtype=torch.uint8)
        self.tokens = max(im.token_offset + im.grid_h * im.grid_w for im in images)
        self.kept = max([im.keep_offset + im.keep for im in images if im.keep > 0] or [0])
        self.keep_idx = torch.empty(max(self.kept, 1), device=self.device, dtype=torch.int32)

    def __call__(self, q, k, fused=None, prio_c=None, stream: Optional[int] = None):
        torch = _torch()
        _check(q, "q")
        _check(k, "k", dtype=q.dtype)
        if _dtype_code(q) != self.params.dtype:
            raise TypeError("q/k dtype does not match the RaggedPruner's")
        for t, name, n in ((fused, "fused", 3 * self.tokens), (prio_c, "prio_c", self.tokens)):
            if t is not None:
                _check(t, name, dtype=torch.float32)
                if t.numel() < n:
                    raise ValueError(f"{name} holds fewer than {n} values")
        _launch("e2s_prune_ragged", (q, k, fused, prio_c, self.workspace), _LIB.e2s_prune_ragged,
                ctypes.byref(self.shape), ctypes.byref(self.params),
                ctypes.addressof(self.images), self.images_dev.data_ptr(), q.data_ptr(),
                k.data_ptr(), self.workspace.data_ptr(), self.workspace.numel(),
                self.keep_idx.data_ptr() if self.kept > 0 else None, _ptr(fused), _ptr(prio_c),
                stream=stream)
        return self.keep_idx


def prune_ragged(q, k, images, num_layers: int, num_heads: int, num_kv_heads: int,
                 head_dim: int, cells: int = 4, lam: float = 0.1, mode="mean_logit",
                 scale: float = 0.0, want_fused=False, want_prio=False, variant="full"):
    """The whole path over a ragged batch: (keep_idx [sum K_b] int32, fused
    [tokens, 3] or None, prio_c [tokens] or None), image b's entries at its
    record's keep_offset / token_offset."""
    torch = _torch()
    p = RaggedPruner(images, num_layers, num_heads, num_kv_heads, head_dim, q.device,
                     _dtype_code(q), mode, scale, cells, lam, variant)
    fused = (torch.empty((p.tokens, 3), device=q.device, dtype=torch.float32)
             if want_fused else None)
    prio = torch.empty(p.tokens, device=q.device, dtype=torch.float32) if want_prio else None
    idx = p(q, k, fused, prio)
    return idx[:p.kept], fused, prio


# ---------------------------------------------------------------------------
# token compaction (e2s_compact_tokens)
# ---------------------------------------------------------------------------

def compact_tokens(src, keep_idx, out=None):
    """Gather the kept tokens' vectors: src [B, R, N, C] (any strides, channels
    contiguous, e.g. a slice of a key/value cache), keep_idx [B, K] int32 ->
    out [B, R, K, C] with out[b, r, j] = src[b, r, keep_idx[b, j]]."""
    torch = _torch()
    if not isinstance(src, torch.Tensor) or src.device.type != "cuda" or src.dim() != 4:
        raise ValueError("src must be a 4-D GPU tensor [B, R, N, C]")
    if src.stride(3) != 1:
        raise ValueError("src's channels must be contiguous")
    if src.dtype not in (torch.bfloat16, torch.float16, torch.float32):
        raise TypeError("src must be bfloat16, float16 or float32")
    _check(keep_idx, "keep_idx", dtype=torch.int32, ndim=2)
    B, R, N, C = src.shape
    if keep_idx.shape[0] != B:
        raise ValueError("keep_idx must be [B, K]")
    K = keep_idx.shape[1]
    if out is None:
        out = torch.empty((B, R, K, C), device=src.device, dtype=src.dtype)
    if tuple(out.shape) != (B, R, K, C) or out.dtype != src.dtype or out.stride(3) != 1:
        raise ValueError("out must be [B, R, K, C] of src's dtype with contiguous channels")
    sh = CompactShape(B, R, N, K, C, src.element_size(),
                      (ctypes.c_int64 * 3)(*src.stride()[:3]),
                      (ctypes.c_int64 * 3)(*out.stride()[:3]))
    _launch("e2s_compact_tokens", (keep_idx, src), _LIB.e2s_compact_tokens, ctypes.byref(sh),
            keep_idx.data_ptr(), src.data_ptr(), out.data_ptr())
    return out

