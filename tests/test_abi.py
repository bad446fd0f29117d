"""C-ABI checks that need no GPU: the library loads, exports every entry point the
header declares, and rejects invalid calls on the host before any launch.

Every call below is invalid in exactly one way, so it returns before it touches
the HIP runtime; the fake device addresses are never dereferenced.
"""
import ctypes

import pytest

from paper_2608_23253_amd import _lib as L

lib = L.lib()
A = 1 << 20          # a fake, 256-byte aligned device address (never dereferenced)


def good_shape(**kw):
    s = dict(batch=2, num_layers=3, num_heads=4, num_kv_heads=2, head_dim=64, num_text=5,
             grid_h=6, grid_w=7)
    s.update(kw)
    return L.make_shape(**s)


def good_params(**kw):
    p = dict(dtype=L.DTYPE_BF16, mode="mean_logit", scale=0.0, cells=3, lam=0.1, keep=10)
    p.update(kw)
    return L.make_params(**p)


def score(shape, params, q=A, k=A, e=A, r=None):
    return lib.e2s_score_heads(ctypes.byref(shape) if shape is not None else None,
                               ctypes.byref(params) if params is not None else None,
                               q, k, e, r, None)


def select(shape, params, c=A, out=A, adj=None, rep=None):
    return lib.e2s_spatial_select(ctypes.byref(shape), ctypes.byref(params), c, out, adj, rep,
                                  None)


def prune(shape, params, q=A, k=A, ws=A, ws_bytes=None, out=A):
    if ws_bytes is None:
        ws_bytes = L.workspace_size(shape, params)
    return lib.e2s_prune(ctypes.byref(shape), ctypes.byref(params), q, k, ws, ws_bytes, out,
                         None, None, None)


def layer_rel(shape, params, q=A, k=A, ws=A, ws_bytes=None, rho=A, pbar=A):
    if ws_bytes is None:
        ws_bytes = L.workspace_size(shape, params)
    return lib.e2s_layer_reliability(ctypes.byref(shape), ctypes.byref(params), q, k, ws,
                                     ws_bytes, rho, pbar, None)


def fuse_sel(shape, params, rho=A, pbar=A, out=A, fused=None, prio=None):
    return lib.e2s_fuse_select(ctypes.byref(shape), ctypes.byref(params), rho, pbar, out, fused,
                               prio, None)


def stage(shape, params, ncand, q=A, k=A, pos=A, mprev=None, ws=A, ws_bytes=None, out=A,
          kpos=None, mout=None):
    if ws_bytes is None:
        ws_bytes = L.workspace_size(shape, params)
    return lib.e2s_prune_stage(ctypes.byref(shape), ctypes.byref(params), ncand, q, k, pos, mprev,
                               ws, ws_bytes, out, kpos, mout, None)


def test_exports_every_declared_entry_point():
    names = L.header_entry_points()
    assert len(names) == 19
    for n in names:
        assert hasattr(lib, n), n
    assert lib.e2s_abi_version() == 9


def test_status_strings():
    for code in range(9):
        s = lib.e2s_status_string(code).decode()
        assert s.startswith("E2S_")
    assert b"unknown" in lib.e2s_status_string(99)


@pytest.mark.parametrize("field,value,expect", [
    ("batch", 0, L.ERR_BAD_SHAPE), ("num_layers", 0, L.ERR_BAD_SHAPE),
    ("num_heads", 0, L.ERR_BAD_SHAPE), ("num_kv_heads", 3, L.ERR_BAD_SHAPE),
    ("num_kv_heads", 0, L.ERR_BAD_SHAPE), ("head_dim", 96, L.ERR_UNSUPPORTED),
    ("head_dim", 0, L.ERR_BAD_SHAPE), ("num_text", 0, L.ERR_BAD_SHAPE),
    ("grid_h", 0, L.ERR_BAD_SHAPE), ("grid_w", -1, L.ERR_BAD_SHAPE),
    ("grid_h", 2000, L.ERR_UNSUPPORTED),         # with grid_w = 1000: N = 2e6 > 2^20
    ("num_heads", 130, L.ERR_UNSUPPORTED),       # with num_kv_heads = 2: H > 128
])
def test_bad_shapes(field, value, expect):
    kw = {field: value}
    if field == "grid_h" and value == 2000:
        kw["grid_w"] = 1000                       # N = 2e6 > 2^20
    assert score(good_shape(**kw), good_params()) == expect


def test_large_grids_accepted_and_cells_capped():
    """Up to 2^20 visual tokens per image; at most 128 cells per side."""
    big = good_shape(grid_h=1024, grid_w=1024)                    # N = 2^20
    assert score(big, good_params(), q=None) == L.ERR_NULL_POINTER  # validated, not rejected
    assert score(good_shape(grid_h=1024, grid_w=1025), good_params()) == L.ERR_UNSUPPORTED
    wide = good_shape(grid_h=130, grid_w=130)
    assert select(wide, good_params(cells=128, keep=5), c=None) == L.ERR_NULL_POINTER
    assert select(wide, good_params(cells=129, keep=5)) == L.ERR_UNSUPPORTED


def test_grid_limits():
    """Every kernel grid stays under 2^32 work-items: B*L*H < 2^22 and
    B*L*ceil(N/64) < 2^24, else E2S_ERR_UNSUPPORTED before any launch."""
    at = good_shape(batch=(1 << 22) // 128 - 1, num_layers=4, num_heads=32, num_kv_heads=32,
                    grid_h=2, grid_w=2)                           # B*L*H = 2^22 - 128
    assert score(at, good_params(keep=1), q=None) == L.ERR_NULL_POINTER
    over = good_shape(batch=(1 << 22) // 128, num_layers=4, num_heads=32, num_kv_heads=32,
                      grid_h=2, grid_w=2)                         # B*L*H = 2^22
    assert score(over, good_params(keep=1)) == L.ERR_UNSUPPORTED
    assert prune(over, good_params(keep=1), ws_bytes=0) == L.ERR_UNSUPPORTED
    tokens = good_shape(batch=1 << 14, num_layers=1, num_heads=1, num_kv_heads=1,
                        grid_h=1024, grid_w=64)                   # B*L*N/64 = 2^24
    assert score(tokens, good_params(keep=1)) == L.ERR_UNSUPPORTED
    fits = good_shape(batch=(1 << 14) - 1, num_layers=1, num_heads=1, num_kv_heads=1,
                      grid_h=1024, grid_w=64)
    assert score(fits, good_params(keep=1), q=None) == L.ERR_NULL_POINTER


def test_fp16_dtype_accepted():
    """E2S_DTYPE_F16 = 2 passes validation (the call then stops at a missing pointer)."""
    assert L.DTYPE_F16 == 2
    assert score(good_shape(), good_params(dtype=L.DTYPE_F16), q=None) == L.ERR_NULL_POINTER
    assert score(good_shape(), good_params(dtype=3)) == L.ERR_BAD_PARAM


@pytest.mark.parametrize("field,value", [
    ("dtype", 5), ("mode", 2), ("scale", -1.0), ("scale", float("nan")), ("scale", float("inf")),
])
def test_bad_score_params(field, value):
    assert score(good_shape(), good_params(**{field: value})) == L.ERR_BAD_PARAM
    assert layer_rel(good_shape(), good_params(**{field: value}), ws_bytes=1 << 30) == \
        L.ERR_BAD_PARAM


@pytest.mark.parametrize("field,value", [
    ("cells", 0), ("cells", 7), ("lam", -0.01), ("lam", 1.5), ("lam", float("nan")),
    ("keep", -1), ("keep", 43),
])
def test_bad_select_params(field, value):
    # grid 6x7 = 42 tokens: cells <= 6, keep <= 42
    assert select(good_shape(), good_params(**{field: value})) == L.ERR_BAD_PARAM
    assert prune(good_shape(), good_params(**{field: value}), ws_bytes=1 << 30) == L.ERR_BAD_PARAM
    assert fuse_sel(good_shape(), good_params(**{field: value})) == L.ERR_BAD_PARAM


def test_null_pointers():
    assert score(None, good_params()) == L.ERR_NULL_POINTER
    assert score(good_shape(), None) == L.ERR_NULL_POINTER
    assert score(good_shape(), good_params(), q=None) == L.ERR_NULL_POINTER
    assert score(good_shape(), good_params(), k=None) == L.ERR_NULL_POINTER
    assert score(good_shape(), good_params(), e=None) == L.ERR_NULL_POINTER
    assert select(good_shape(), good_params(), c=None) == L.ERR_NULL_POINTER
    assert select(good_shape(), good_params(), out=None) == L.ERR_NULL_POINTER
    assert prune(good_shape(), good_params(), ws=None) == L.ERR_NULL_POINTER
    assert prune(good_shape(), good_params(), out=None) == L.ERR_NULL_POINTER
    sh = good_shape()
    assert lib.e2s_head_reliability(ctypes.byref(sh), None, A, A, None) == L.ERR_NULL_POINTER
    assert lib.e2s_head_masses(ctypes.byref(sh), A, None, A, None) == L.ERR_NULL_POINTER
    assert lib.e2s_ds_combine_layers(ctypes.byref(sh), A, None, None, None, None) == \
        L.ERR_NULL_POINTER
    assert lib.e2s_fuse_evidence(ctypes.byref(sh), None, None, None, A, None) == \
        L.ERR_NULL_POINTER
    for kw in ({"q": None}, {"k": None}, {"ws": None}, {"rho": None}, {"pbar": None}):
        assert layer_rel(good_shape(), good_params(), **kw) == L.ERR_NULL_POINTER, kw
    for kw in ({"rho": None}, {"pbar": None}, {"out": None}):
        assert fuse_sel(good_shape(), good_params(), **kw) == L.ERR_NULL_POINTER, kw
    n = ctypes.c_size_t()
    assert lib.e2s_prune_workspace_size(None, ctypes.byref(good_params()), ctypes.byref(n)) == \
        L.ERR_NULL_POINTER


def test_misaligned_pointers():
    assert score(good_shape(), good_params(), q=A + 8) == L.ERR_MISALIGNED
    assert score(good_shape(), good_params(), k=A + 2) == L.ERR_MISALIGNED
    assert score(good_shape(), good_params(), e=A + 2) == L.ERR_MISALIGNED
    assert select(good_shape(), good_params(), adj=A + 4) == L.ERR_MISALIGNED
    assert prune(good_shape(), good_params(), ws=A + 16) == L.ERR_MISALIGNED
    assert layer_rel(good_shape(), good_params(), ws=A + 16) == L.ERR_MISALIGNED
    assert layer_rel(good_shape(), good_params(), q=A + 4) == L.ERR_MISALIGNED
    assert layer_rel(good_shape(), good_params(), rho=A + 2) == L.ERR_MISALIGNED
    assert fuse_sel(good_shape(), good_params(), pbar=A + 1) == L.ERR_MISALIGNED
    assert fuse_sel(good_shape(), good_params(), prio=A + 2) == L.ERR_MISALIGNED


def test_workspace_size_and_too_small():
    sh, pa = good_shape(), good_params()
    need = L.workspace_size(sh, pa)
    e = 2 * 3 * 4 * 42 * 4          # supports [B, L, H, N]
    rel = 2 * 3 * 42 * 4            # rho or pbar_c [B, L, N]
    assert need == -(-e // 256) * 256 + 2 * (-(-rel // 256) * 256)
    assert prune(sh, pa, ws_bytes=need - 1) == L.ERR_WORKSPACE_TOO_SMALL
    assert layer_rel(sh, pa, ws_bytes=need - 1) == L.ERR_WORKSPACE_TOO_SMALL


def test_keep_zero_allows_null_output():
    """K = 0 (the paper's 20 -> 8 -> 0 schedule) is valid and needs no output buffer;
    the call is only validated here: a misaligned score pointer, checked after the
    output pointer, stops it before any launch."""
    assert select(good_shape(), good_params(keep=0), c=A + 2, out=None) == L.ERR_MISALIGNED
    assert select(good_shape(), good_params(keep=1), c=A + 2, out=None) == L.ERR_NULL_POINTER
    assert fuse_sel(good_shape(), good_params(keep=0), rho=A + 2, out=None) == L.ERR_MISALIGNED


def test_binding_rejects_cpu_tensors():
    torch = pytest.importorskip("torch")
    q = torch.zeros((1, 1, 1, 1, 64), dtype=torch.bfloat16)
    with pytest.raises(ValueError):
        L.score_heads(q, q, 1, 1)


def test_binding_requires_one_device():
    """Every tensor of a call must live on one GPU; the call then runs with that GPU
    current (checked on stand-in objects: no GPU is touched)."""
    torch = pytest.importorskip("torch")

    class T:
        def __init__(self, dev):
            self.device = torch.device(dev)

    assert L._device_of(T("cuda:1"), None, T("cuda:1")) == torch.device("cuda:1")
    with pytest.raises(ValueError):
        L._device_of(T("cuda:0"), T("cuda:1"))
    with pytest.raises(ValueError):
        L._device_of(None)


@pytest.mark.parametrize("variant", [-1, 6])
def test_bad_variant(variant):
    assert prune(good_shape(), good_params(variant=variant)) == L.ERR_BAD_PARAM
    assert fuse_sel(good_shape(), good_params(variant=variant)) == L.ERR_BAD_PARAM
    assert stage(good_shape(), good_params(variant=variant), 42) == L.ERR_BAD_PARAM


def test_fuse_select_has_no_attention_topk():
    """A1 needs the per-head supports, which e2s_fuse_select does not receive."""
    assert fuse_sel(good_shape(), good_params(variant="a1_attention_topk")) == L.ERR_UNSUPPORTED


def test_stage_validation():
    sh = good_shape()                      # grid 6 x 7 = 42 positions
    assert stage(sh, good_params(keep=5), 0) == L.ERR_BAD_SHAPE
    assert stage(sh, good_params(keep=5), 43) == L.ERR_BAD_SHAPE
    assert stage(sh, good_params(keep=5), 20, pos=None) == L.ERR_BAD_SHAPE   # positions needed
    assert stage(sh, good_params(keep=21), 20) == L.ERR_BAD_PARAM            # K > N_l
    assert stage(sh, good_params(keep=5), 20, out=None) == L.ERR_NULL_POINTER
    assert stage(sh, good_params(keep=0), 20, out=None, pos=A + 2) == L.ERR_MISALIGNED
    assert stage(sh, good_params(keep=5), 20, mprev=A + 2) == L.ERR_MISALIGNED
    assert stage(sh, good_params(keep=5), 20, kpos=A + 1) == L.ERR_MISALIGNED
    assert stage(sh, good_params(keep=5), 20, ws_bytes=16) == L.ERR_WORKSPACE_TOO_SMALL
    assert stage(sh, good_params(keep=5), 20, q=None) == L.ERR_NULL_POINTER
    assert stage(sh, good_params(keep=5, cells=7), 20) == L.ERR_BAD_PARAM


# ---------------------------------------------------------------------------
# ragged batches
# ---------------------------------------------------------------------------

RAGGED_DIMS = [(6, 7, 5, 10), (4, 9, 1, 0), (8, 8, 12, 64)]


def ragged_images(dims=RAGGED_DIMS, L_=3, H=4, Hkv=2, D=64):
    arr, _, _, _, _ = L.packed_images(dims, L_, H, Hkv, D)
    return arr


def ragged(images, params=None, shape=None, dev=A, q=A, k=A, ws=A, ws_bytes=None, out=A):
    shape = L.RaggedShape(len(images), 3, 4, 2, 64) if shape is None else shape
    params = good_params() if params is None else params
    if ws_bytes is None:
        n = ctypes.c_size_t(0)
        st = lib.e2s_prune_ragged_workspace_size(ctypes.byref(shape), ctypes.addressof(images),
                                                 ctypes.byref(n))
        ws_bytes = n.value if st == L.OK else 1 << 30
    return lib.e2s_prune_ragged(ctypes.byref(shape), ctypes.byref(params),
                                ctypes.addressof(images), dev, q, k, ws, ws_bytes, out, None,
                                None, None)


def test_ragged_workspace_size_is_the_token_span():
    imgs = ragged_images()
    n = ctypes.c_size_t(0)
    sh = L.RaggedShape(3, 3, 4, 2, 64)
    assert lib.e2s_prune_ragged_workspace_size(ctypes.byref(sh), ctypes.addressof(imgs),
                                               ctypes.byref(n)) == L.OK
    T = 42 + 36 + 64

    def up(x):
        return (x + 255) // 256 * 256
    assert n.value == up(3 * 4 * T * 4) + 2 * up(3 * T * 4)
    # a uniform batch packed as ragged records needs what e2s_prune needs
    imgs = ragged_images([(6, 7, 5, 10)] * 2)
    sh = L.RaggedShape(2, 3, 4, 2, 64)
    assert lib.e2s_prune_ragged_workspace_size(ctypes.byref(sh), ctypes.addressof(imgs),
                                               ctypes.byref(n)) == L.OK
    assert n.value == L.workspace_size(good_shape(), good_params())


def test_ragged_rejects_invalid_records():
    imgs = ragged_images()
    assert ragged(imgs, ws_bytes=1) == L.ERR_WORKSPACE_TOO_SMALL   # otherwise valid
    bad = ragged_images()
    bad[1].token_offset = 10                                        # overlaps image 0
    assert ragged(bad) == L.ERR_BAD_SHAPE
    bad = ragged_images()
    bad[2].keep_offset = 5                                          # overlaps image 0's keep
    assert ragged(bad) == L.ERR_BAD_SHAPE
    bad = ragged_images()
    bad[1].keep_offset = 0                                          # K_b = 0: no range
    assert ragged(bad, ws_bytes=1) == L.ERR_WORKSPACE_TOO_SMALL
    bad = ragged_images()
    bad[0].q_offset = 4                                             # bf16: 8-element steps
    assert ragged(bad) == L.ERR_MISALIGNED
    bad = ragged_images()
    bad[2].keep = 65                                                # K_b > N_b
    assert ragged(bad) == L.ERR_BAD_PARAM
    bad = ragged_images()
    bad[0].num_text = 0
    assert ragged(bad) == L.ERR_BAD_SHAPE
    bad = ragged_images()
    bad[0].grid_h, bad[0].grid_w = 2000, 1000                       # N_b > 2^20
    assert ragged(bad) == L.ERR_UNSUPPORTED
    bad = ragged_images()
    bad[1].k_offset = -8
    assert ragged(bad) == L.ERR_BAD_SHAPE
    assert ragged(imgs, params=good_params(cells=5)) == L.ERR_BAD_PARAM   # image 1 is 4x9
    assert ragged(imgs, params=good_params(lam=1.5)) == L.ERR_BAD_PARAM
    assert ragged(imgs, dev=None) == L.ERR_NULL_POINTER
    assert ragged(imgs, dev=A + 4) == L.ERR_MISALIGNED
    assert ragged(imgs, out=None) == L.ERR_NULL_POINTER           # some K_b > 0
    assert ragged(imgs, q=A + 8) == L.ERR_MISALIGNED
    assert ragged(imgs, shape=L.RaggedShape(3, 3, 4, 3, 64)) == L.ERR_BAD_SHAPE   # H % Hkv
    assert ragged(imgs, shape=L.RaggedShape(3, 3, 4, 2, 96)) == L.ERR_UNSUPPORTED
    # every K_b = 0: keep_idx may be NULL (then only the workspace is missing here)
    zero = ragged_images([(6, 7, 5, 0), (4, 9, 1, 0)])
    assert ragged(zero, shape=L.RaggedShape(2, 3, 4, 2, 64), out=None, ws_bytes=1) == \
        L.ERR_WORKSPACE_TOO_SMALL


# ---------------------------------------------------------------------------
# token compaction
# ---------------------------------------------------------------------------

def compact(B=2, R=3, N=10, K=4, C=64, eb=2, ss=None, ds=None, keep=A, src=A, dst=A * 2):
    ss = (R * N * C, N * C, C) if ss is None else ss
    ds = (R * K * C, K * C, C) if ds is None else ds
    sh = L.CompactShape(B, R, N, K, C, eb, (ctypes.c_int64 * 3)(*ss), (ctypes.c_int64 * 3)(*ds))
    return lib.e2s_compact_tokens(ctypes.byref(sh), keep, src, dst, None)


def test_compact_rejects_invalid_calls():
    assert lib.e2s_compact_tokens(None, A, A, A, None) == L.ERR_NULL_POINTER
    assert compact(B=0) == L.ERR_BAD_SHAPE
    assert compact(K=-1) == L.ERR_BAD_SHAPE
    assert compact(eb=8) == L.ERR_BAD_PARAM
    assert compact(C=12) == L.ERR_MISALIGNED                   # 24 bytes per vector
    assert compact(ss=(640, 64, 4)) == L.ERR_MISALIGNED         # token stride 8 bytes
    assert compact(ds=(-1, 64, 64)) == L.ERR_BAD_SHAPE
    assert compact(keep=None) == L.ERR_NULL_POINTER
    assert compact(src=A + 8) == L.ERR_MISALIGNED
    assert compact(dst=None) == L.ERR_NULL_POINTER
    assert compact(K=0, keep=None, src=None, dst=None) == L.OK   # nothing to move



def good_views(L_=3, q_strides=(3 * 4 * 5 * 64, 5 * 64, 64), k_strides=(3 * 2 * 42 * 64, 42 * 64, 64)):
    v = L.QKViews()
    for l in range(L_):
        v.q[l] = A + l * (1 << 16)
        v.k[l] = A + (1 << 24) + l * (1 << 16)
    v.q_stride_image, v.q_stride_head, v.q_stride_text = q_strides
    v.k_stride_image, v.k_stride_head, v.k_stride_token = k_strides
    return v


def views(shape, params, v, ws=A, ws_bytes=None, out=A):
    if ws_bytes is None:
        ws_bytes = L.workspace_size(shape, params)
    return lib.e2s_prune_views(ctypes.byref(shape), ctypes.byref(params),
                               ctypes.byref(v) if v is not None else None, ws, ws_bytes, out,
                               None, None, None)


def test_views_validation():
    sh, pa = good_shape(), good_params()
    assert views(sh, pa, good_views(), out=None) == L.ERR_NULL_POINTER      # K > 0
    assert views(sh, pa, None) == L.ERR_NULL_POINTER
    v = good_views()
    v.k[2] = None                                                             # layer 2 < L
    assert views(sh, pa, v) == L.ERR_NULL_POINTER
    v = good_views()
    v.q[1] = A + 8                                                            # unaligned base
    assert views(sh, pa, v) == L.ERR_MISALIGNED
    v = good_views(q_strides=(3 * 4 * 5 * 64, 5 * 64, 68))                  # 136-byte rows
    assert views(sh, pa, v) == L.ERR_MISALIGNED
    v = good_views(k_strides=(-64, 42 * 64, 64))
    assert views(sh, pa, v) == L.ERR_BAD_SHAPE
    assert views(good_shape(num_layers=17), pa, good_views(L_=16)) == L.ERR_UNSUPPORTED
    assert views(sh, pa, good_views(), ws_bytes=1) == L.ERR_WORKSPACE_TOO_SMALL
    assert views(sh, good_params(cells=7), good_views()) == L.ERR_BAD_PARAM
    assert views(sh, good_params(mode=2), good_views()) == L.ERR_BAD_PARAM
    # the packed strides of f32 rows (d = 64: 256 bytes) are accepted by validation
    v = good_views()
    assert views(sh, good_params(dtype=L.DTYPE_F32), v, out=None) == L.ERR_NULL_POINTER


def noalloc(shape, params, q=A, k=A, out=A):
    return lib.e2s_prune_noalloc(ctypes.byref(shape), ctypes.byref(params), q, k, out, None,
                                 None, None)


def test_noalloc_validation():
    """e2s_prune_noalloc validates like e2s_prune and refuses a shape whose workspace
    exceeds the static scratch before it looks the scratch up."""
    pa = good_params()
    assert noalloc(good_shape(), pa, q=None) == L.ERR_NULL_POINTER
    assert noalloc(good_shape(), pa, k=A + 2) == L.ERR_MISALIGNED
    assert noalloc(good_shape(head_dim=96), pa) == L.ERR_UNSUPPORTED
    assert noalloc(good_shape(), good_params(keep=43)) == L.ERR_BAD_PARAM
    assert noalloc(good_shape(), pa, out=None) == L.ERR_NULL_POINTER
    # 256 LLaVA-shaped images: 80 MB of workspace against 64 MiB of scratch
    big = good_shape(batch=256, num_layers=4, num_heads=32, num_kv_heads=32, head_dim=128,
                     num_text=64, grid_h=24, grid_w=24)
    assert L.workspace_size(big, pa) > L.NOALLOC_SCRATCH_BYTES
    assert noalloc(big, pa) == L.ERR_SCRATCH_TOO_SMALL
    with open(L.HEADER) as f:
        assert "#define E2S_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)" in f.read()
    # 64 of them fit
    fits = good_shape(batch=64, num_layers=4, num_heads=32, num_kv_heads=32, head_dim=128,
                      num_text=64, grid_h=24, grid_w=24)
    assert L.workspace_size(fits, pa) <= L.NOALLOC_SCRATCH_BYTES


def test_read_probe_validation():
    """The measurement helper rejects bad arguments before any launch."""
    f = lib.e2s_read_probe
    assert f(None, 1024, 8, A, None) == L.ERR_NULL_POINTER
    assert f(A, 1024, 8, None, None) == L.ERR_NULL_POINTER
    assert f(A + 4, 1024, 8, A, None) == L.ERR_MISALIGNED
    assert f(A, 1024, 8, A + 2, None) == L.ERR_MISALIGNED
    assert f(A, 0, 8, A, None) == L.ERR_BAD_SHAPE
    assert f(A, 1000, 8, A, None) == L.ERR_BAD_SHAPE
    assert f(A, 1024, 0, A, None) == L.ERR_BAD_PARAM
    assert f(A, 1024, 65536, A, None) == L.ERR_BAD_PARAM
