"""GPU check of token compaction (e2s_compact_tokens): every gathered vector equals
the oracle's gather bit for bit, for packed hidden states, a strided slice of a
key/value cache, fp32, several rows, out-of-range indices (left unwritten), K = 0,
and the kept indices e2s_prune returns."""
import numpy as np
import pytest

import oracle as O
import synth
from _helpers import log, to_device

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
E = pytest.importorskip("paper_2608_23253_amd")


def _keep(rng, B, N, K):
    return np.stack([np.sort(rng.choice(N, K, replace=False)) for _ in range(B)]).astype(np.int32)


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_compact_hidden_states(dtype):
    rng = np.random.default_rng(1)
    B, N, C, K = 3, 37, 4096 if dtype == torch.bfloat16 else 192, 11
    x = torch.randn(B, 1, N, C, dtype=torch.float32).to(dtype).cuda()
    keep = _keep(rng, B, N, K)
    out = E.compact_tokens(x, torch.from_numpy(keep).cuda())
    torch.cuda.synchronize()
    ref = np.stack([O.compact_tokens(x[b].float().cpu().numpy(), keep[b]) for b in range(B)])
    assert torch.equal(out.float().cpu(), torch.from_numpy(ref))


def test_compact_kv_cache_slice():
    """The visual tokens of a key/value cache [B, Hkv, S, d]: a strided slice."""
    rng = np.random.default_rng(2)
    B, Hkv, S, d, v0, N, K = 2, 4, 700, 128, 35, 576, 128
    cache = torch.randn(B, Hkv, S, d, dtype=torch.float32).to(torch.bfloat16).cuda()
    src = cache[:, :, v0:v0 + N, :]
    keep = _keep(rng, B, N, K)
    out = E.compact_tokens(src, torch.from_numpy(keep).cuda())
    torch.cuda.synchronize()
    for b in range(B):
        ref = O.compact_tokens(src[b].float().cpu().numpy(), keep[b])
        assert np.array_equal(out[b].float().cpu().numpy(), ref)


def test_compact_out_of_range_and_empty():
    B, R, N, C = 2, 3, 10, 8
    x = torch.arange(B * R * N * C, dtype=torch.float32).reshape(B, R, N, C).cuda()
    keep = torch.tensor([[0, 10, 3], [-1, 9, 2]], dtype=torch.int32).cuda()
    out = torch.full((B, R, 3, C), -7.0, device="cuda")
    E.compact_tokens(x, keep, out=out)
    torch.cuda.synchronize()
    assert torch.equal(out[0, :, 0], x[0, :, 0]) and torch.equal(out[0, :, 2], x[0, :, 3])
    assert torch.equal(out[1, :, 1], x[1, :, 9]) and torch.equal(out[1, :, 2], x[1, :, 2])
    assert (out[0, :, 1] == -7).all() and (out[1, :, 0] == -7).all()   # unwritten
    empty = E.compact_tokens(x, torch.zeros((B, 0), dtype=torch.int32, device="cuda"))
    assert empty.shape == (B, R, 0, C)


def test_compact_after_prune():
    """Keys of the kept tokens, straight from e2s_prune's output."""
    cfg = synth.config_by_name("llava").replace(batch=4)
    q, k, _ = synth.gen_batch(cfg)
    kd = to_device(k, "bf16")
    keep, _, _ = E.prune(to_device(q, "bf16"), kd, 24, 24, cfg.keep)
    kk = kd.reshape(4, cfg.num_layers * cfg.num_kv_heads, 576, 128)
    out = E.compact_tokens(kk, keep)
    torch.cuda.synchronize()
    kn = keep.cpu().numpy()
    for b in range(4):
        ref = O.compact_tokens(synth.to_bf16_bits(k[b].reshape(-1, 576, 128)), kn[b])
        got = out[b].view(torch.int16).cpu().numpy().view(np.uint16)
        assert np.array_equal(got, ref)
    log(f"  compacted {tuple(kk.shape)} -> {tuple(out.shape)}")
