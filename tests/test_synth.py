"""The seeded input generator: determinism, storage rounding, salient placement."""
import numpy as np
import pytest

import synth


def test_bf16_rounding_known_values():
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -2.5, 0.0, 1.0 + 2 ** -9], np.float32)
    bits = synth.to_bf16_bits(x)
    # 1 + 2^-8 is a tie -> even (0x3F80); 1 + 3*2^-8 is a tie -> even (0x3F82)
    assert bits.tolist() == [0x3F80, 0x3F80, 0x3F82, 0xC020, 0x0000, 0x3F80]
    back = synth.bf16_bits_to_f32(bits)
    assert back[3] == -2.5


def test_generator_deterministic_and_per_image_independent():
    cfg = synth.config_by_name("llava").replace(batch=3)
    q1, k1, s1 = synth.gen_batch(cfg)
    q2, k2, s2 = synth.gen_batch(cfg, images=[2, 0])
    np.testing.assert_array_equal(q1[2], q2[0])
    np.testing.assert_array_equal(k1[0], k2[1])
    assert s1[2].tolist() == s2[0].tolist()
    assert not np.array_equal(q1[0], q1[1])


@pytest.mark.parametrize("name", ["tiny", "llava", "qwen2vl_gqa"])
def test_storage_values_and_salient_counts(name):
    cfg = synth.config_by_name(name)
    q, k, sal = synth.gen_image(cfg, 0)
    assert q.shape == cfg.q_shape()[1:] and k.shape == cfg.k_shape()[1:]
    if cfg.dtype == "bf16":
        np.testing.assert_array_equal(synth.bf16_bits_to_f32(synth.to_bf16_bits(k)), k)
    assert len(sal) == cfg.num_salient == len(set(sal.tolist()))
    expected = {"tiny": 4, "llava": 29, "qwen2vl_gqa": 51}[name]
    assert len(sal) == expected
    assert abs(q.std() * np.sqrt(cfg.head_dim) - 1) < 0.05


def test_salient_keys_shifted_toward_mean_query():
    """The projection of a salient key on the group's mean query exceeds the
    non-salient keys' by about k sigma."""
    cfg = synth.config_by_name("llava")
    q, k, sal = synth.gen_image(cfg, 1)
    u = q[0, 0].astype(np.float64).mean(axis=0)
    u /= np.linalg.norm(u)
    proj = k[0, 0].astype(np.float64) @ u
    non = np.setdiff1d(np.arange(cfg.num_visual), sal)
    gap = proj[sal].mean() - proj[non].mean()
    assert abs(gap / cfg.sigma - cfg.shift_sigmas) < 0.6


def test_clusters_are_compact():
    cfg = synth.config_by_name("llava")
    rng = np.random.Generator(np.random.Philox(7))
    s = synth.salient_set(rng, cfg)
    assert len(s) == 29
    rows, cols = np.divmod(s, cfg.grid_w)
    # three clusters of ~10 tokens: each token has a salient 8-neighbour
    for r, c in zip(rows, cols):
        near = ((np.abs(rows - r) <= 1) & (np.abs(cols - c) <= 1)).sum()
        assert near >= 2


def test_hires_near_duplicates():
    cfg = synth.config_by_name("hires").replace(num_layers=1, num_heads=2, num_kv_heads=2,
                                                num_text=4)
    q, k, sal = synth.gen_image(cfg, 0)
    kk = k[0, 0].astype(np.float64)
    # count tokens whose key is within 0.05 sigma*sqrt(d) of a neighbour's key
    n = cfg.num_visual
    close = 0
    for t in range(n):
        r, c = divmod(t, cfg.grid_w)
        best = np.inf
        for rr in range(max(0, r - 2), min(cfg.grid_h, r + 3)):
            for cc in range(max(0, c - 2), min(cfg.grid_w, c + 3)):
                o = rr * cfg.grid_w + cc
                if o != t:
                    best = min(best, np.linalg.norm(kk[t] - kk[o]))
        close += best < 0.05
    assert close >= int(round(0.1 * n))


def test_ragged_workload_is_seeded_and_in_range():
    rc = synth.ragged_by_name("qwen2vl_dynamic")
    d1, d2 = synth.ragged_dims(rc), synth.ragged_dims(rc)
    assert d1 == d2 and len(d1) == rc.batch
    for gh, gw, nt, keep in d1:
        assert rc.grid_sides[0] <= gh <= rc.grid_sides[1]
        assert rc.grid_sides[0] <= gw <= rc.grid_sides[1]
        assert rc.num_text[0] <= nt <= rc.num_text[1]
        assert keep == max(1, round(rc.keep_frac * gh * gw))
    assert len({(gh, gw) for gh, gw, _, _ in d1}) > rc.batch // 2   # grids really differ
    # image b is gen_image of the base shape with image b's sizes: reproducible alone
    qs, ks, _, dims = synth.gen_ragged(rc, dims=d1[:3], threads=1)
    q1, k1, _ = synth.gen_image(synth.image_config(rc, d1[1]), 1)
    assert np.array_equal(qs[1], q1) and np.array_equal(ks[1], k1)
    assert qs[1].shape == (4, 28, d1[1][2], 128) and ks[1].shape == (4, 4, d1[1][0] * d1[1][1], 128)
