"""Pins of the oracle's progressive schedule (Algorithm 1 with shrinking candidate
sets, Eq. 24) and of its ablation variants (Sec. 5, Table 2), against printed
values, identities the method fixes, and brute force on tiny inputs.  CPU only."""
import math
import os

import numpy as np
import pytest

import oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rng(seed):
    return np.random.default_rng(seed)


def _read_schedules():
    rows = []
    with open(os.path.join(GOLDEN, "avg_tokens_schedules.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            src, kept, avg = (x.strip() for x in line.split("|"))
            rows.append((src, [int(x) for x in kept.split()], int(avg)))
    return rows


# ---------------------------------------------------------------------------
# Eq. (24)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("row", _read_schedules(), ids=lambda r: f"{r[0]}-{'-'.join(map(str, r[1]))}")
def test_avg_tokens_printed_schedules(row):
    """Every printed LLaVA-1.5-7B schedule averages to its stated budget exactly."""
    _, kept, avg = row
    assert O.avg_tokens(32, 576, [3, 17, 22], kept) == avg


def test_avg_tokens_without_pruning_and_one_shot():
    assert O.avg_tokens(32, 576, [], []) == 576
    # pruning once before the first layer: every layer sees the kept count
    assert O.avg_tokens(32, 576, [0], [64]) == 64
    # pruning after the last layer changes nothing
    assert O.avg_tokens(32, 576, [32], [0]) == 576


# ---------------------------------------------------------------------------
# Progressive schedule
# ---------------------------------------------------------------------------

def _layers(rng, L, H, Hkv, NT, N, d, salient=()):
    q = rng.standard_normal((L, H, NT, d)) / math.sqrt(d)
    k = rng.standard_normal((L, Hkv, N, d)) / math.sqrt(d)
    for n in salient:
        k[:, :, n, :] += 3.0 * q.mean(axis=(1, 2))[:, None, :] / math.sqrt(d)
    return q, k


@pytest.mark.parametrize("mode", O.SCORE_MODES)
def test_progressive_without_early_pruning_equals_one_shot(mode):
    """Budgets N, ..., N, K (nothing pruned before the last operation) reproduce the
    one-shot path over the same layers (every operation keeps all candidates,
    N_l = N throughout, and the carried mass continues the same recursion)."""
    rng = _rng(101)
    gh, gw, L = 6, 6, 3
    q, k = _layers(rng, L, 4, 2, 5, gh * gw, 16, salient=(3, 20))
    one = O.prune_image(q, k, gh, gw, keep=10, cells=3, lam=0.2, mode=mode)
    ops = O.prune_progressive([q[l:l + 1] for l in range(L)], [k[l:l + 1] for l in range(L)],
                              gh, gw, [36, 36, 10], cells=3, lam=0.2, mode=mode)
    assert ops[-1].keep_pos.tolist() == one.keep.tolist()
    np.testing.assert_allclose(ops[-1].fused, one.fused, rtol=0, atol=1e-15)
    np.testing.assert_allclose(ops[-1].q, one.q, rtol=0, atol=1e-15)


def test_single_operation_equals_one_shot():
    rng = _rng(102)
    q, k = _layers(rng, 2, 4, 4, 6, 64, 16, salient=(9,))
    one = O.prune_image(q, k, 8, 8, keep=12)
    op = O.prune_progressive([q], [k], 8, 8, [12])[0]
    assert op.keep_pos.tolist() == one.keep.tolist()
    np.testing.assert_array_equal(op.m_out, one.fused[one.keep])


def test_shrinking_sets_and_carried_masses():
    rng = _rng(103)
    gh, gw = 8, 8
    q, k = _layers(rng, 3, 4, 4, 6, 64, 16, salient=(1, 2, 40))
    ops = O.prune_progressive([q[l:l + 1] for l in range(3)], [k[l:l + 1] for l in range(3)],
                              gh, gw, [30, 12, 5], cells=4, lam=0.1)
    prev = set(range(64))
    for op, budget in zip(ops, [30, 12, 5]):
        assert len(op.keep_pos) == budget
        assert set(op.keep_pos.tolist()) <= prev
        assert list(op.keep_pos) == sorted(op.keep_pos)
        prev = set(op.keep_pos.tolist())
    # the second operation starts from the first one's kept masses
    np.testing.assert_array_equal(ops[0].m_out, ops[0].fused[ops[0].keep])


def test_eq9_uses_the_current_candidate_count():
    """Eq. (9) with N_l = |V_l|: candidates with identical keys get r = 1/N_l and
    p = 1/2 exactly, whatever the original grid size."""
    rng = _rng(104)
    q = rng.standard_normal((1, 2, 4, 8))
    k = np.repeat(rng.standard_normal((1, 2, 1, 8)), 7, axis=2)
    res = O.prune_stage(q, k, np.array([0, 5, 9, 30, 31, 50, 63]), 8, 8, keep=3)
    np.testing.assert_allclose(res.r, 1 / 7, rtol=1e-13)
    np.testing.assert_allclose(res.p, 0.5, rtol=1e-13)


def test_vacuous_carried_mass_is_the_identity():
    """Dempster's rule with the vacuous mass (0, 0, 1) returns the other mass and no
    conflict, so carrying it is the same as starting afresh."""
    rng = _rng(105)
    q, k = _layers(rng, 2, 4, 4, 5, 36, 16)
    pos = np.arange(36)
    a = O.prune_stage(q, k, pos, 6, 6, keep=9, cells=3)
    b = O.prune_stage(q, k, pos, 6, 6, keep=9, cells=3, m_prev=np.tile([0.0, 0.0, 1.0], (36, 1)))
    assert a.keep.tolist() == b.keep.tolist()
    np.testing.assert_allclose(a.fused, b.fused, rtol=0, atol=1e-15)
    assert np.abs(b.conflict[0]).max() == 0.0


def test_occupied_cells_brute_force():
    """Representatives exist only for cells holding a candidate, and each is the
    candidate of highest q in its cell (lowest position on ties): explicit loops."""
    rng = _rng(106)
    gh, gw, G = 8, 8, 4
    pos = np.array(sorted(rng.choice(64, size=14, replace=False)))
    qv = rng.integers(0, 3, size=14) / 2.0           # ties
    b = O.cell_representatives(qv, gh, gw, G, pos)
    expect = np.zeros(14, dtype=np.int64)
    groups = {}
    for i, p in enumerate(pos.tolist()):
        row, col = p // gw, p % gw
        groups.setdefault(((row * G) // gh, (col * G) // gw), []).append(i)
    for members in groups.values():
        expect[max(members, key=lambda i: (qv[i], -i))] = 1
    np.testing.assert_array_equal(b, expect)
    assert b.sum() == len(groups) < G * G


# ---------------------------------------------------------------------------
# Ablation variants (Table 2)
# ---------------------------------------------------------------------------

def _softmax(xs):
    m = max(xs)
    e = [math.exp(x - m) for x in xs]
    s = sum(e)
    return [v / s for v in e]


def test_a1_attention_topk_brute_force():
    """A1: top-K of the attention averaged over layers and heads, pure-Python loops."""
    rng = _rng(107)
    L, H, NT, N, d = 2, 3, 4, 9, 5
    q = rng.standard_normal((L, H, NT, d))
    k = rng.standard_normal((L, H, N, d))
    s = 1 / math.sqrt(d)
    score = [0.0] * N
    for l in range(L):
        for h in range(H):
            a = [sum(sum(q[l, h, t, i] * k[l, h, n, i] for i in range(d)) * s for t in range(NT)) / NT
                 for n in range(N)]
            for n, r in enumerate(_softmax(a)):
                score[n] += r / (L * H)
    res = O.prune_image(q, k, 3, 3, keep=4, variant="a1_attention_topk")
    expect = sorted(sorted(range(N), key=lambda n: (-score[n], n))[:4])
    assert res.keep.tolist() == expect
    np.testing.assert_allclose(res.score, score, rtol=1e-12)


def test_a2_bayesian_masses_normalized_product():
    """A2 (rho = 1): Bayesian layer masses fuse to the normalized product of Dempster's
    rule for Bayesian masses, P / (P + R), with 1 - K^(L) = Z_L / Z_{L-1}."""
    rng = _rng(108)
    q, k = _layers(rng, 3, 4, 4, 5, 16, 8, salient=(2,))
    res = O.prune_image(q, k, 4, 4, keep=5, variant="a2_no_head_reliability")
    pbar = res.p.mean(axis=1)                       # [L, N]
    P, R = np.prod(pbar, axis=0), np.prod(1 - pbar, axis=0)
    P2, R2 = np.prod(pbar[:2], axis=0), np.prod(1 - pbar[:2], axis=0)
    np.testing.assert_allclose(res.fused[:, 0], P / (P + R), rtol=1e-12)
    np.testing.assert_allclose(res.fused[:, 2], 0.0, atol=1e-15)
    np.testing.assert_allclose(1 - res.conflict[-1], (P + R) / (P2 + R2), rtol=1e-12)
    np.testing.assert_allclose(1 - res.q, R / (P2 + R2), rtol=1e-12)


def test_a3_is_the_last_layer_alone():
    rng = _rng(109)
    q, k = _layers(rng, 3, 4, 2, 5, 36, 16, salient=(7, 8))
    a3 = O.prune_image(q, k, 6, 6, keep=8, cells=3, variant="a3_no_layer_fusion")
    last = O.prune_image(q[-1:], k[-1:], 6, 6, keep=8, cells=3)
    assert a3.keep.tolist() == last.keep.tolist()
    np.testing.assert_array_equal(a3.q, last.q)


def test_a4_ranks_by_plausibility():
    """A4: q = Pl(I) = 1 - m~(U), so with lambda = 0 the kept set is the K tokens of
    smallest fused m(U) (ties to the lowest index); with one layer K = 0 and A4 is
    the full method."""
    rng = _rng(110)
    q, k = _layers(rng, 3, 4, 4, 5, 25, 8, salient=(4,))
    a4 = O.prune_image(q, k, 5, 5, keep=6, lam=0.0, variant="a4_no_conflict_protection")
    mu = a4.fused[:, 1]
    assert a4.keep.tolist() == sorted(sorted(range(25), key=lambda n: (mu[n], n))[:6])
    one = O.prune_image(q[:1], k[:1], 5, 5, keep=6, variant="a4_no_conflict_protection")
    full = O.prune_image(q[:1], k[:1], 5, 5, keep=6)
    assert one.keep.tolist() == full.keep.tolist()


def test_a5_is_lambda_zero():
    rng = _rng(111)
    q, k = _layers(rng, 2, 4, 4, 5, 36, 8, salient=(0, 1, 2))
    a5 = O.prune_image(q, k, 6, 6, keep=10, lam=0.7, variant="a5_no_spatial_novelty")
    plain = sorted(sorted(range(36), key=lambda n: (-a5.q[n], n))[:10])
    assert a5.keep.tolist() == plain


def test_unknown_variant_rejected():
    with pytest.raises(ValueError):
        O.prune_image(np.zeros((1, 1, 1, 4)), np.zeros((1, 1, 4, 4)), 2, 2, 1, variant="nope")
