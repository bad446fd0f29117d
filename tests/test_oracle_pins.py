"""Pins of the CPU oracle against what the paper and mathematics fix.

Each test checks an oracle function against something other than the oracle's
own formula: values the paper prints (with hand-derived consequences, stored
under tests/golden/), closed forms, invariants, a textbook implementation of
Dempster's rule over the power set, an independent library routine, or brute
force on tiny inputs.
"""
import itertools
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import scipy.special

import oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rng(seed):
    return np.random.default_rng(seed)


def _frac_expr(s: str) -> Fraction:
    """Parse '[1-]a/b' or 'a/b' with decimal a, b into an exact Fraction."""
    s = s.strip()
    neg_from_one = s.startswith("1-")
    if neg_from_one:
        s = s[2:]
    num, den = s.split("/")
    v = Fraction(num) / Fraction(den)
    return 1 - v if neg_from_one else v


# ---------------------------------------------------------------------------
# Eq. (1): text-to-visual logits
# ---------------------------------------------------------------------------

def test_logits_brute_force_tiny():
    """Eq. (1) summand z[t,n] = Q_t . K_n / sqrt(d): pure-Python dot products."""
    rng = _rng(1)
    q = rng.standard_normal((3, 5))
    k = rng.standard_normal((4, 5))
    z = O.text_visual_logits(q, k, 1 / math.sqrt(5))
    for t in range(3):
        for n in range(4):
            dot = sum(float(q[t, i]) * float(k[n, i]) for i in range(5))
            assert z[t, n] == pytest.approx(dot / math.sqrt(5), rel=1e-13, abs=1e-15)


def test_mean_logit_equals_mean_query_by_linearity():
    """Eq. (1) is linear in Q_t: the mean of the logits equals (mean_t Q_t) . K / sqrt(d)."""
    rng = _rng(2)
    L, H, nt, n, d = 2, 3, 7, 11, 8
    q = rng.standard_normal((L, H, nt, d))
    k = rng.standard_normal((L, H, n, d))
    r, _ = O.score_heads(q, k, "mean_logit")
    for l in range(L):
        for h in range(H):
            a = (k[l, h] @ q[l, h].mean(axis=0)) / math.sqrt(d)
            np.testing.assert_allclose(r[l, h], scipy.special.softmax(a), rtol=1e-12)


def test_gqa_head_mapping():
    """Query head h reads KV head floor(h*Hkv/H): with H=4, Hkv=2, heads 2 and 3
    read KV head 1.  Making every key of KV head 1 identical must make exactly
    heads 2 and 3 uniform (r = 1/N)."""
    rng = _rng(3)
    q = rng.standard_normal((1, 4, 5, 8))
    k = rng.standard_normal((1, 2, 9, 8))
    k[0, 1] = k[0, 1, 0]
    for mode in O.SCORE_MODES:
        r, _ = O.score_heads(q, k, mode)
        for h in range(4):
            uniform = np.allclose(r[0, h], 1 / 9, rtol=0, atol=1e-15)
            assert uniform == (h >= 2), (mode, h)


# ---------------------------------------------------------------------------
# Eq. (8): softmax over visual tokens; the two score modes
# ---------------------------------------------------------------------------

def test_softmax_matches_library_and_sums_to_one():
    rng = _rng(4)
    x = rng.standard_normal((6, 50)) * 5
    r = O.softmax_over_visual(x)
    np.testing.assert_allclose(r, scipy.special.softmax(x, axis=-1), rtol=1e-13)
    np.testing.assert_allclose(r.sum(axis=-1), 1.0, rtol=0, atol=1e-14)
    assert (r > 0).all()
    big = O.softmax_over_visual(np.array([1000.0, 1000.0, 999.0]))
    np.testing.assert_allclose(big, scipy.special.softmax([1000.0, 1000.0, 999.0]), rtol=1e-14)


@pytest.mark.parametrize("mode", O.SCORE_MODES)
def test_normalized_attention_rows_sum_to_one(mode):
    rng = _rng(5)
    z = rng.standard_normal((10, 40)) * 3
    r = O.normalized_attention(z, mode)
    assert r.shape == (40,)
    assert abs(r.sum() - 1.0) < 1e-14 and (r > 0).all()


def test_modes_agree_for_one_query_and_for_identical_queries():
    """With a single text query, or identical queries, softmax and query-mean commute."""
    rng = _rng(6)
    z1 = rng.standard_normal((1, 30))
    np.testing.assert_allclose(O.normalized_attention(z1, "mean_prob"),
                               O.normalized_attention(z1, "mean_logit"), rtol=1e-14)
    zr = np.repeat(rng.standard_normal((1, 30)), 7, axis=0)
    np.testing.assert_allclose(O.normalized_attention(zr, "mean_prob"),
                               O.normalized_attention(zr, "mean_logit"), rtol=1e-13)


def test_mean_prob_closed_form_one_peaked_query():
    """Queries 1..T-1 see all-zero logits (softmax = 1/N); query 0 puts +inf-like mass
    on token j.  Then r_j = (1 + (T-1)/N)/T and every other r_n = ((T-1)/N)/T.  The
    mean-of-logits reading gives a different r, so this separates the two modes."""
    T, N, j = 5, 12, 7
    z = np.zeros((T, N))
    z[0, j] = 800.0
    r = O.normalized_attention(z, "mean_prob")
    expect = np.full(N, ((T - 1) / N) / T)
    expect[j] = (1 + (T - 1) / N) / T
    np.testing.assert_allclose(r, expect, rtol=1e-14)
    r1 = O.normalized_attention(z, "mean_logit")
    assert r1[j] > 0.999999


# ---------------------------------------------------------------------------
# Eq. (9): support map
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("n", [1, 7, 576, 4096])
def test_support_closed_forms(n):
    """r = 1/N_l gives p = 0.5 exactly (Sec. 4.1 after Eq. (9)); r = 3/N gives 0.75;
    r -> 1 stays below N/(N+1)."""
    assert O.support_from_attention(np.array([1.0 / n]), n)[0] == 0.5
    assert O.support_from_attention(np.array([3.0 / n]), n)[0] == pytest.approx(0.75, abs=1e-15)
    assert O.support_from_attention(np.array([1.0]), n)[0] == pytest.approx(n / (n + 1), rel=1e-15)
    assert O.support_from_attention(np.array([0.0]), n)[0] == 0.0


# ---------------------------------------------------------------------------
# Eq. (10)-(11): reliability and masses
# ---------------------------------------------------------------------------

def _read_reliability_golden():
    rows = []
    with open(os.path.join(GOLDEN, "reliability_four_heads.txt")) as f:
        for line in f:
            if not line.strip() or line.startswith("#"):
                continue
            name, p, pbar, rho, m = [c.strip() for c in line.split("|")]
            rows.append((name, [float(x) for x in p.split()], float(pbar), float(rho),
                         [float(x) for x in m.split()]))
    return rows


@pytest.mark.parametrize("row", _read_reliability_golden(), ids=lambda r: r[0])
def test_reliability_four_head_examples(row):
    _, p, pbar, rho, m = row
    p = np.array(p).reshape(4, 1)
    got_rho, got_pbar = O.head_reliability(p)
    assert got_pbar[0] == pytest.approx(pbar, abs=1e-15)
    assert got_rho[0] == pytest.approx(rho, abs=1e-15)
    got_m = O.head_masses(got_rho, got_pbar)[0]
    np.testing.assert_allclose(got_m, m, rtol=0, atol=1e-15)


def test_reliability_single_head_and_equal_heads():
    """H = 1, or all heads equal: consistency = 1, so rho = |2p - 1|."""
    p = np.array([[0.0, 0.2, 0.5, 0.75, 0.99]])
    rho, pbar = O.head_reliability(p)
    np.testing.assert_allclose(rho, np.abs(2 * p[0] - 1), atol=1e-15)
    np.testing.assert_allclose(pbar, p[0])
    p4 = np.repeat(p, 4, axis=0)
    rho4, _ = O.head_reliability(p4)
    np.testing.assert_allclose(rho4, np.abs(2 * p[0] - 1), atol=1e-15)


def test_reliability_range_and_mass_axioms():
    """rho in [0,1]; masses are a basic probability assignment (Eq. (2))."""
    rng = _rng(7)
    p = rng.uniform(0, 1, size=(3, 16, 200))
    rho, pbar = O.head_reliability(p)
    assert (rho >= 0).all() and (rho <= 1).all()
    m = O.head_masses(rho, pbar)
    assert (m >= 0).all()
    np.testing.assert_allclose(m.sum(axis=-1), 1.0, atol=1e-15)


def test_reliability_opposed_heads_give_zero():
    """Half the heads at p=1-x and half at x: sum of (p-0.5) cancels, so clarity = 0."""
    p = np.array([[0.9], [0.1], [0.9], [0.1]])
    rho, _ = O.head_reliability(p)
    assert rho[0] == pytest.approx(0.0, abs=1e-15)


# ---------------------------------------------------------------------------
# Eq. (12)-(19): Dempster fusion across layers
# ---------------------------------------------------------------------------

I_, U_ = frozenset("I"), frozenset("U")
TH = I_ | U_


def _textbook_dempster(m1: dict, m2: dict):
    """Dempster's rule over the power set of Theta (Eq. (3)-(4)) with set algebra."""
    conflict = 0.0
    out = {}
    for b, mb in m1.items():
        for c, mc in m2.items():
            inter = b & c
            if not inter:
                conflict += mb * mc
            else:
                out[inter] = out.get(inter, 0.0) + mb * mc
    return {a: v / (1 - conflict) for a, v in out.items()}, conflict


def _random_masses(rng, n):
    m = rng.dirichlet([1.0, 1.0, 1.0], size=n)
    return m


def test_dempster_step_equals_textbook_rule():
    rng = _rng(8)
    a = _random_masses(rng, 50)
    b = _random_masses(rng, 50)
    fused, K = O.dempster_step(a, b)
    for i in range(50):
        m1 = {I_: a[i, 0], U_: a[i, 1], TH: a[i, 2]}
        m2 = {I_: b[i, 0], U_: b[i, 1], TH: b[i, 2]}
        ref, kref = _textbook_dempster(m1, m2)
        assert K[i] == pytest.approx(kref, rel=1e-12, abs=1e-15)
        np.testing.assert_allclose(fused[i], [ref.get(I_, 0), ref.get(U_, 0), ref.get(TH, 0)],
                                   rtol=1e-12, atol=1e-15)


def test_dempster_commutative_associative_and_vacuous_identity():
    rng = _rng(9)
    a, b, c = (_random_masses(rng, 40) for _ in range(3))
    ab, kab = O.dempster_step(a, b)
    ba, kba = O.dempster_step(b, a)
    np.testing.assert_allclose(ab, ba, rtol=1e-13)
    np.testing.assert_allclose(kab, kba, rtol=1e-13)
    left, _ = O.dempster_step(ab, c)
    bc, _ = O.dempster_step(b, c)
    right, _ = O.dempster_step(a, bc)
    np.testing.assert_allclose(left, right, rtol=1e-12, atol=1e-15)
    vac = np.tile([0.0, 0.0, 1.0], (40, 1))
    same, k0 = O.dempster_step(a, vac)
    np.testing.assert_allclose(same, a, rtol=1e-15)
    assert (k0 == 0).all()


def test_fused_mass_order_independent_but_priority_uses_last_conflict():
    """m~ does not depend on layer order (commutative + associative); q uses the last
    step's conflict K^(L) (Eq. (19)), so it generally does for L >= 3 but not L = 2."""
    rng = _rng(10)
    m = np.stack([_random_masses(rng, 30) for _ in range(3)])
    base = O.ds_combine_layers(m)
    for perm in itertools.permutations(range(3)):
        f = O.ds_combine_layers(m[list(perm)])
        np.testing.assert_allclose(f[0], base[0], rtol=1e-12, atol=1e-15)
    swapped = O.ds_combine_layers(m[[0, 2, 1]])
    assert np.abs(swapped[3] - base[3]).max() > 1e-6
    two = O.ds_combine_layers(m[:2])
    two_sw = O.ds_combine_layers(m[[1, 0]])
    np.testing.assert_allclose(two[3], two_sw[3], rtol=1e-13)


def _read_intro_golden():
    rows = []
    with open(os.path.join(GOLDEN, "intro_three_layers.txt")) as f:
        for line in f:
            if not line.strip() or line.startswith("#"):
                continue
            cols = [c.strip() for c in line.split("|")]
            rows.append((int(cols[0]), [Fraction(x) for x in cols[1].split()],
                         *[_frac_expr(c) for c in cols[2:]]))
    return rows


def test_intro_example_bayesian_closed_form():
    """The introduction's three-token example with Bayesian masses (rho = 1):
    Eq. (12)-(19) must reproduce the normalized-product closed form; plain averaging
    of token 1 must reproduce the printed 0.57."""
    rows = _read_intro_golden()
    for tok, s, mean, mI, mU, K3, q in rows:
        s = np.array([float(x) for x in s])
        masses = np.stack([s, 1 - s, np.zeros(3)], axis=-1)[:, None, :]   # [L=3, N=1, 3]
        fused, conflict, pl, prio, bel = O.ds_combine_layers(masses)
        assert fused[0, 0] == pytest.approx(float(mI), rel=1e-13)
        assert fused[0, 1] == pytest.approx(float(mU), rel=1e-13)
        assert fused[0, 2] == pytest.approx(0.0, abs=1e-15)
        assert conflict[2, 0] == pytest.approx(float(K3), rel=1e-13)
        assert prio[0] == pytest.approx(float(q), rel=1e-13)
        assert bel[0] == fused[0, 0]
        if tok == 1:
            assert round(float(mean), 2) == 0.57


def test_total_conflict_branch():
    """(1,0,0) + (0,1,0): K = 1; the fused mass becomes vacuous and q = 1 (Eq. (19))."""
    m = np.array([[[1.0, 0.0, 0.0]], [[0.0, 1.0, 0.0]]])
    fused, conflict, pl, q, _ = O.ds_combine_layers(m)
    assert conflict[1, 0] == 1.0
    np.testing.assert_array_equal(fused[0], [0.0, 0.0, 1.0])
    assert q[0] == 1.0
    m3 = np.concatenate([m, np.array([[[0.2, 0.3, 0.5]]])])
    fused3, conflict3, _, _, _ = O.ds_combine_layers(m3)
    np.testing.assert_allclose(fused3[0], [0.2, 0.3, 0.5], rtol=1e-15)
    assert conflict3[2, 0] == 0.0


def test_single_layer_priority_is_plausibility():
    rng = _rng(11)
    m = _random_masses(rng, 20)[None]
    fused, conflict, pl, q, _ = O.ds_combine_layers(m)
    np.testing.assert_array_equal(fused, m[0])
    assert (conflict == 0).all()
    np.testing.assert_allclose(q, pl, rtol=0, atol=1e-15)


def test_fusion_invariants_random():
    """Eq. (2), (3), (17)-(19) invariants on random layer masses."""
    rng = _rng(12)
    m = np.stack([_random_masses(rng, 500) for _ in range(5)])
    fused, conflict, pl, q, bel = O.ds_combine_layers(m)
    assert (fused >= 0).all()
    np.testing.assert_allclose(fused.sum(-1), 1.0, atol=1e-13)
    assert (conflict >= 0).all() and (conflict <= 1).all()
    np.testing.assert_allclose(pl, 1 - fused[:, 1], atol=1e-13)            # Eq. (18)
    assert (bel <= pl + 1e-15).all()
    assert (q >= pl - 1e-15).all() and (q >= 0).all() and (q <= 1 + 1e-15).all()
    # conflict bound: K^(l) <= (1 - m~(Theta)^(l-1)) (1 - m_l(Theta))
    acc = m[0]
    for l in range(1, 5):
        nxt, K = O.dempster_step(acc, m[l])
        assert (K <= (1 - acc[:, 2]) * (1 - m[l][:, 2]) + 1e-15).all()
        acc = nxt


# ---------------------------------------------------------------------------
# Eq. (20)-(23): spatial novelty and top-K
# ---------------------------------------------------------------------------

def _cells_by_ranges(grid_h, grid_w, G):
    """Members of each cell from explicit row/column ranges (brute force)."""
    out = []
    for gr in range(G):
        for gc in range(G):
            rows = [r for r in range(grid_h) if (r * G) // grid_h == gr]
            cols = [c for c in range(grid_w) if (c * G) // grid_w == gc]
            out.append(sorted(r * grid_w + c for r in rows for c in cols))
    return out


def test_cell_partition_even_grid_by_hand():
    """24x24 with G = 4: 16 cells of 6x6 tokens (Sec. 4.3)."""
    cell = O.cell_of_token(24, 24, 4)
    assert cell[0] == 0 and cell[5] == 0 and cell[6] == 1 and cell[23] == 3
    assert cell[6 * 24] == 4 and cell[575] == 15
    counts = np.bincount(cell)
    assert counts.tolist() == [36] * 16


@pytest.mark.parametrize("gh,gw,G", [(4, 4, 2), (5, 7, 3), (8, 8, 4), (3, 9, 3), (6, 4, 4)])
def test_cell_representatives_brute_force(gh, gw, G):
    rng = _rng(gh * 100 + gw * 10 + G)
    q = rng.integers(0, 4, size=gh * gw) / 4.0     # many exact ties
    b = O.cell_representatives(q, gh, gw, G)
    expect = np.zeros(gh * gw, dtype=np.int64)
    for members in _cells_by_ranges(gh, gw, G):
        if members:
            best = max(members, key=lambda i: (q[i], -i))
            expect[best] = 1
    np.testing.assert_array_equal(b, expect)


def _brute_force_topk(q, b, lam, K):
    """Maximise sum of q~ over all K-subsets; ties -> lexicographically smallest tuple.
    Exact rational arithmetic."""
    lam = Fraction(lam)
    qt = [(1 - lam) * Fraction(float(x)) + lam * int(bb) for x, bb in zip(q, b)]
    best, best_key = None, None
    for sub in itertools.combinations(range(len(q)), K):
        key = (-sum(qt[i] for i in sub), sub)
        if best_key is None or key < best_key:
            best, best_key = sub, key
    return list(best)


@pytest.mark.parametrize("G", [2, 4])
@pytest.mark.parametrize("lam", [0.0, 0.25, 0.5, 1.0])
def test_topk_brute_force_tiny_grid(G, lam):
    """Eq. (23) on a 4x4 grid: the rank rule equals exhaustive subset search."""
    rng = _rng(13 + G)
    for trial in range(4):
        q = rng.integers(0, 5, size=16) / 8.0       # exact in binary, many ties
        for K in (0, 1, 3, 6):
            kept, qt, b = O.spatial_select(q, 4, 4, G, lam, K)
            assert kept.tolist() == _brute_force_topk(q, b, lam, K), (trial, K)


def test_lambda_zero_is_plain_topk_and_lambda_one_is_representatives_first():
    rng = _rng(14)
    q = rng.uniform(size=64)
    q[5] = q[9] = q[40]        # ties
    K = 20
    kept0, _, _ = O.spatial_select(q, 8, 8, 4, 0.0, K)
    plain = sorted(sorted(range(64), key=lambda i: (-q[i], i))[:K])
    assert kept0.tolist() == plain
    kept1, _, b = O.spatial_select(q, 8, 8, 4, 1.0, K)
    reps = [i for i in range(64) if b[i]]
    rest = [i for i in range(64) if not b[i]][:K - len(reps)]
    assert kept1.tolist() == sorted(reps + rest)
    kept_small, _, _ = O.spatial_select(q, 8, 8, 4, 1.0, 5)
    assert kept_small.tolist() == reps[:5]


def test_large_lambda_keeps_every_representative():
    """lam > 1/2 and K >= G^2: every cell representative is kept."""
    rng = _rng(15)
    for lam in (0.51, 0.75, 0.9):
        q = rng.uniform(size=576)
        kept, _, b = O.spatial_select(q, 24, 24, 4, lam, 16)
        assert set(np.nonzero(b)[0]) == set(kept.tolist())


def test_soft_bonus_does_not_force_every_cell():
    """Sec. 4.3: the bonus is soft, so a cell can end with no kept token."""
    q = np.full(64, 0.9)
    cell = O.cell_of_token(8, 8, 4)
    q[cell == 0] = 0.1           # every token of cell 0 far below the rest
    kept, _, b = O.spatial_select(q, 8, 8, 4, 0.1, 16)
    assert not any(cell[i] == 0 for i in kept)
    assert b[cell == 0].sum() == 1


def test_identical_keys_whole_pipeline_closed_form():
    """All keys identical: r = 1/N, p = 1/2, rho = 0, m = (0,0,1), fused vacuous, K = 0,
    q = 1 for every token.  With lam > 0 the kept set is the lowest-index token of
    each cell first (8x8, G = 4: tokens 16*i + 2*j), then the lowest indices."""
    rng = _rng(16)
    q = rng.standard_normal((2, 4, 6, 16))
    k = np.repeat(rng.standard_normal((2, 4, 1, 16)), 64, axis=2)
    for mode in O.SCORE_MODES:
        res = O.prune_image(q, k, 8, 8, keep=20, cells=4, lam=0.3, mode=mode)
        np.testing.assert_allclose(res.r, 1 / 64, rtol=1e-13)
        np.testing.assert_allclose(res.p, 0.5, rtol=1e-13)
        assert np.abs(res.rho).max() < 1e-12
        np.testing.assert_allclose(res.fused, np.tile([0, 0, 1.0], (64, 1)), atol=1e-12)
        assert np.abs(res.q - 1).max() < 1e-12
        reps = sorted(16 * i + 2 * j for i in range(4) for j in range(4))
        first_non_reps = [i for i in range(64) if i not in reps][:4]
        assert res.keep.tolist() == sorted(reps + first_non_reps)


def test_keep_zero_and_keep_all():
    q = _rng(17).uniform(size=36)
    kept, _, _ = O.spatial_select(q, 6, 6, 2, 0.1, 0)
    assert kept.size == 0
    kept, _, _ = O.spatial_select(q, 6, 6, 2, 0.1, 36)
    assert kept.tolist() == list(range(36))


def test_compact_tokens_gather():
    """Token compaction: a hand-worked case, the identity, and composition of two
    compactions (keeping b of the survivors of a keeps a[b])."""
    x = np.arange(2 * 5 * 3, dtype=np.float64).reshape(2, 5, 3)   # [R, N, C]
    got = O.compact_tokens(x, [4, 0, 2])
    want = [[[12, 13, 14], [0, 1, 2], [6, 7, 8]], [[27, 28, 29], [15, 16, 17], [21, 22, 23]]]
    assert got.tolist() == want
    assert np.array_equal(O.compact_tokens(x, np.arange(5)), x)
    rng = np.random.default_rng(3)
    y = rng.standard_normal((3, 4, 40, 8))
    a = np.sort(rng.choice(40, 17, replace=False))
    b = np.sort(rng.choice(17, 6, replace=False))
    assert np.array_equal(O.compact_tokens(O.compact_tokens(y, a), b), O.compact_tokens(y, a[b]))
    assert O.compact_tokens(y, []).shape == (3, 4, 0, 8)
