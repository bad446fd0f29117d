"""CPU checks of the parity rules the GPU tests apply: the fused-mass bar (both
gates) and the set comparison with its tie and representative-flip excuses."""
import numpy as np

import oracle as O
from _helpers import SelectGeom, assert_mass_bar, compare_sets, mass_errors

import pytest


def _ref(q, gh, gw, G, lam, K):
    """An oracle result carrying only what the set comparison reads."""
    kept, qt, b = O.spatial_select(q, gh, gw, G, lam, K)
    n = q.shape[0]
    nan = np.full(n, np.nan)
    return O.ImageResult(nan, nan, nan, nan, nan, nan, nan, nan, q, qt, b, kept)


def test_mass_bar_both_gates():
    ref = np.array([[1e-4, 2e-4, 1 - 3e-4]])
    assert_mass_bar(ref + 1e-9, ref)
    # absolute gate: 2e-4 on the Theta component is within 2e-3 relative but above 1e-4
    with pytest.raises(AssertionError):
        assert_mass_bar(ref + np.array([[0, 0, 2e-4]]), ref)
    # relative gate: 5e-6 on m(I) = 1e-4 is below 1e-4 absolute but 5 % relative
    with pytest.raises(AssertionError):
        assert_mass_bar(ref + np.array([[5e-6, 0, 0]]), ref)
    a, r = mass_errors(ref + np.array([[1e-7, 0, 0]]), ref)
    assert a == pytest.approx(1e-7) and r < 1.0


def test_compare_sets_exact_tie_fail():
    gh = gw = 4
    q = np.linspace(0.5, 0.9, 16)[::-1].copy()       # token 0 best, 15 worst
    ref = _ref(q, gh, gw, 2, 0.0, 4)
    assert compare_sets(ref.keep, ref).verdict == "exact"
    # a token just below the boundary, within the tie window
    q2 = q.copy()
    q2[4] = q2[3] - 5e-6
    ref2 = _ref(q2, gh, gw, 2, 0.0, 4)
    swapped = np.array([0, 1, 2, 4])
    c = compare_sets(swapped, ref2)
    assert c.verdict == "tie" and c.swaps == 1
    # the same swap with a gap above the window fails
    assert compare_sets(swapped, ref).verdict == "fail"


def test_compare_sets_representative_flip():
    """A cell whose two best tokens are within the window may give its bonus to
    either; the excuse recomputes the ranking with the other representative."""
    gh = gw = 4
    G, lam, K = 2, 0.5, 4
    q = np.full(16, 0.2)
    # cell 0 holds tokens 0, 1, 4, 5: tokens 0 and 5 nearly tied at the top
    q[0], q[5] = 0.6, 0.6 - 1e-7
    q[[2, 8, 10]] = [0.5, 0.45, 0.4]             # representatives of cells 1, 2, 3
    q[1] = 0.59                                   # runner-up in cell 0, clearly below
    ref = _ref(q, gh, gw, G, lam, K)
    assert ref.keep.tolist() == [0, 2, 8, 10]
    # the GPU gave the bonus of cell 0 to token 5 instead
    flipped = np.array([2, 5, 8, 10])
    geom = SelectGeom(gh, gw, G, lam)
    assert compare_sets(flipped, ref).verdict == "fail"
    c = compare_sets(flipped, ref, geom=geom)
    assert c.verdict == "rep_flip"
    # token 1 is not within the window of the cell's best: no excuse
    assert compare_sets(np.array([1, 2, 8, 10]), ref, geom=geom).verdict == "fail"
