"""Pins for the oracle's position reassignment (Sec. 3.2, Eq. (8)-(10)).

PCR's worked values at the tiny fp32 workload are written out in closed form from
Eq. (10); the remaining PCR checks are the properties the paper states for it
(entries inside (p_txt - L, p_txt + 1), next text position unchanged, relative
layout kept) plus translation/scale invariance and exact endpoint values.
"""
from fractions import Fraction

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from oracle import ERR_INDEX, reassign, reassign_batch


def _c1_coords():
    # 6x6 sub-grid, rows 5..10, cols 3..8 of a 16x16 image at t = 0
    return np.array([(0, h, w) for h in range(5, 11) for w in range(3, 9)])


def test_pcr_worked_example_tiny_workload():
    # p_txt = 299, L = 2, K = 36, h and w spans of 5:
    #   p = 297 + 3 (1 + 35 n / 5) / 37 = (10992 + 21 n) / 37,  n = 0..5
    # t is constant (degenerate), so it sits at the interval centre 297 + 3/2.
    pos, nxt = reassign(_c1_coords(), 299, "pcr", 2)
    assert nxt == 300
    vals = [float(Fraction(10992 + 21 * n, 37)) for n in range(6)]
    assert vals[0] == pytest.approx(297.08108108, abs=1e-8)
    assert vals[-1] == pytest.approx(299.91891892, abs=1e-8)
    c = _c1_coords()
    for j in range(36):
        assert pos[j, 0] == 298.5
        assert pos[j, 1] == vals[c[j, 1] - 5]
        assert pos[j, 2] == vals[c[j, 2] - 3]


def test_shift_worked_example_tiny_workload():
    pos, nxt = reassign(_c1_coords(), 299, "shift", 2)
    c = _c1_coords()
    assert np.array_equal(pos[:, 0], np.full(36, 300.0))
    assert np.array_equal(pos[:, 1], 300.0 + (c[:, 1] - 5))
    assert np.array_equal(pos[:, 2], 300.0 + (c[:, 2] - 3))
    assert nxt == 306


def test_identity_lpa_uir_examples():
    c = np.array([[0, 4, 9], [0, 2, 1], [1, 7, 7]])
    pos, nxt = reassign(c, 50, "identity")
    assert np.array_equal(pos, c.astype(float)) and nxt == 51
    pos, nxt = reassign(c, 50, "lpa")
    assert pos[:, 0].tolist() == [51.0, 52.0, 53.0] and nxt == 54
    assert np.array_equal(pos[:, 0], pos[:, 1]) and np.array_equal(pos[:, 1], pos[:, 2])
    pos, nxt = reassign(c, 50, "uir")
    assert pos[:, 2].tolist() == [50.25, 50.5, 50.75] and nxt == 51


def test_single_token_sits_at_interval_centre():
    for L in (0, 1, 2, 5):
        pos, nxt = reassign(np.array([[3, 9, 4]]), 1000, "pcr", L)
        assert np.array_equal(pos[0], np.full(3, (1000 - L) + (L + 1) / 2))
        assert nxt == 1001


def test_empty_selection():
    for mode in ("pcr", "shift", "identity", "uir", "pcr_right"):
        pos, nxt = reassign(np.zeros((0, 3), int), 77, mode)
        assert pos.shape == (0, 3) and nxt == 78
    assert reassign(np.zeros((0, 3), int), 77, "lpa")[1] == 78


coord = st.integers(min_value=-50, max_value=200)


@settings(max_examples=150, deadline=None)
@given(pts=st.lists(st.tuples(coord, coord, coord), min_size=1, max_size=40),
       p_txt=st.integers(min_value=0, max_value=200_000), L=st.integers(min_value=0, max_value=8))
def test_pcr_properties(pts, p_txt, L):
    c = np.array(pts, dtype=np.int64)
    K = len(c)
    pos, nxt = reassign(c, p_txt, "pcr", L)
    assert nxt == p_txt + 1                                  # next text position unchanged
    assert (pos > p_txt - L).all() and (pos < p_txt + 1).all()   # inside the interval
    for a in range(3):
        mn, mx = c[:, a].min(), c[:, a].max()
        if mx == mn:
            assert (pos[:, a] == (p_txt - L) + (L + 1) / 2).all()
            continue
        lo = float((p_txt - L) + Fraction(L + 1, K + 1))
        hi = float((p_txt - L) + Fraction((L + 1) * K, K + 1))
        assert pos[c[:, a] == mn, a].tolist() == [lo] * int((c[:, a] == mn).sum())
        assert pos[c[:, a] == mx, a].tolist() == [hi] * int((c[:, a] == mx).sum())
        # relative layout: order of coordinates is kept, ties stay tied
        order = np.argsort(c[:, a], kind="stable")
        assert (np.diff(pos[order, a]) >= 0).all()
        same = c[:, a][:, None] == c[:, a][None, :]
        assert ((pos[:, a][:, None] == pos[:, a][None, :]) == same).all()
    # invariance under per-axis translation and positive scaling of the coordinates
    shift = np.array([7, -3, 11])
    assert np.array_equal(reassign(c + shift, p_txt, "pcr", L)[0], pos)
    assert np.array_equal(reassign(c * 3, p_txt, "pcr", L)[0], pos)
    # permutation equivariance
    perm = np.random.default_rng(K).permutation(K)
    assert np.array_equal(reassign(c[perm], p_txt, "pcr", L)[0], pos[perm])


@settings(max_examples=60, deadline=None)
@given(pts=st.lists(st.tuples(coord, coord, coord), min_size=1, max_size=30),
       p_txt=st.integers(min_value=0, max_value=100_000))
def test_shift_properties(pts, p_txt):
    c = np.array(pts, dtype=np.int64)
    pos, nxt = reassign(c, p_txt, "shift")
    assert (pos.min(axis=0) == p_txt + 1).all()          # region starts at the current position
    assert np.array_equal(pos - pos[0], (c - c[0]).astype(float))   # relative layout kept
    assert nxt == pos.max() + 1


def test_batch_flags_and_skips_bad_indices():
    coords = np.zeros((2, 4, 3), np.int32)
    coords[0, :, 1] = [0, 1, 2, 3]
    coords[1, :, 2] = [5, 6, 7, 8]
    sel_off = np.array([0, 3, 5])
    sel_idx = np.array([0, 9, 3, 1, 2])          # 9 is out of range for sequence 0
    new_pos, nxt, err = reassign_batch(coords, np.array([4, 4]), sel_off, sel_idx,
                                       np.array([10, 20]), "pcr", 2)
    assert err == ERR_INDEX
    assert np.isnan(new_pos[1]).all()
    # the valid tokens of sequence 0 span h = 0..3 with K = 3
    assert new_pos[0, 1] == float(8 + Fraction(3, 4)) and new_pos[2, 1] == float(8 + Fraction(9, 4))
    assert nxt.tolist() == [11, 21]


@settings(max_examples=100, deadline=None)
@given(pts=st.lists(st.tuples(coord, coord, coord), min_size=1, max_size=30),
       p_txt=st.integers(min_value=0, max_value=200_000), L=st.integers(min_value=0, max_value=8))
def test_rightward_pcr_is_leftward_moved_past_the_next_text_position(pts, p_txt, L):
    """Reading R6: rightward re-anchoring puts the same relative layout in
    (p_txt + 1, p_txt + L + 2).  In exact arithmetic every coordinate is the
    leftward one plus L + 1.  The text position is not moved, so the entries sit
    on future text positions, which is the competition the ablation describes."""
    c = np.array(pts, dtype=np.int64)
    left, nl = reassign(c, p_txt, "pcr", L)
    right, nr = reassign(c, p_txt, "pcr_right", L)
    assert nl == nr == p_txt + 1
    assert (right > p_txt + 1).all() and (right < p_txt + L + 2).all()
    # each side is the correctly rounded double of its rational: compare in Fractions
    for j in range(len(c)):
        for a in range(3):
            assert Fraction(right[j, a]) - Fraction(left[j, a]) == pytest.approx(L + 1, abs=1e-9)


def test_rightward_pcr_worked_example_tiny_workload():
    # p_txt = 299, L = 2, K = 36: the interval starts at 300 instead of 297, so
    #   p = 300 + 3 (1 + 35 n / 5) / 37 = (11103 + 21 n) / 37,  n = 0..5; t at 301.5
    pos, nxt = reassign(_c1_coords(), 299, "pcr_right", 2)
    assert nxt == 300
    c = _c1_coords()
    vals = [float(Fraction(11103 + 21 * n, 37)) for n in range(6)]
    for j in range(36):
        assert pos[j, 0] == 301.5
        assert pos[j, 1] == vals[c[j, 1] - 5]
        assert pos[j, 2] == vals[c[j, 2] - 3]
