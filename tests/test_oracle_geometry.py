"""Pins for the oracle's prior geometry (Sec. 3.1, Eqs. 1, 2, 5; Algorithm 1)."""
import json
import os

import numpy as np
import pytest

import oracle
from oracle import Track


def _separable_dilate(A, r):
    """Square dilation as a row pass then a column pass of running maxima
    (the textbook decomposition of a square structuring element)."""
    A = np.asarray(A, dtype=bool)
    m, n = A.shape
    rows = np.zeros_like(A)
    for x in range(n):
        rows[:, x] = A[:, max(0, x - r):x + r + 1].any(axis=1)
    out = np.zeros_like(A)
    for y in range(m):
        out[y, :] = rows[max(0, y - r):y + r + 1, :].any(axis=0)
    return out


def _box_count(box, r, m, n):
    y0, x0, y1, x1 = box
    return (min(m - 1, y1 + r) - max(0, y0 - r) + 1) * (min(n - 1, x1 + r) - max(0, x0 - r) + 1)


def test_dilate_golden(golden_dir):
    g = json.load(open(os.path.join(golden_dir, "dilate_6x7.json")))
    A = np.zeros((g["m"], g["n"]), dtype=bool)
    for y, x in g["cells"]:
        A[y, x] = True
    for r, rows in g["expected"].items():
        exp = np.array([[c == "1" for c in row] for row in rows])
        np.testing.assert_array_equal(oracle.dilate(A, int(r)), exp)


@pytest.mark.parametrize("seed", range(6))
def test_dilate_matches_separable(seed):
    rng = np.random.default_rng(seed)
    m, n = rng.integers(3, 30, size=2)
    A = rng.random((m, n)) < rng.uniform(0.01, 0.3)
    for r in (0, 1, 2, 4, 7, 40):
        np.testing.assert_array_equal(oracle.dilate(A, r), _separable_dilate(A, r))


def test_dilate_identity_and_monotone():
    rng = np.random.default_rng(7)
    A = rng.random((20, 17)) < 0.1
    np.testing.assert_array_equal(oracle.dilate(A, 0), A)
    prev = A
    for r in range(1, 8):
        cur = oracle.dilate(A, r)
        assert np.all(cur >= prev)
        prev = cur


def test_box_closed_form():
    m, n = 40, 33
    for box in [(0, 0, 0, 0), (5, 7, 9, 20), (30, 1, 39, 32), (12, 12, 12, 30)]:
        for r in (0, 1, 3, 9, 50):
            P = oracle.dilate(oracle.fill_box(box, m, n), r)
            assert P.sum() == _box_count(box, r, m, n)


def test_down_s_and_bbox():
    M = np.zeros((8, 12), dtype=np.uint8)
    M[2, 5] = 1
    M[6, 2] = 1
    assert oracle.bbox(M) == (2, 2, 6, 5)
    assert oracle.bbox(np.zeros((3, 3))) is None
    np.testing.assert_array_equal(oracle.down_s(M, 1), M.astype(bool))
    # stride 2 samples pixel (2y, 2x): (2,5) is odd-x -> dropped, (6,2) -> cell (3,1)
    d = oracle.down_s(M, 2)
    assert d.shape == (4, 6)
    assert d.sum() == 1 and d[3, 1]
    assert oracle.down_s_box((2, 2, 6, 5), 2) == (1, 1, 3, 2)


def test_streak_radii_and_reset():
    """Algorithm 1: the radius is r_s + min(streak, c) while the object is
    missing, and the streak resets when it reappears."""
    m = n = 64
    r_s, c = 4, 14
    M = np.zeros((m, n), dtype=np.uint8)
    M[10:21, 12:16] = 1
    box = (10, 12, 20, 15)
    empty = np.zeros_like(M)
    tr = Track()
    P, tr = oracle.prior_object(M, 1, m, n, tr, r_s, c)
    assert tr.box == box and tr.delta == 0 and tr.has_box == 1
    assert P.sum() == _box_count(box, r_s, m, n)  # the mask is its own box here
    for d in range(1, 21):
        P, tr = oracle.prior_object(empty, 1, m, n, tr, r_s, c)
        assert tr.delta == d
        assert P.sum() == _box_count(box, r_s + min(d, c), m, n)
    M2 = np.zeros_like(M)
    M2[40, 40] = 1
    P, tr = oracle.prior_object(M2, 1, m, n, tr, r_s, c)
    assert tr.delta == 0 and tr.box == (40, 40, 40, 40)
    assert P.sum() == (2 * r_s + 1) ** 2


def test_no_box_yet_is_empty_prior():
    tr = Track()
    P, tr2 = oracle.prior_object(np.zeros((9, 9), np.uint8), 1, 9, 9, tr, 4, 14)
    assert P.sum() == 0 and tr2.has_box == 0 and tr2.delta == 1


def test_seed_box_mode():
    m = n = 32
    M = np.zeros((m, n), dtype=np.uint8)
    M[3, 4] = 1
    M[9, 20] = 1
    P, tr = oracle.prior_object(M, 1, m, n, Track(), 2, 14, seed_box=True)
    assert P.sum() == _box_count((3, 4, 9, 20), 2, m, n)
    P2, _ = oracle.prior_object(M, 1, m, n, Track(), 2, 14, seed_box=False)
    assert P2.sum() == 2 * 25


def test_union_bounds():
    rng = np.random.default_rng(3)
    m, n = 24, 24
    masks = (rng.random((3, m, n)) < 0.02).astype(np.uint8)
    X = rng.standard_normal((1, m * n, 8))
    tracks = [Track()] * 3
    sel, priors, _ = oracle.select_queries(masks, 1, m, n, tracks, X, [m * n], 2, 14, union_objects=True)
    per = [oracle.prior_object(masks[o], 1, m, n, Track(), 2, 14)[0].reshape(-1) for o in range(3)]
    Pg = priors[0]
    for p in per:
        assert np.all(Pg >= p)
    assert Pg.sum() <= sum(p.sum() for p in per)
    assert Pg.sum() == np.logical_or.reduce(per).sum()
