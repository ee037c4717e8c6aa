"""Pins for the oracle's closure of the decoded masks and the palette argmax
(Sec. 3.3 and the end of Algorithm 1)."""
import numpy as np
import pytest
from scipy import ndimage

import oracle.post as post


def _scipy_close(B, k):
    # the same closing by the library: dilation with the outside unset, then
    # erosion with the outside counted as set
    se = np.ones((k, k), dtype=bool)
    d = ndimage.binary_dilation(B, structure=se, border_value=0)
    return ndimage.binary_erosion(d, structure=se, border_value=1)


@pytest.mark.parametrize("k,p", [(9, 0.03), (9, 0.3), (3, 0.1), (5, 0.6), (1, 0.2)])
def test_closing_matches_the_library(k, p):
    rng = np.random.default_rng(k * 10 + int(p * 100))
    B = rng.random((37, 29)) < p
    assert np.array_equal(post.close_square(B, k), _scipy_close(B, k))


def test_closing_fills_holes_smaller_than_the_element():
    # a filled square with an interior hole: holes up to 8x8 close under 9x9,
    # a 9x9 hole does not (dilation shrinks it to one pixel, erosion regrows it)
    for hole, filled in ((1, True), (5, True), (8, True), (9, False), (12, False)):
        B = np.zeros((60, 60), dtype=bool)
        B[10:50, 10:50] = True
        B[20:20 + hole, 20:20 + hole] = False
        C = post.close_square(B, 9)
        assert C[20:20 + hole, 20:20 + hole].all() == filled
        assert np.array_equal(C[10:50, 10:50] | ~B[10:50, 10:50], np.ones((40, 40), bool))


def test_closing_keeps_the_outer_boundary_and_is_extensive():
    # a rectangle (convex) is unchanged, also when it touches the border; any
    # mask is contained in its closing; closing twice changes nothing
    for box in ((5, 20, 7, 30), (0, 12, 0, 9), (30, 40, 25, 40)):
        B = np.zeros((40, 40), dtype=bool)
        B[box[0]:box[1], box[2]:box[3]] = True
        assert np.array_equal(post.close_square(B, 9), B)
    rng = np.random.default_rng(1)
    for _ in range(5):
        B = rng.random((30, 33)) < 0.15
        C = post.close_square(B, 9)
        assert np.all(C[B])
        assert np.array_equal(post.close_square(C, 9), C)


def test_thin_gap_is_reknit():
    B = np.zeros((30, 40), dtype=bool)
    B[10:20, 5:18] = True
    B[10:20, 22:35] = True          # a 4-pixel gap between two blocks
    C = post.close_square(B, 9)
    assert C[10:20, 18:22].all()
    assert not C[:10].any() and not C[20:].any()


def test_palette_by_brute_force_and_ties():
    rng = np.random.default_rng(4)
    L = rng.standard_normal((3, 12, 13))
    closed = rng.random((3, 12, 13)) < 0.5
    P = post.palette(L, closed)
    for y in range(12):
        for x in range(13):
            cov = [o for o in range(3) if closed[o, y, x]]
            if not cov:
                assert P[y, x] == 0
            else:
                assert P[y, x] == 1 + max(cov, key=lambda o: (L[o, y, x], -o))
    # equal logits: the lower object index wins
    L2 = np.zeros((2, 2, 2))
    assert np.array_equal(post.palette(L2, np.ones((2, 2, 2), bool)), np.ones((2, 2), np.uint8))


def test_close_masks_hole_takes_the_covering_object():
    # a pixel inside object 1's hole with a larger logit of object 0 that
    # does not cover it: the closed object 1 owns it
    L = -np.ones((2, 20, 20))
    L[1, 5:15, 5:15] = 2.0
    L[1, 9, 9] = -3.0               # a hole of object 1
    L[0, 9, 9] = -0.5               # object 0 is not set there
    closed, P = post.close_masks(L, 9)
    assert closed[1, 9, 9] == 1 and closed[0].sum() == 0
    assert P[9, 9] == 2 and P[0, 0] == 0
    assert (P == 2).sum() == 100
