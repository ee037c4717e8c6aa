"""Pins for the oracle's fixed write keep-set (Sec. 3.2, Eq. 8; the
fall-through and the containment statement of Sec. 3.2 and of the discussion
of Algorithm 1)."""
import numpy as np
import pytest

import oracle
from workloads import fall_counts


def _brute_keep(foot, D):
    """Cell kept iff some footprint cell lies within Chebyshev distance D."""
    m, n = foot.shape
    pts = list(zip(*np.nonzero(foot)))
    out = np.zeros((m, n), dtype=bool)
    for y in range(m):
        for x in range(n):
            out[y, x] = any(max(abs(y - py), abs(x - px)) <= D for py, px in pts)
    return out


def _rand_masks(rng, n_obj, H, W, p):
    return (rng.random((n_obj, H, W)) < p).astype(np.uint8)


@pytest.mark.parametrize("s,D", [(1, 0), (1, 2), (2, 3), (1, 24)])
def test_keepset_is_union_of_dilated_footprints(s, D):
    rng = np.random.default_rng(10 + D)
    m, n = 9, 11
    seeds = _rand_masks(rng, 3, m * s, n * s, 0.02)
    keep, count, fell = oracle.write_keepset(seeds, s, m, n, D)
    assert not fell
    foot = np.zeros((m, n), dtype=bool)
    for M in seeds:
        foot |= M[::s, ::s].astype(bool)   # nearest-neighbour sample (y*s, x*s)
    assert count == int(foot.sum())
    assert np.array_equal(keep, _brute_keep(foot, D))
    if D == 0:
        assert np.array_equal(keep, foot)


def test_keepset_grows_with_D_w_and_contains_the_footprint():
    rng = np.random.default_rng(3)
    seeds = _rand_masks(rng, 2, 20, 20, 0.01)
    prev = None
    for D in range(0, 8):
        keep, count, _ = oracle.write_keepset(seeds, 1, 20, 20, D)
        if prev is not None:
            assert np.all(keep >= prev)
        prev = keep
    foot = seeds.any(axis=0)
    assert np.all(prev[foot])


def test_fall_through_thresholds_are_strict():
    m = n = 10
    mn = m * n
    lo, hi = fall_counts(0.05, 0.95, mn)   # count < 5 or > 95 falls through
    assert (lo, hi) == (5, 95)
    for cnt, falls in ((4, True), (5, False), (95, False), (96, True), (0, True)):
        seed = np.zeros((1, m, n), np.uint8)
        seed.reshape(-1)[:cnt] = 1
        keep, count, fell = oracle.write_keepset(seed, 1, m, n, 2, lo, hi)
        assert count == cnt and fell == falls
        if falls:
            assert keep.all()
        else:
            assert np.array_equal(keep, _brute_keep(seed[0].astype(bool), 2))


def test_fall_through_is_decided_before_dilation():
    # a footprint just above 5 % stays pruned even when its dilation covers
    # almost the whole grid
    m = n = 20
    lo, hi = fall_counts(0.05, 0.95, m * n)
    seed = np.zeros((1, m, n), np.uint8)
    seed[0, 10, 0:20] = 1            # 20 cells = 5 %
    keep, count, fell = oracle.write_keepset(seed, 1, m, n, 9, lo, hi)
    assert count == 20 and not fell
    assert keep.sum() == 19 * 20      # rows 1..19


def _track_run(seed_px, masks_px, s, m, n, r_s, c):
    """Priors of a mask sequence after the seed, by the oracle's tracker."""
    P, tr = oracle.prior_object(seed_px, s, m, n, oracle.Track(), r_s, c)
    out = [P]
    for M in masks_px:
        P, tr = oracle.prior_object(M, s, m, n, tr, r_s, c)
        out.append(P)
    return out


def test_containment_when_masks_stay_inside_the_seed():
    # D_w >= r_s + c and every later mask inside the seed footprint: the
    # read prior stays inside K_w, through the streak fallback too when the
    # seed is its own bounding box (a filled rectangle)
    r_s, c = 4, 14
    m = n = 64
    seed = np.zeros((m, n), np.uint8)
    seed[20:35, 25:40] = 1
    keep, _, _ = oracle.write_keepset(seed[None], 1, m, n, r_s + c)
    rng = np.random.default_rng(7)
    later = [(seed * (rng.random((m, n)) < 0.6)).astype(np.uint8) for _ in range(3)]
    later += [np.zeros((m, n), np.uint8)] * (c + 3)   # streak beyond the cap
    for P in _track_run(seed, later, 1, m, n, r_s, c):
        assert np.all(keep[P])
    # with a smaller D_w the capped box fallback leaves K_w
    small, _, _ = oracle.write_keepset(seed[None], 1, m, n, r_s + c - 1)
    assert not all(np.all(small[P]) for P in _track_run(seed, later, 1, m, n, r_s, c))


def test_containment_fails_for_a_box_far_from_the_mask():
    # the stated containment is conditional: an L-shaped seed's bounding box
    # has a corner farther than D_w from every seed cell, and the streak
    # fallback dilates that box
    r_s, c = 1, 2
    m = n = 40
    seed = np.zeros((m, n), np.uint8)
    seed[5:35, 5] = 1
    seed[34, 5:35] = 1
    keep, _, _ = oracle.write_keepset(seed[None], 1, m, n, r_s + c)
    priors = _track_run(seed, [seed, np.zeros((m, n), np.uint8)], 1, m, n, r_s, c)
    assert np.all(keep[priors[1]])          # mask path: inside
    assert not np.all(keep[priors[2]])      # box path: corner (5, 34) region outside


def test_fixed_keepset_gives_a_constant_stride():
    # every write stores |K_w| rows, so unpinned frames sit in fixed slots
    # pin_end + j*|K_w| of a ring sized for them
    rng = np.random.default_rng(1)
    m = n = 12
    seed = np.zeros((1, m, n), np.uint8)
    seed[0, 4:7, 3:8] = 1
    keep, _, _ = oracle.write_keepset(seed, 1, m, n, 1)
    L = int(keep.sum())
    n_slots, f_max = 3, 4
    ring = oracle.RingBank(L + n_slots * L, f_max, 1, 4, np.float32)
    mask = keep.astype(np.uint8).reshape(-1)
    starts = []
    for t in range(9):
        K = rng.standard_normal((m * n, 4)).astype(np.float32)
        assert ring.commit(K, K, mask, t, t == 0) == L
        if t > 0:
            newest = ring.frames[-1]
            starts.append((newest.start, newest.length))
    assert ring.pin_end == L
    assert all(ln == L for _, ln in starts)
    assert [st for st, _ in starts] == [L + L * (j % n_slots) for j in range(8)]
