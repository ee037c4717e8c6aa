"""Pins for the oracle's energy ranking and read keep-set (Sec. 3.1, Eq. 4)."""
import itertools
import json
import math
import os

import numpy as np
import pytest

import oracle
from workloads import k_from_rho


def test_keep_budget_matches_table(golden_dir):
    g = json.load(open(os.path.join(golden_dir, "keep_ratio_table.json")))
    for rho, kmax in g["rows"]:
        assert k_from_rho(rho, g["mn"]) == kmax
    # rounding instead of flooring would give 1229 at rho = 0.3
    assert round(0.3 * 4096) == 1229


def test_energy_integer_inputs_exact():
    rng = np.random.default_rng(0)
    X = rng.integers(-50, 50, size=(40, 33)).astype(np.float64)
    e = oracle.energy(X)
    exact = [sum(int(v) * int(v) for v in row) for row in X]
    assert [int(v) for v in e] == exact


def test_energy_channel_order():
    """Ascending-order accumulation from +0.0: four squares of 2^-54 after 1.0
    are each absorbed, while the exact sum 1 + 2^-52 is representable."""
    a = 2.0 ** -27
    e_fwd = oracle.energy(np.array([[1.0, a, a, a, a]]))[0]
    e_rev = oracle.energy(np.array([[a, a, a, a, 1.0]]))[0]
    assert e_fwd == 1.0
    assert e_rev == 1.0 + 2.0 ** -52


def test_energy_error_bound():
    rng = np.random.default_rng(1)
    X = rng.standard_normal((200, 256)).astype(np.float32).astype(np.float64)
    e = oracle.energy(X)
    for i in range(0, 200, 17):
        ex = math.fsum(float(v) * float(v) for v in X[i])
        assert abs(e[i] - ex) <= 255 * 2.0 ** -53 * ex


def _check_topk(P, e, k, sel):
    cand = np.flatnonzero(P)
    assert len(sel) == min(len(cand), k)
    assert np.all(np.diff(sel) > 0)
    assert set(sel.tolist()) <= set(cand.tolist())
    rest = sorted(set(cand.tolist()) - set(sel.tolist()))
    if len(sel) and rest:
        worst_kept = min((e[i], -i) for i in sel)
        best_dropped = max((e[i], -i) for i in rest)
        assert worst_kept > best_dropped


@pytest.mark.parametrize("seed", range(10))
def test_topk_characterisation(seed):
    rng = np.random.default_rng(seed)
    mn = int(rng.integers(1, 60))
    P = rng.random(mn) < 0.6
    e = rng.integers(0, 6, size=mn).astype(np.float64)   # many ties
    for k in (0, 1, 3, mn // 2, mn):
        _check_topk(P, e, k, oracle.topk_keep(P, e, k))


def test_topk_brute_force_tiny():
    """Among all k-subsets of P, the kept set is the unique one whose sorted
    key list (energy desc, index asc) is lexicographically largest."""
    rng = np.random.default_rng(11)
    for _ in range(30):
        mn = int(rng.integers(1, 9))
        P = rng.random(mn) < 0.7
        e = rng.integers(0, 3, size=mn).astype(np.float64)
        cand = np.flatnonzero(P).tolist()
        for k in range(0, len(cand) + 1):
            best = max(itertools.combinations(cand, k),
                       key=lambda S: sorted(((e[i], -i) for i in S), reverse=True))
            assert oracle.topk_keep(P, e, k).tolist() == sorted(best)


def test_topk_special_cases():
    mn = 50
    P = np.zeros(mn, bool)
    P[[3, 7, 8, 20, 41]] = True
    e = np.ones(mn)
    assert oracle.topk_keep(P, e, 3).tolist() == [3, 7, 8]
    assert oracle.topk_keep(np.ones(mn, bool), np.random.default_rng(0).random(mn), mn).tolist() == list(range(mn))
    assert oracle.topk_keep(P, e, 0).tolist() == []
    assert oracle.topk_keep(np.zeros(mn, bool), e, 10).tolist() == []
    # a hand example: energies 5,9,9,1 on cells 0..3, k = 2 -> cells 1 and 2
    assert oracle.topk_keep(np.ones(4, bool), np.array([5.0, 9, 9, 1]), 2).tolist() == [1, 2]
    assert oracle.topk_keep(np.ones(4, bool), np.array([9.0, 5, 9, 9]), 2).tolist() == [0, 2]


def _brute_prior(mask_px, s, m, n, r):
    """Chebyshev dilation by r of the down-sampled mask, one cell at a time."""
    cells = [(y, x) for y in range(m) for x in range(n) if mask_px[y * s, x * s]]
    P = np.zeros(m * n, dtype=bool)
    for y in range(m):
        for x in range(n):
            P[y * n + x] = any(max(abs(y - yy), abs(x - xx)) <= r for yy, xx in cells)
    return P


@pytest.mark.parametrize("shared_x", [True, False])
def test_per_object_groups(shared_x):
    """union_objects = False: group o is object o alone, ranked on its own
    token grid (shared or per object) with its own budget k[o].  Each group
    must equal a one-object call on that object, and a brute-force prior,
    integer energy and full sort; the tracker states must match too."""
    rng = np.random.default_rng(11)
    m, n, s, C, n_obj, r_s, c = 12, 10, 2, 6, 3, 2, 3
    n_x = 1 if shared_x else n_obj
    # integer-valued tokens: the energies are exact integers, and each
    # object's grid differs, so ranking on another object's grid shows
    X = rng.integers(-9, 10, size=(n_x, m * n, C)).astype(np.float64)
    k = [5, 17, 60]
    tracks = [oracle.Track() for _ in range(n_obj)]
    single = [oracle.Track() for _ in range(n_obj)]
    for frame in range(3):
        masks = (rng.random((n_obj, m * s, n * s)) < 0.04).astype(np.uint8)
        if frame == 2:
            masks[1] = 0      # object 1 lost: its cached box with a grown radius
        sel, pri, tracks = oracle.select_queries(masks, s, m, n, tracks, X, k, r_s, c, False, False)
        assert pri.shape == (n_obj, m * n)
        for o in range(n_obj):
            xo = 0 if shared_x else o
            so, po, to = oracle.select_queries(masks[o:o + 1], s, m, n, [single[o]], X[xo:xo + 1], [k[o]],
                                               r_s, c, False, True)
            single[o] = to[0]
            assert np.array_equal(sel[o], so[0])
            assert np.array_equal(pri[o], po[0])
            assert tracks[o].as_list() == single[o].as_list()
            # brute force: prior, exact integer energies, full sort
            if masks[o].any():
                bp = _brute_prior(masks[o], s, m, n, r_s)
            else:
                y0, x0, y1, x1 = (v // s for v in tracks[o].box)
                r = r_s + min(tracks[o].delta, c)
                bp = np.zeros(m * n, dtype=bool)
                for y in range(m):
                    for x in range(n):
                        bp[y * n + x] = (y0 - r <= y <= y1 + r) and (x0 - r <= x <= x1 + r)
            assert np.array_equal(pri[o], bp)
            e = [sum(int(v) * int(v) for v in X[xo, i]) for i in range(m * n)]
            ranked = sorted(np.flatnonzero(bp).tolist(), key=lambda i: (-e[i], i))
            assert sel[o].tolist() == sorted(ranked[:k[o]])
    # the objects' lists differ, so a group ranked on the wrong grid, with the
    # wrong budget or the wrong prior would have shown above
    assert len({tuple(v.tolist()) for v in sel}) == n_obj
