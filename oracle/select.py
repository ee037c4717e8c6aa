"""Token energy and the read keep-set (test infrastructure; see package doc).

Eq. 4 keeps, inside the prior P, at most floor(rho*mn) tokens with the largest
energy ||z_i||^2 (Sec. 3.1; Algorithm 1 ranks within the union prior).

Readings:
  * k = floor(rho*mn) is an integer computed by the caller (the keep-ratio
    ablation table lists 819, 1228, 2048, 2867, 4096 at mn = 4096);
  * energies are float64 sums of the exact squares, added in ascending channel
    order starting from +0.0, so any implementation that adds the same terms in
    the same order reproduces them bit for bit;
  * ties rank the lower cell index first; the kept list is returned ascending;
  * groups: one group = the union over all objects (the paper), or one group
    per object.
"""
from __future__ import annotations

from typing import List, Sequence

import numpy as np

from .geometry import Track, prior_object


def energy(X: np.ndarray) -> np.ndarray:
    """e_i = sum_c x_{i,c}^2 in float64, channels added in ascending order."""
    X = np.asarray(X, dtype=np.float64)
    e = np.zeros(X.shape[0], dtype=np.float64)
    for c in range(X.shape[1]):
        e = e + X[:, c] * X[:, c]
    return e


def topk_keep(P: np.ndarray, e: np.ndarray, k: int) -> np.ndarray:
    """Cells of P (flat bool) ranked by (energy desc, index asc); the first k,
    returned in ascending index order.  If |P| <= k all of P is kept."""
    cand = [int(i) for i in np.flatnonzero(np.asarray(P).reshape(-1))]
    if len(cand) > k:
        ranked = sorted(cand, key=lambda i: (-float(e[i]), i))
        cand = sorted(ranked[:k])
    return np.asarray(cand, dtype=np.int32)


def select_queries(masks: np.ndarray, s: int, m: int, n: int, tracks: List[Track],
                   X: np.ndarray, k: Sequence[int], r_s: int, c: int,
                   seed_box: bool = False, union_objects: bool = True):
    """Read keep-sets for one frame.

    masks : uint8 [n_obj][m*s][n*s], previous-frame masks per object
    X     : float64 [n_x][mn][C]; n_x = 1 (shared grid) or n_obj
    k     : per-group budgets
    Returns (sel: list of int32 arrays per group, priors: bool [n_groups][mn],
             new tracks)."""
    n_obj = masks.shape[0]
    priors_o, new_tracks = [], []
    for o in range(n_obj):
        P, tr = prior_object(masks[o], s, m, n, tracks[o], r_s, c, seed_box)
        priors_o.append(P.reshape(-1))
        new_tracks.append(tr)
    if union_objects:
        groups = [list(range(n_obj))]
    else:
        groups = [[o] for o in range(n_obj)]
    sel, priors = [], []
    for g, objs in enumerate(groups):
        Pg = np.zeros(m * n, dtype=bool)
        for o in objs:
            Pg |= priors_o[o]
        xi = 0 if X.shape[0] == 1 else objs[0]
        e = energy(X[xi])
        sel.append(topk_keep(Pg, e, int(k[g])))
        priors.append(Pg)
    return sel, np.stack(priors), new_tracks
