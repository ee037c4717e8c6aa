"""The paper's own write keep-set (test infrastructure; see package doc).

Sec. 3.2, Eq. 8: for every object, take its mask in the frame tau_o where it
is first seen, reduce it to the encoder grid by nearest-neighbour sampling
and grow it by D_w cells; K_w is the union of the grown regions.  It is computed once and
every later write of the sequence stores the tokens at K_w, so each stored
frame has the same |K_w| tokens (a constant per-frame stride).  When the
seed footprint covers more than 95 % or less than 5 % of the grid, the write
falls through to the dense path (every cell).  With D_w >= r_s + c the
read-side prior stays inside K_w (Sec. 3.2 and the discussion of Algorithm 1;
this holds while the predicted masks stay inside the seed footprint and the
prior is built from a mask, see the tests).

Readings:
  * the fall-through is decided on the undilated footprint (the union of the
    down-sampled seed masks), with strict thresholds given as integer counts:
    count < fall_min or count > fall_max;
  * an empty footprint falls through like any footprint below the lower
    threshold;
  * dilation is the Chebyshev radius of `geometry.dilate`.
"""
from __future__ import annotations

from typing import Optional

import numpy as np

from .geometry import dilate, down_s


def write_keepset(seed_masks, s: int, m: int, n: int, D_w: int, fall_min: int = 0,
                  fall_max: Optional[int] = None):
    """seed_masks: [n_obj][m*s][n*s] pixel masks at each object's first
    frame.  Returns (keep bool [m][n], footprint count, fell_through)."""
    grids = [down_s(np.asarray(M), s).astype(bool) for M in seed_masks]
    foot = np.zeros((m, n), dtype=bool)
    for g in grids:
        foot |= g
    count = int(foot.sum())
    if fall_max is None:
        fall_max = m * n
    if count < fall_min or count > fall_max:
        return np.ones((m, n), dtype=bool), count, True
    keep = np.zeros((m, n), dtype=bool)
    for g in grids:                 # Eq. 8: union of the per-object dilations
        keep |= dilate(g, D_w)
    return keep, count, False
