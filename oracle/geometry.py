"""Grid geometry of the read-side prior (test infrastructure; see package doc).

Sec. 3.1 builds the spatial prior from per-object masks: project to the token
grid by nearest-neighbour down-sampling with stride s (pixel coordinates
divided by s), then dilate by a radius counted in grid cells (Eqs. 1 and 2).
When an object's previous mask is empty, its cached bounding box is dilated by
a radius that grows with the empty streak, capped at r_s + c (Eq. 5), and the
box/streak state is updated as in Algorithm 1 (per-frame tracker update).

Readings taken where the text is silent or inconsistent:
  * cell index i = y*n + x (row-major);
  * down-sampling samples pixel (y*s, x*s) for cell (y, x); boxes map their
    inclusive pixel corners by floor division;
  * dilate_r is the Chebyshev (square) dilation of radius r, clipped at the
    border -- the text counts the radius in grid cells; its mention of an
    (r_s-1)x(r_s-1) element would grow a set by one cell and is not followed;
  * boxes are filled inclusive rectangles;
  * the streak update that Algorithm 1 performs after decoding frame t-1 is
    applied at the start of the selection for frame t, which yields the same
    radii (r_s+1 on the first empty frame, up to r_s+c).
"""
from __future__ import annotations

from dataclasses import dataclass, replace
from typing import Optional, Tuple

import numpy as np

Box = Tuple[int, int, int, int]   # (y0, x0, y1, x1), inclusive, pixel coordinates


@dataclass(frozen=True)
class Track:
    """Per-object tracker state: last non-empty box and the empty streak."""
    y0: int = 0
    x0: int = 0
    y1: int = 0
    x1: int = 0
    delta: int = 0
    has_box: int = 0

    @property
    def box(self) -> Box:
        return (self.y0, self.x0, self.y1, self.x1)

    def as_list(self):
        return [self.y0, self.x0, self.y1, self.x1, self.delta, self.has_box]


def down_s(M: np.ndarray, s: int) -> np.ndarray:
    """Nearest-neighbour projection of a pixel mask to the token grid:
    cell (y, x) takes pixel (y*s, x*s)."""
    return np.asarray(M)[::s, ::s].astype(bool)


def bbox(M: np.ndarray) -> Optional[Box]:
    """Tight inclusive bounding box of the set pixels, or None if empty."""
    ys, xs = np.nonzero(np.asarray(M))
    if ys.size == 0:
        return None
    return (int(ys.min()), int(xs.min()), int(ys.max()), int(xs.max()))


def down_s_box(box: Box, s: int) -> Box:
    """Pixel box -> grid box by flooring each inclusive corner."""
    y0, x0, y1, x1 = box
    return (y0 // s, x0 // s, y1 // s, x1 // s)


def fill_box(box: Box, m: int, n: int) -> np.ndarray:
    """Filled inclusive rectangle on the m x n grid."""
    A = np.zeros((m, n), dtype=bool)
    y0, x0, y1, x1 = box
    A[y0:y1 + 1, x0:x1 + 1] = True
    return A


def dilate(A: np.ndarray, r: int) -> np.ndarray:
    """Chebyshev dilation by r cells, by its definition: a cell is set iff some
    set cell of A lies within max(|dy|, |dx|) <= r of it."""
    A = np.asarray(A, dtype=bool)
    m, n = A.shape
    out = np.zeros((m, n), dtype=bool)
    for y, x in zip(*np.nonzero(A)):
        out[max(0, y - r):y + r + 1, max(0, x - r):x + r + 1] = True
    return out


def prior_object(M: np.ndarray, s: int, m: int, n: int, tr: Track,
                 r_s: int, c: int, seed_box: bool = False):
    """One object's prior for the current frame and its updated tracker state.

    M is the object's previous-frame mask at pixel resolution (m*s x n*s).
      non-empty : prior = dilate_{r_s}(down_s(M))            (Eq. 2)
                  or, on a seed frame, the dilated filled box (Eq. 1);
                  the cached box becomes bbox(M) and the streak resets;
      empty     : the streak grows by one; with a cached box the prior is
                  dilate_{r_s + min(streak, c)}(down_s(box))   (Eq. 5),
                  otherwise it is empty.
    Returns (bool [m][n], Track)."""
    b = bbox(M)
    if b is not None:
        if seed_box:
            base = fill_box(down_s_box(b, s), m, n)
        else:
            base = down_s(M, s)
        P = dilate(base, r_s)
        return P, Track(b[0], b[1], b[2], b[3], 0, 1)
    d = tr.delta + 1
    tr2 = replace(tr, delta=d)
    if tr.has_box:
        P = dilate(fill_box(down_s_box(tr.box, s), m, n), r_s + min(d, c))
    else:
        P = np.zeros((m, n), dtype=bool)
    return P, tr2
