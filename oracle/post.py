"""Per-frame closure of the decoded masks and the palette argmax (test
infrastructure; see package doc).

Sec. 3.3 and the end of Algorithm 1: each object's predicted binary mask is
closed with a k x k square structuring element (k = 9 in the paper): first
dilated, then eroded, on the full-resolution decoder output; only
then is the per-pixel argmax over objects taken to give the palette mask.
The closed masks are what the tracker state of the next frame is updated
from (bounding box or streak, Eq. 5).

Readings (the paper names the operations, not their conventions):
  * an object's binary mask is logit > 0 (probability above one half);
  * the dilation ignores pixels outside the image (they are unset) and the
    erosion ignores them too (they count as set), so the closing never
    shrinks a mask, also at the image border;
  * palette value 0 is background; otherwise 1 + the object with the largest
    logit among the objects whose closed mask covers the pixel, the lowest
    index on ties; a pixel no closed mask covers is background.
"""
from __future__ import annotations

import numpy as np


def binarize(logits: np.ndarray) -> np.ndarray:
    return np.asarray(logits, np.float64) > 0.0


def dilate_square(B: np.ndarray, k: int) -> np.ndarray:
    """k x k (k odd) square dilation: a pixel is set iff some set pixel of B
    lies in the k x k window centred on it (window clipped to the image)."""
    B = np.asarray(B, dtype=bool)
    H, W = B.shape
    r = k // 2
    out = np.zeros((H, W), dtype=bool)
    for y in range(H):
        for x in range(W):
            out[y, x] = B[max(0, y - r):y + r + 1, max(0, x - r):x + r + 1].any()
    return out


def erode_square(B: np.ndarray, k: int) -> np.ndarray:
    """k x k square erosion: a pixel stays set iff every in-image pixel of the
    window centred on it is set (outside pixels do not count)."""
    B = np.asarray(B, dtype=bool)
    H, W = B.shape
    r = k // 2
    out = np.zeros((H, W), dtype=bool)
    for y in range(H):
        for x in range(W):
            out[y, x] = B[max(0, y - r):y + r + 1, max(0, x - r):x + r + 1].all()
    return out


def close_square(B: np.ndarray, k: int) -> np.ndarray:
    """Closing: dilation, then erosion, with the same k x k square."""
    return erode_square(dilate_square(B, k), k)


def palette(logits: np.ndarray, closed: np.ndarray) -> np.ndarray:
    """Per-pixel argmax over the objects covering the pixel (see readings).
    logits, closed: [n_obj][H][W].  Returns uint8 [H][W]."""
    L = np.asarray(logits, np.float64)
    C = np.asarray(closed, dtype=bool)
    n_obj, H, W = L.shape
    out = np.zeros((H, W), dtype=np.uint8)
    for y in range(H):
        for x in range(W):
            best, arg = None, -1
            for o in range(n_obj):
                if C[o, y, x] and (best is None or L[o, y, x] > best):
                    best, arg = L[o, y, x], o
            out[y, x] = arg + 1
    return out


def close_masks(logits: np.ndarray, k: int):
    """The whole step: (closed masks uint8 [n_obj][H][W], palette [H][W])."""
    L = np.asarray(logits, np.float64)
    closed = np.stack([close_square(binarize(L[o]), k) for o in range(L.shape[0])])
    return closed.astype(np.uint8), palette(L, closed)
