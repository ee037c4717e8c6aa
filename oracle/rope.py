"""Rotary positions on the gathered subset (test infrastructure; see package doc).

Sec. 3.1 ("RoPE on the sparse subset", Eq. 7): the memory attention rotates
its queries by a precomputed table f with one row of C/2 complex factors per
cell of the m x n grid.  After the query gather of Eq. 6, the table must be
gathered with the same keep-set, f~ = f[K_r], so that each kept query turns
by the factors of the cell it came from and not by those of its position in
the compacted list.  With keep-all the gather is the identity and the sparse
readout equals the dense one.

Readings (the paper gives the table's shape and the gather, nothing else):
  * channels 2p and 2p+1 of a head form the complex number x_2p + i x_2p+1,
    which is multiplied by f[cell][p] (a rotation: |f| = 1);
  * the heads share one table of d_h/2 columns (C/2 for the paper's single
    head);
  * bank keys are rotated by the row of the cell they were kept from (the
    position stored with each bank row); values are not rotated;
  * the table used by the measured workloads is the axial two-dimensional
    one: for p < d_h/4 the angle is column * theta^(-4p/d_h), for the other
    d_h/4 entries it is row * theta^(-4(p - d_h/4)/d_h), cell = row*n + col.
Parity of the axial construction itself is unpinned against the paper (it is
a reading); the tests pin its stated form through special cases and
invariants, and pin the gather (Eq. 7) through the keep-all and row
independence properties stated at the end of Sec. 3.1.
"""
from __future__ import annotations

import numpy as np


def axial_table(m: int, n: int, d_h: int, theta: float) -> np.ndarray:
    """Axial rotary table, complex128 [m*n][d_h/2] (see the module readings)."""
    if d_h % 4 != 0:
        raise ValueError("the axial table needs d_h divisible by 4")
    quarter = d_h // 4
    f = np.zeros((m * n, d_h // 2), dtype=np.complex128)
    for cell in range(m * n):
        row, col = divmod(cell, n)
        for p in range(quarter):
            freq = float(theta) ** (-4.0 * p / d_h)
            f[cell, p] = np.exp(1j * col * freq)
            f[cell, quarter + p] = np.exp(1j * row * freq)
    return f


def table_from_pairs(pairs: np.ndarray) -> np.ndarray:
    """[rows][d_h/2][2] (cos, sin) array -> complex128 table [rows][d_h/2]."""
    pairs = np.asarray(pairs, np.float64)
    return pairs[..., 0] + 1j * pairs[..., 1]


def rotate(v: np.ndarray, f_row: np.ndarray) -> np.ndarray:
    """One head-width vector v (real, even length) turned by the complex
    factors f_row (length len(v)/2): pair p becomes (v_2p + i v_2p+1) f_row[p]."""
    v = np.asarray(v, np.float64)
    z = (v[0::2] + 1j * v[1::2]) * np.asarray(f_row, np.complex128)
    out = np.empty_like(v)
    out[0::2] = z.real
    out[1::2] = z.imag
    return out


def rotate_heads(v: np.ndarray, f_row: np.ndarray, H: int) -> np.ndarray:
    """A D-wide row of H heads, each head turned by the same f_row."""
    v = np.asarray(v, np.float64)
    d_h = v.shape[0] // H
    return np.concatenate([rotate(v[h * d_h:(h + 1) * d_h], f_row) for h in range(H)])
