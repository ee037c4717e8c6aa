"""Sparse memory readout (test infrastructure; see package doc).

Eq. 6 gathers the kept queries, runs softmax attention against the memory
bank on those rows only, and scatters the result back to the mn-row grid with
zeros elsewhere (Sec. 3.1, "Sparse memory attention"; Algorithm 1).

Readings:
  * the readout returns the residual stream Y = X + S(A): rows outside the
    keep-set receive a zero update and are returned as the input values, bit
    for bit (not as x + 0.0, which would turn -0.0 into +0.0);
  * the layer is one cross-attention of SAM2's shape: q = x W_q (C -> D),
    bank keys/values are projected K^ = K W_k, V^ = V W_v (d_kv -> D), H heads
    of width d_h = D/H over column blocks, logits scaled by 1/sqrt(d_h) (the
    C_k of Eq. 6), output o W_o (D -> C);
  * with an empty bank or an empty keep-set, Y = X.
At keep-all the gather and scatter are identities and the readout equals the
dense layer (end of Sec. 3.1), which `readout_dense` computes independently.

With a rotary table (Eq. 7, readings in `rope`), each kept query is turned by
the table row of its own cell and each bank key by the row of the cell stored
with it; `readout_dense` turns its rows by the cells it is given.
"""
from __future__ import annotations

import math

import numpy as np

from .rope import rotate_heads


def project_bank(Kraw: np.ndarray, Vraw: np.ndarray, Wk: np.ndarray, Wv: np.ndarray):
    """Bank keys and values in the attention space: K^ = K W_k, V^ = V W_v."""
    return (np.asarray(Kraw, np.float64) @ np.asarray(Wk, np.float64),
            np.asarray(Vraw, np.float64) @ np.asarray(Wv, np.float64))


def rotate_keys(Kh: np.ndarray, rope, kpos, H: int) -> np.ndarray:
    """Projected bank keys turned by the table rows of their stored cells
    (unchanged without a table)."""
    if rope is None:
        return Kh
    kpos = np.asarray(kpos, dtype=np.int64)
    return np.stack([rotate_heads(Kh[j], rope[kpos[j]], H) for j in range(Kh.shape[0])]) if len(kpos) else Kh


def attention_weights(q_h: np.ndarray, Kh_h: np.ndarray) -> np.ndarray:
    """Softmax over the bank of <q_h, K^_j> / sqrt(d_h) for one query/head."""
    d_h = q_h.shape[0]
    s = (Kh_h @ q_h) / math.sqrt(d_h)
    w = np.exp(s - s.max())
    return w / w.sum()


def readout(X, sel, Kraw, Vraw, Wq, Wk, Wv, Wo, H: int, rope=None, kpos=None) -> np.ndarray:
    """Row-by-row readout.  X: [mn][C]; sel: kept cell indices; Kraw/Vraw:
    [N][d_kv] bank rows in key order.  rope: optional complex table
    [mn][d_h/2] with kpos [N], the cell of each bank row.  Returns float64
    [mn][C]."""
    X = np.asarray(X, np.float64)
    Wq, Wo = np.asarray(Wq, np.float64), np.asarray(Wo, np.float64)
    Y = X.copy()
    N = np.asarray(Kraw).shape[0]
    if N == 0:
        return Y
    Kh, Vh = project_bank(Kraw, Vraw, Wk, Wv)
    Kh = rotate_keys(Kh, rope, kpos, H)
    D = Wq.shape[1]
    d_h = D // H
    for i in np.asarray(sel, dtype=np.int64):
        q = X[i] @ Wq
        if rope is not None:
            q = rotate_heads(q, rope[i], H)   # f~ = f[K_r] (Eq. 7)
        o = np.zeros(D)
        for h in range(H):
            cols = slice(h * d_h, (h + 1) * d_h)
            p = attention_weights(q[cols], Kh[:, cols])
            o[cols] = p @ Vh[:, cols]
        Y[i] = X[i] + o @ Wo
    return Y


def readout_dense(X, Kraw, Vraw, Wq, Wk, Wv, Wo, H: int, rope=None, kpos=None, qpos=None) -> np.ndarray:
    """Unpruned layer on all rows of X as whole-matrix products (no gather or
    scatter): Y = X + softmax(Q K^T / sqrt(d_h)) V W_o per head.  With a
    rotary table, row r of X is turned by rope[qpos[r]] (qpos defaults to
    0..rows-1, the cells of a whole grid)."""
    X = np.asarray(X, np.float64)
    N = np.asarray(Kraw).shape[0]
    if N == 0:
        return X.copy()
    Kh, Vh = project_bank(Kraw, Vraw, Wk, Wv)
    Kh = rotate_keys(Kh, rope, kpos, H)
    return readout_dense_projected(X, Kh, Vh, Wq, Wo, H, rope=rope, qpos=qpos)


def readout_dense_projected(X, Kh, Vh, Wq, Wo, H: int, rope=None, qpos=None) -> np.ndarray:
    """The whole-matrix layer of `readout_dense` on a bank already in the
    attention space (K^ turned by its cells when there is a table), so that
    callers can evaluate many row blocks against one projection."""
    X = np.asarray(X, np.float64)
    if Kh.shape[0] == 0:
        return X.copy()
    Q = X @ np.asarray(Wq, np.float64)
    if rope is not None:
        qpos = np.arange(X.shape[0]) if qpos is None else np.asarray(qpos, dtype=np.int64)
        Q = np.stack([rotate_heads(Q[r], rope[qpos[r]], H) for r in range(Q.shape[0])])
    D = Q.shape[1]
    d_h = D // H
    O = np.zeros_like(Q)
    for h in range(H):
        cols = slice(h * d_h, (h + 1) * d_h)
        S = Q[:, cols] @ Kh[:, cols].T / math.sqrt(d_h)
        S = S - S.max(axis=1, keepdims=True)
        P = np.exp(S)
        P = P / P.sum(axis=1, keepdims=True)
        O[:, cols] = P @ Vh[:, cols]
    return X + O @ np.asarray(Wo, np.float64)


def attend(Q, K, V, H: int) -> np.ndarray:
    """Bare Eq. 6 core on already-projected tensors: per head,
    softmax(Q_h K_h^T / sqrt(d_h)) V_h.  Q: [n_q][D], K, V: [n_kv][D]."""
    Q, K, V = (np.asarray(a, np.float64) for a in (Q, K, V))
    D = Q.shape[1]
    d_h = D // H
    O = np.zeros((Q.shape[0], D))
    if K.shape[0] == 0:
        return O
    for h in range(H):
        cols = slice(h * d_h, (h + 1) * d_h)
        for r in range(Q.shape[0]):
            O[r, cols] = attention_weights(Q[r, cols], K[:, cols]) @ V[:, cols]
    return O
