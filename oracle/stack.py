"""The L-layer memory-attention stack on the kept queries (test
infrastructure; see package doc).

Sec. 3.1 ("Sparse memory attention"): the memory module of the VOS models
consists of L layers, each with a self-attention and a cross-attention, and
the sparse readout applies at the input of every layer: each layer runs on
the gathered kept queries only, and its update is zero at every dropped
cell.  The paper defines no layer
and its trained weights are not available, so the stack here is a reading
with synthetic weights:

  * one layer is pre-norm residual, in the shape of SAM2-class memory
    attention layers:
        z <- z + SA(LN1(z))           self-attention among the kept rows
        z <- z + CA(LN2(z), bank)     the cross-attention readout of Eq. 6
        z <- z + MLP(LN3(z))          ReLU between two linear maps C -> F -> C
  * SA: H_s heads over column blocks of width C/H_s, q, k, v = a W_qs, a W_ks,
    a W_vs (C -> C), logits scaled by 1/sqrt(C/H_s), output o W_os; its keys
    and values are the kept rows themselves: the dropped rows are not
    queries, and their update is zero, so they take no part;
  * CA: the layer of module `readout` (W_q: C -> D, bank rows projected by
    W_k, W_v: d_kv -> D, H_c heads, logits scaled by 1/sqrt(D/H_c), W_o:
    D -> C), evaluated on LN2(z);
  * LN normalises each row by its mean and biased variance (eps = 1e-5) and
    applies a per-channel gain and shift;
  * the linear maps have no bias;
  * the rows are gathered once before the first layer and scattered once
    after the last: a dropped row gets a zero update at every layer (the
    residual reading U1 of `readout`), so gathering at the input of each layer
    gives the same result; the dropped rows come back bit for bit;
  * no norm follows the last layer (it would change the dropped rows).

Two evaluations: `stack` takes the rows one at a time inside each layer
(explicit loops over rows and heads), `stack_dense` whole matrices.  With
every cell kept the two must agree (the keep-all limit at the end of
Sec. 3.1).  Layer weights are dicts with the keys of LAYER_KEYS.
"""
from __future__ import annotations

import math
from typing import Dict, Sequence

import numpy as np

from .readout import attention_weights, project_bank, readout_dense_projected

LN_EPS = 1e-5
LAYER_KEYS = ("ln1_g", "ln1_b", "Wqs", "Wks", "Wvs", "Wos", "ln2_g", "ln2_b", "Wq", "Wk", "Wv", "Wo",
              "ln3_g", "ln3_b", "W1", "W2")


def layer_norm_row(z, g, b) -> np.ndarray:
    """One row: (z - mean) / sqrt(var + eps) * g + b, biased variance."""
    z = np.asarray(z, np.float64)
    mean = sum(float(v) for v in z) / z.shape[0]
    var = sum((float(v) - mean) ** 2 for v in z) / z.shape[0]
    return (z - mean) / math.sqrt(var + LN_EPS) * np.asarray(g, np.float64) + np.asarray(b, np.float64)


def layer_norm(Z, g, b) -> np.ndarray:
    """Whole-matrix form of layer_norm_row."""
    Z = np.asarray(Z, np.float64)
    mean = Z.mean(axis=1, keepdims=True)
    var = ((Z - mean) ** 2).mean(axis=1, keepdims=True)
    return (Z - mean) / np.sqrt(var + LN_EPS) * np.asarray(g, np.float64) + np.asarray(b, np.float64)


def _heads(q, K, V, H: int) -> np.ndarray:
    """One query row against key/value rows K, V [n][D], H heads of
    width D/H over column blocks: the concatenated head outputs."""
    D = q.shape[0]
    d_h = D // H
    o = np.zeros(D)
    for h in range(H):
        cols = slice(h * d_h, (h + 1) * d_h)
        o[cols] = attention_weights(q[cols], K[:, cols]) @ V[:, cols]
    return o


def _layer_rows(Z: np.ndarray, Kh, Vh, w: Dict[str, np.ndarray], H_s: int, H_c: int) -> np.ndarray:
    """One layer on the kept rows Z [n][C], row by row.  Kh, Vh: the bank in
    the layer's attention space ([N][D]; N = 0 for an empty bank)."""
    n = Z.shape[0]
    if n == 0:
        return Z.copy()
    # self-attention among the kept rows
    A = [layer_norm_row(Z[r], w["ln1_g"], w["ln1_b"]) for r in range(n)]
    Ks = np.array([a @ w["Wks"] for a in A]).reshape(n, -1)
    Vs = np.array([a @ w["Wvs"] for a in A]).reshape(n, -1)
    Z1 = np.array([Z[r] + _heads(A[r] @ w["Wqs"], Ks, Vs, H_s) @ w["Wos"] for r in range(n)]).reshape(Z.shape)
    # cross-attention readout of the bank (Eq. 6); an empty bank adds nothing
    Z2 = Z1.copy()
    if Kh.shape[0]:
        for r in range(n):
            b = layer_norm_row(Z1[r], w["ln2_g"], w["ln2_b"])
            Z2[r] = Z1[r] + _heads(b @ w["Wq"], Kh, Vh, H_c) @ w["Wo"]
    # MLP
    Z3 = Z2.copy()
    for r in range(n):
        c = layer_norm_row(Z2[r], w["ln3_g"], w["ln3_b"])
        Z3[r] = Z2[r] + np.maximum(c @ w["W1"], 0.0) @ w["W2"]
    return Z3


def _f64(w: Dict[str, np.ndarray]) -> Dict[str, np.ndarray]:
    return {k: np.asarray(w[k], np.float64) for k in LAYER_KEYS}


def stack(X, sel, Kraw, Vraw, layers: Sequence[Dict[str, np.ndarray]], H_s: int, H_c: int) -> np.ndarray:
    """Y for the grid X [mn][C]: the kept rows sel (gathered once, in the
    given order) go through the layers; every other row is X's.  Kraw, Vraw:
    the bank's raw rows [N][d_kv] in key order."""
    X = np.asarray(X, np.float64)
    sel = np.asarray(sel, dtype=np.int64)
    Z = X[sel].copy()
    for w in map(_f64, layers):
        Kh, Vh = project_bank(Kraw, Vraw, w["Wk"], w["Wv"])
        Z = _layer_rows(Z, Kh, Vh, w, H_s, H_c)
    Y = X.copy()
    Y[sel] = Z
    return Y


def stack_dense(Xrows, Kraw, Vraw, layers: Sequence[Dict[str, np.ndarray]], H_s: int, H_c: int) -> np.ndarray:
    """The layers on the rows Xrows [n][C] (all of them kept) as whole-matrix
    products; returns the n output rows."""
    Z = np.asarray(Xrows, np.float64).copy()
    n_kv = np.asarray(Kraw).shape[0]
    for w in map(_f64, layers):
        A = layer_norm(Z, w["ln1_g"], w["ln1_b"])
        Q, K, V = A @ w["Wqs"], A @ w["Wks"], A @ w["Wvs"]
        d_h = Q.shape[1] // H_s
        O = np.zeros_like(Q)
        for h in range(H_s):
            cols = slice(h * d_h, (h + 1) * d_h)
            S = Q[:, cols] @ K[:, cols].T / math.sqrt(d_h)
            P = np.exp(S - S.max(axis=1, keepdims=True))
            O[:, cols] = (P / P.sum(axis=1, keepdims=True)) @ V[:, cols]
        Z = Z + O @ w["Wos"]
        if n_kv:
            B = layer_norm(Z, w["ln2_g"], w["ln2_b"])
            Kh, Vh = project_bank(Kraw, Vraw, w["Wk"], w["Wv"])
            Z = Z + (readout_dense_projected(B, Kh, Vh, w["Wq"], w["Wo"], H_c) - B)
        Cn = layer_norm(Z, w["ln3_g"], w["ln3_b"])
        Z = Z + np.maximum(Cn @ w["W1"], 0.0) @ w["W2"]
    return Z
