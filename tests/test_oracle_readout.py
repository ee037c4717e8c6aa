"""Pins for the oracle's sparse readout (Sec. 3.1, Eq. 6 and the keep-all
limit stated at the end of Sec. 3.1)."""
import json
import math
import os

import numpy as np
import pytest

import oracle


def _rand_layer(rng, C, H, d_h, d_kv, N, mn):
    D = H * d_h
    W = dict(Wq=rng.standard_normal((C, D)) / math.sqrt(C),
             Wk=rng.standard_normal((d_kv, D)) / math.sqrt(d_kv),
             Wv=rng.standard_normal((d_kv, D)) / math.sqrt(d_kv),
             Wo=rng.standard_normal((D, C)) / math.sqrt(D))
    X = rng.standard_normal((mn, C))
    K = rng.standard_normal((N, d_kv))
    V = rng.standard_normal((N, d_kv))
    return X, K, V, W


def test_closed_forms(golden_dir):
    g = json.load(open(os.path.join(golden_dir, "readout_closed_forms.json")))
    W = {k: np.array(v, dtype=np.float64) for k, v in g["weights"].items()}
    x = np.array([g["x"]], dtype=np.float64)
    V = np.array(g["bank_V"], dtype=np.float64)
    for case in g["cases"]:
        K = np.array(case["bank_K"] + [[0, 0]], dtype=np.float64)
        Y = oracle.readout(x, [0], K, V, W["Wq"], W["Wk"], W["Wv"], W["Wo"], case["H"])
        np.testing.assert_allclose(Y[0], case["expected_y"], rtol=0, atol=1e-12)
        Yd = oracle.readout_dense(x, K, V, W["Wq"], W["Wk"], W["Wv"], W["Wo"], case["H"])
        np.testing.assert_allclose(Yd[0], case["expected_y"], rtol=0, atol=1e-12)


@pytest.mark.parametrize("H,d_h", [(1, 16), (4, 8)])
def test_keep_all_equals_dense_and_row_independence(H, d_h):
    rng = np.random.default_rng(5)
    mn, C, d_kv, N = 30, H * d_h, 6, 23
    X, K, V, W = _rand_layer(rng, C, H, d_h, d_kv, N, mn)
    dense = oracle.readout_dense(X, K, V, **W, H=H)
    full = oracle.readout(X, np.arange(mn), K, V, **W, H=H)
    np.testing.assert_allclose(full, dense, rtol=0, atol=1e-12)
    sel = np.sort(rng.choice(mn, 11, replace=False))
    part = oracle.readout(X, sel, K, V, **W, H=H)
    np.testing.assert_allclose(part[sel], dense[sel], rtol=0, atol=1e-12)
    unsel = np.setdiff1d(np.arange(mn), sel)
    assert np.array_equal(part[unsel].view(np.uint64), X[unsel].view(np.uint64))


def test_negative_zero_passes_through():
    rng = np.random.default_rng(2)
    X, K, V, W = _rand_layer(rng, 8, 1, 8, 4, 5, 6)
    X[3] = -0.0
    Y = oracle.readout(X, [0, 1], K, V, **W, H=1)
    assert np.all(np.signbit(Y[3]))


def test_softmax_sums_to_one():
    rng = np.random.default_rng(3)
    for _ in range(5):
        q = rng.standard_normal(32) * 3
        Kh = rng.standard_normal((100, 32))
        p = oracle.attention_weights(q, Kh)
        assert abs(p.sum() - 1.0) < 1e-12
        assert np.all(p >= 0)


def test_single_key_and_identical_keys():
    rng = np.random.default_rng(4)
    X, K, V, W = _rand_layer(rng, 16, 2, 8, 5, 7, 9)
    Y1 = oracle.readout(X, [2, 5], K[:1], V[:1], **W, H=2)
    vh = V[:1] @ W["Wv"]
    np.testing.assert_allclose(Y1[[2, 5]], X[[2, 5]] + vh @ W["Wo"], atol=1e-12)
    Ksame = np.repeat(K[:1], 7, axis=0)
    Ys = oracle.readout(X, [1], Ksame, V, **W, H=2)
    np.testing.assert_allclose(Ys[1], X[1] + (V @ W["Wv"]).mean(axis=0) @ W["Wo"], atol=1e-12)


def test_bank_permutation_invariance_and_empty_bank():
    rng = np.random.default_rng(6)
    X, K, V, W = _rand_layer(rng, 12, 3, 4, 5, 19, 10)
    perm = rng.permutation(19)
    a = oracle.readout(X, [0, 4, 9], K, V, **W, H=3)
    b = oracle.readout(X, [0, 4, 9], K[perm], V[perm], **W, H=3)
    np.testing.assert_allclose(a, b, atol=1e-12)
    e = oracle.readout(X, [0, 4, 9], K[:0], V[:0], **W, H=3)
    assert np.array_equal(e, X)


def test_explicit_loops_2x2_grid():
    """Brute force with scalar loops on a 2x2 grid and a 3-token bank."""
    rng = np.random.default_rng(8)
    C, H, d_h, d_kv = 4, 2, 2, 3
    X, K, V, W = _rand_layer(rng, C, H, d_h, d_kv, 3, 4)
    sel = [1, 3]
    Y = oracle.readout(X, sel, K, V, **W, H=H)
    D = H * d_h
    for i in range(4):
        if i not in sel:
            assert np.array_equal(Y[i], X[i])
            continue
        q = [sum(X[i][c] * W["Wq"][c][d] for c in range(C)) for d in range(D)]
        kh = [[sum(K[j][a] * W["Wk"][a][d] for a in range(d_kv)) for d in range(D)] for j in range(3)]
        vh = [[sum(V[j][a] * W["Wv"][a][d] for a in range(d_kv)) for d in range(D)] for j in range(3)]
        o = [0.0] * D
        for h in range(H):
            logits = [sum(q[h * d_h + t] * kh[j][h * d_h + t] for t in range(d_h)) / math.sqrt(d_h)
                      for j in range(3)]
            den = sum(math.exp(s) for s in logits)
            for t in range(d_h):
                o[h * d_h + t] = sum(math.exp(logits[j]) / den * vh[j][h * d_h + t] for j in range(3))
        y = [X[i][c] + sum(o[d] * W["Wo"][d][c] for d in range(D)) for c in range(C)]
        np.testing.assert_allclose(Y[i], y, atol=1e-12)


def test_attend_core():
    rng = np.random.default_rng(9)
    Q = rng.standard_normal((5, 8))
    K = rng.standard_normal((11, 8))
    V = rng.standard_normal((11, 8))
    O = oracle.attend(Q, K, V, H=2)
    Ksame = np.repeat(K[:1], 11, axis=0)
    np.testing.assert_allclose(oracle.attend(Q, Ksame, V, H=2), np.tile(V.mean(axis=0), (5, 1)), atol=1e-12)
    # equals the readout with identity projections and zero residual weights
    I = np.eye(8)
    Y = oracle.readout(Q, np.arange(5), K, V, I, I, I, I, H=2)
    np.testing.assert_allclose(Y - Q, O, atol=1e-12)
