"""Pins for the oracle's L-layer memory-attention stack on the kept queries
(Sec. 3.1, "Sparse memory attention": the sparse readout applies at the
input of each layer; the layer itself is the reading stated in
oracle/stack.py).

Each pin holds for a reason outside the stack code: a textbook closed form
(LayerNorm moments, softmax over one key), a reduction to the separately
pinned single-layer readout or bare attention core, the keep-all limit
against the whole-matrix evaluation, or an invariant of the gather (dropped
rows neither change nor influence, order of the gathered rows, layers
compose)."""
import math

import numpy as np
import pytest

import oracle
from oracle import stack as ostack
from workloads import make_stack_weights, storage_to_f64, STACK_MATRICES

C, D_KV, F = 16, 8, 32


def _weights(n_layers, seed=0, **zero):
    ws = make_stack_weights(C, D_KV, F, n_layers, dtype="f32", seed=seed)
    out = []
    for w in ws:
        d = {k: storage_to_f64(v, "f32") for k, v in w.items()}
        for k in zero:
            d[k] = np.zeros_like(d[k])
        out.append(d)
    return out


def _inputs(seed, mn=24, N=13):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((mn, C)), rng.standard_normal((N, D_KV)), rng.standard_normal((N, D_KV)))


def _ln(z, g, b):
    z = np.asarray(z, np.float64)
    return (z - z.mean(axis=-1, keepdims=True)) / np.sqrt(z.var(axis=-1, keepdims=True) + 1e-5) * g + b


def test_layer_norm_closed_form():
    # z = (1, 3): mean 2, biased variance 1
    y = ostack.layer_norm_row([1.0, 3.0], [1.0, 1.0], [0.0, 0.0])
    s = 1.0 / math.sqrt(1.0 + 1e-5)
    np.testing.assert_allclose(y, [-s, s], rtol=0, atol=1e-15)
    y = ostack.layer_norm_row([1.0, 3.0], [2.0, -1.0], [0.5, 0.25])
    np.testing.assert_allclose(y, [-2 * s + 0.5, -s + 0.25], rtol=0, atol=1e-15)
    rng = np.random.default_rng(1)
    Z = rng.standard_normal((7, C)) * 3 + 1
    one, zero = np.ones(C), np.zeros(C)
    A = ostack.layer_norm(Z, one, zero)
    np.testing.assert_allclose(A.mean(axis=1), 0, atol=1e-14)
    v = Z.var(axis=1)
    np.testing.assert_allclose(A.var(axis=1), v / (v + 1e-5), rtol=1e-12)
    for r in range(7):
        np.testing.assert_allclose(ostack.layer_norm_row(Z[r], one, zero), A[r], rtol=0, atol=1e-13)


@pytest.mark.parametrize("H_s,H_c,N", [(1, 1, 13), (2, 1, 13), (4, 2, 70), (2, 2, 0)])
def test_keep_all_equals_dense(H_s, H_c, N):
    X, K, V = _inputs(3, N=N)
    ws = _weights(2, seed=1)
    full = ostack.stack(X, np.arange(X.shape[0]), K, V, ws, H_s, H_c)
    dense = ostack.stack_dense(X, K, V, ws, H_s, H_c)
    np.testing.assert_allclose(full, dense, rtol=0, atol=1e-12)
    assert np.abs(full - X).max() > 0.1   # every layer does change the rows


def test_single_row_empty_bank_closed_form():
    # softmax over a single key is 1 in every head: SA(a) = a W_vs W_os
    X, K, V = _inputs(4, N=0)
    w = _weights(1, seed=2)[0]
    x = X[5]
    z1 = x + _ln(x, w["ln1_g"], w["ln1_b"]) @ w["Wvs"] @ w["Wos"]
    y = z1 + np.maximum(_ln(z1, w["ln3_g"], w["ln3_b"]) @ w["W1"], 0.0) @ w["W2"]
    for H_s in (1, 4):
        Y = ostack.stack(X, [5], K, V, [w], H_s, 1)
        np.testing.assert_allclose(Y[5], y, rtol=0, atol=1e-13)


@pytest.mark.parametrize("H_s", [1, 2, 4])
def test_self_attention_reduces_to_attention_core(H_s):
    # no bank and no MLP: z + attend(a W_qs, a W_ks, a W_vs) W_os over the
    # kept rows, with the pinned bare attention core (scale 1/sqrt(C/H_s))
    X, K, V = _inputs(5, N=0)
    w = _weights(1, seed=3, W2=True)[0]
    sel = np.array([1, 4, 6, 9, 17, 22])
    A = _ln(X[sel], w["ln1_g"], w["ln1_b"])
    want = X[sel] + oracle.attend(A @ w["Wqs"], A @ w["Wks"], A @ w["Wvs"], H_s) @ w["Wos"]
    Y = ostack.stack(X, sel, K, V, [w], H_s, 1)
    np.testing.assert_allclose(Y[sel], want, rtol=0, atol=1e-13)


@pytest.mark.parametrize("H_c", [1, 2])
def test_cross_attention_reduces_to_single_layer_readout(H_c):
    # W_os = W_2 = 0: each kept row gets the pinned readout's update of
    # LN2(x) (Eq. 6), the rows independent of each other
    X, K, V = _inputs(6, N=40)
    w = _weights(1, seed=4, Wos=True, W2=True)[0]
    sel = np.array([0, 3, 7, 8, 15, 23])
    B = _ln(X[sel], w["ln2_g"], w["ln2_b"])
    R = oracle.readout(B, np.arange(len(sel)), K, V, w["Wq"], w["Wk"], w["Wv"], w["Wo"], H_c)
    Y = ostack.stack(X, sel, K, V, [w], 2, H_c)
    np.testing.assert_allclose(Y[sel], X[sel] + (R - B), rtol=0, atol=1e-12)


def test_dropped_rows_unchanged_and_without_influence():
    X, K, V = _inputs(7, N=20)
    ws = _weights(2, seed=5)
    sel = np.array([2, 5, 6, 11, 19])
    Y = ostack.stack(X, sel, K, V, ws, 2, 1)
    drop = np.setdiff1d(np.arange(X.shape[0]), sel)
    assert np.array_equal(Y[drop].view(np.uint64), X[drop].view(np.uint64))
    X2 = X.copy()
    X2[drop] += np.random.default_rng(8).standard_normal((len(drop), C))
    Y2 = ostack.stack(X2, sel, K, V, ws, 2, 1)
    assert np.array_equal(Y2[sel].view(np.uint64), Y[sel].view(np.uint64))


def test_negative_zero_of_dropped_rows_passes_through():
    X, K, V = _inputs(9, N=5)
    X[3] = -0.0
    Y = ostack.stack(X, [0, 1], K, V, _weights(1, seed=6), 1, 1)
    assert np.all(np.signbit(Y[3]))


def test_gather_order_is_irrelevant():
    X, K, V = _inputs(10, N=30)
    ws = _weights(2, seed=7)
    sel = np.array([1, 2, 9, 12, 13, 20, 23])
    perm = np.random.default_rng(11).permutation(len(sel))
    a = ostack.stack(X, sel, K, V, ws, 2, 2)
    b = ostack.stack(X, sel[perm], K, V, ws, 2, 2)
    np.testing.assert_allclose(a, b, rtol=0, atol=1e-12)


def test_self_attention_couples_the_kept_rows_only():
    X, K, V = _inputs(12, N=30)
    sel = np.array([3, 4, 10, 16])
    X2 = X.copy()
    X2[4] += np.random.default_rng(15).standard_normal(C)   # (a constant shift would vanish in LN1)
    with_sa = _weights(1, seed=8)
    a, b = ostack.stack(X, sel, K, V, with_sa, 1, 1), ostack.stack(X2, sel, K, V, with_sa, 1, 1)
    assert np.abs(a[10] - b[10]).max() > 1e-4
    no_sa = _weights(1, seed=8, Wos=True)
    a, b = ostack.stack(X, sel, K, V, no_sa, 1, 1), ostack.stack(X2, sel, K, V, no_sa, 1, 1)
    assert np.array_equal(a[10].view(np.uint64), b[10].view(np.uint64))


def test_layers_compose():
    # gathering once equals gathering at the input of each layer
    X, K, V = _inputs(13, N=25)
    ws = _weights(3, seed=9)
    sel = np.array([0, 5, 6, 7, 14, 21])
    once = ostack.stack(X, sel, K, V, ws, 2, 1)
    Y = X
    for w in ws:
        Y = ostack.stack(Y, sel, K, V, [w], 2, 1)
    np.testing.assert_allclose(once, Y, rtol=0, atol=1e-12)


def test_empty_keep_set():
    X, K, V = _inputs(14, N=9)
    Y = ostack.stack(X, np.zeros(0, dtype=np.int64), K, V, _weights(2), 2, 1)
    assert np.array_equal(Y.view(np.uint64), X.view(np.uint64))


def test_generator_draws_every_matrix():
    ws = make_stack_weights(C, D_KV, F, 2, dtype="bf16", seed=0)
    for name in STACK_MATRICES:
        assert ws[0][name].dtype == np.uint16
        assert not np.array_equal(ws[0][name], ws[1][name])
