"""Pins for the oracle's rotary positions on the gathered subset (Sec. 3.1,
"RoPE on the sparse subset", Eq. 7, and the keep-all statement after it).

The table construction is a reading (only its shape is given); these tests pin
the stated form by special cases and invariants, and pin the gather of Eq. 7
through keep-all = dense and row independence, which the paper states and
which the prefix slice it warns about breaks."""
import cmath
import math

import numpy as np
import pytest

import oracle


def test_axial_width4_is_pure_column_and_row_phase():
    # with d_h = 4 every frequency is theta^0 = 1, whatever theta is
    m, n = 3, 5
    for theta in (10.0, 10000.0):
        f = oracle.axial_table(m, n, 4, theta)
        for r in range(m):
            for c in range(n):
                assert f[r * n + c, 0] == pytest.approx(cmath.exp(1j * c), abs=1e-15)
                assert f[r * n + c, 1] == pytest.approx(cmath.exp(1j * r), abs=1e-15)


def test_axial_frequency_ladder():
    # d_h = 8, theta = 100: the second frequency is 100^(-1/2) = 0.1, so ten
    # columns (rows) turn it by exactly one radian
    f = oracle.axial_table(11, 11, 8, 100.0)
    assert f[0 * 11 + 10, 1] == pytest.approx(cmath.exp(1j), abs=1e-14)
    assert f[10 * 11 + 0, 3] == pytest.approx(cmath.exp(1j), abs=1e-14)
    # d_h = 16, theta = 10^4: third frequency 10^-2
    g = oracle.axial_table(1, 51, 16, 1e4)
    assert g[50, 2] == pytest.approx(cmath.exp(0.5j), abs=1e-14)


def test_axial_unit_modulus_origin_and_separability():
    m, n, d_h = 6, 7, 32
    f = oracle.axial_table(m, n, d_h, 10000.0)
    np.testing.assert_allclose(np.abs(f), 1.0, rtol=0, atol=1e-14)
    np.testing.assert_allclose(f[0], 1.0, rtol=0, atol=0)
    q = d_h // 4
    F = f.reshape(m, n, d_h // 2)
    # the first quarter depends on the column only, the second on the row only
    assert np.array_equal(F[:, :, :q], np.broadcast_to(F[:1, :, :q], F[:, :, :q].shape))
    assert np.array_equal(F[:, :, q:], np.broadcast_to(F[:, :1, q:], F[:, :, q:].shape))


def test_rotation_closed_forms():
    rng = np.random.default_rng(0)
    v = rng.standard_normal(8)
    # a quarter turn maps (a, b) to (-b, a)
    out = oracle.rotate(v, np.full(4, 1j))
    np.testing.assert_allclose(out[0::2], -v[1::2], atol=1e-15)
    np.testing.assert_allclose(out[1::2], v[0::2], atol=1e-15)
    # the identity factor changes nothing
    assert np.array_equal(oracle.rotate(v, np.ones(4)), v)
    # rotations preserve the norm and compose by multiplying the factors
    a = np.exp(1j * rng.uniform(0, 2 * np.pi, 4))
    b = np.exp(1j * rng.uniform(0, 2 * np.pi, 4))
    assert np.linalg.norm(oracle.rotate(v, a)) == pytest.approx(np.linalg.norm(v), rel=1e-14)
    np.testing.assert_allclose(oracle.rotate(oracle.rotate(v, a), b), oracle.rotate(v, a * b), atol=1e-14)
    np.testing.assert_allclose(oracle.rotate(oracle.rotate(v, a), np.conj(a)), v, atol=1e-14)


def test_scores_depend_on_displacement_only():
    # <R_a q, R_b k> under the axial table is unchanged when both cells move
    # by the same grid displacement
    m, n, d_h = 9, 10, 16
    f = oracle.axial_table(m, n, d_h, 10000.0)
    rng = np.random.default_rng(1)
    q, k = rng.standard_normal(d_h), rng.standard_normal(d_h)
    cell = lambda r, c: r * n + c
    base = oracle.rotate(q, f[cell(2, 3)]) @ oracle.rotate(k, f[cell(4, 1)])
    for dr, dc in ((1, 0), (0, 4), (3, 2), (4, 5)):
        moved = oracle.rotate(q, f[cell(2 + dr, 3 + dc)]) @ oracle.rotate(k, f[cell(4 + dr, 1 + dc)])
        assert moved == pytest.approx(base, rel=1e-12, abs=1e-12)
    # and changes when only one of them moves
    other = oracle.rotate(q, f[cell(2, 4)]) @ oracle.rotate(k, f[cell(4, 1)])
    assert abs(other - base) > 1e-6


def _layer(rng, C, H, d_kv, N, mn):
    D = C
    W = dict(Wq=rng.standard_normal((C, D)) / math.sqrt(C), Wk=rng.standard_normal((d_kv, D)) / math.sqrt(d_kv),
             Wv=rng.standard_normal((d_kv, D)) / math.sqrt(d_kv), Wo=rng.standard_normal((D, C)) / math.sqrt(D))
    return rng.standard_normal((mn, C)), rng.standard_normal((N, d_kv)), rng.standard_normal((N, d_kv)), W


@pytest.mark.parametrize("H,d_h", [(1, 16), (2, 8)])
def test_keep_all_equals_dense_and_rows_are_independent(H, d_h):
    rng = np.random.default_rng(3)
    m, n = 5, 6
    mn, C, d_kv, N = m * n, H * d_h, 6, 19
    X, K, V, W = _layer(rng, C, H, d_kv, N, mn)
    f = oracle.axial_table(m, n, d_h, 10000.0)
    kpos = rng.integers(0, mn, N)
    dense = oracle.readout_dense(X, K, V, **W, H=H, rope=f, kpos=kpos)
    full = oracle.readout(X, np.arange(mn), K, V, **W, H=H, rope=f, kpos=kpos)
    np.testing.assert_allclose(full, dense, rtol=0, atol=1e-12)
    sel = np.sort(rng.choice(mn, 9, replace=False))
    part = oracle.readout(X, sel, K, V, **W, H=H, rope=f, kpos=kpos)
    np.testing.assert_allclose(part[sel], dense[sel], rtol=0, atol=1e-12)
    unsel = np.setdiff1d(np.arange(mn), sel)
    assert np.array_equal(part[unsel].view(np.uint64), X[unsel].view(np.uint64))
    # the dense layer on a subset of rows, told their cells, gives the same rows
    sub = oracle.readout_dense(X[sel], K, V, **W, H=H, rope=f, kpos=kpos, qpos=sel)
    np.testing.assert_allclose(sub, dense[sel], rtol=0, atol=1e-12)
    # the rotation matters: without it the rows differ
    plain = oracle.readout(X, sel, K, V, **W, H=H)
    assert np.max(np.abs(plain[sel] - dense[sel])) > 1e-3


def test_prefix_slice_breaks_row_independence():
    # the mistake Eq. 7 corrects: the r-th gathered query paired with f[r]
    # instead of f[sel[r]].  Feeding the oracle a table whose row sel[r] holds
    # f[r] reproduces it; it must disagree with the dense rows.
    rng = np.random.default_rng(4)
    m, n, H, d_h = 6, 6, 1, 16
    mn, d_kv, N = m * n, 8, 15
    X, K, V, W = _layer(rng, d_h, H, d_kv, N, mn)
    f = oracle.axial_table(m, n, d_h, 10000.0)
    kpos = rng.integers(0, mn, N)
    sel = np.array([3, 7, 8, 20, 31])
    dense = oracle.readout_dense(X, K, V, **W, H=H, rope=f, kpos=kpos)
    prefix = f.copy()
    prefix[sel] = f[:len(sel)]
    wrong = oracle.readout(X, sel, K, V, **W, H=H, rope=prefix, kpos=kpos)
    right = oracle.readout(X, sel, K, V, **W, H=H, rope=f, kpos=kpos)
    np.testing.assert_allclose(right[sel], dense[sel], rtol=0, atol=1e-12)
    assert np.max(np.abs(wrong[sel] - dense[sel])) > 1e-3


def test_identity_table_and_same_cell_keys_reduce_to_plain_readout():
    rng = np.random.default_rng(5)
    m, n, H, d_h = 4, 4, 2, 8
    mn, C, d_kv, N = m * n, H * d_h, 8, 11
    X, K, V, W = _layer(rng, C, H, d_kv, N, mn)
    kpos = rng.integers(0, mn, N)
    sel = np.array([0, 5, 9, 15])
    plain = oracle.readout(X, sel, K, V, **W, H=H)
    ones = oracle.readout(X, sel, K, V, **W, H=H, rope=np.ones((mn, d_h // 2), np.complex128), kpos=kpos)
    np.testing.assert_allclose(ones, plain, rtol=0, atol=1e-13)
    # every key kept from the query's own cell: the common rotation cancels
    # in each logit, so that row equals the plain readout
    f = oracle.axial_table(m, n, d_h, 100.0)
    same = oracle.readout(X, [9], K, V, **W, H=H, rope=f, kpos=np.full(N, 9))
    np.testing.assert_allclose(same[9], plain[9], rtol=0, atol=1e-12)
    moved = oracle.readout(X, [9], K, V, **W, H=H, rope=f, kpos=np.full(N, 10))
    assert np.max(np.abs(moved[9] - plain[9])) > 1e-4


def test_table_from_pairs():
    pairs = np.array([[[1.0, 0.0], [0.0, 1.0]], [[-1.0, 0.0], [0.6, 0.8]]])
    np.testing.assert_array_equal(oracle.table_from_pairs(pairs), np.array([[1, 1j], [-1, 0.6 + 0.8j]]))
