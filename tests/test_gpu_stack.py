"""GPU parity of the L-layer memory-attention stack on the kept queries
(rs3_stack_readout) with the oracle (oracle/stack.py), on seeded inputs of the
single-object workload's shapes: 64x64 grid, d_model 256, bank rows of 64
from store-sparse commits of a seeded sequence (bit-exact against the
oracle's ring bank), synthetic stack weights of 2048 hidden units.

The oracle side is `stack` row by row for the small keep-sets and, for the
large ones, `stack_dense` on the gathered rows (equal to `stack` by the
keep-all and gather pins of tests/test_oracle_stack.py).

Tolerance: the stack rounds to bf16 at every MFMA operand (LayerNorm outputs,
q/k/v, the softmax weights, the per-split and merged attention outputs, the
hidden units, the absorbed weight products) while the residual stream stays
fp32.  A CPU emulation of exactly these roundings on 600 kept rows, four
layers and 6000 bank keys deviates from the fp64 oracle by at most 0.009
(|y| up to 6, rms 1.25), so fp32 outputs are held to STACK_TOL = 0.03; bf16
outputs also carry their own rounding, at most 2^-8 |y|."""
import math

import numpy as np
import pytest

import oracle
from harness import OraclePipeline, compare_bank, record_margin
from oracle import stack as ostack
from workloads import (CONFIGS, k_from_rho, make_frame, make_sequence, make_stack_weights, make_weights,
                       storage_to_f64, to_storage)

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

STACK_TOL = 0.03
CFG = CONFIGS["sam2_single"]
F = 2048


def _log(*a):
    print(*a, flush=True)


def _dev(a):
    from paper_2608_22526_amd.session import to_device
    return to_device(a)


def _host(t):
    from paper_2608_22526_amd.session import to_host
    return to_host(t)


def _bank(n_frames, seed_frames=0):
    """An absorbed-layer bank after n_frames store-sparse commits of the
    seeded sequence, checked bit for bit against the oracle's ring bank;
    returns (bank, its raw key and value rows as float64)."""
    import paper_2608_22526_amd as P
    cfg = CFG
    W = make_weights(cfg)
    layer = P.Layer(cfg.C, 1, cfg.d_kv, P.RS3_BF16, W.Wq, W.Wk, W.Wv, W.Wo, absorb=True)
    bank = P.Bank(layer, cfg.cap, cfg.f_max, cfg.n_pin)
    orc = OraclePipeline(cfg, W)
    seq = make_sequence(cfg, max(n_frames, 1))
    for t in range(n_frames):
        fr = make_frame(cfg, seed_frames + t)
        m = seq.masks[t]
        P.commit([bank], (cfg.m, cfg.n, cfg.s), _dev(fr.Kmem), _dev(fr.Vmem), cfg.mn * cfg.d_kv, _dev(m), t,
                 int(t == 0), 0, cfg.mn)
        orc.commit(fr.Kmem, fr.Vmem, m, t, t == 0)
    torch.cuda.synchronize()
    compare_bank(bank.export(), orc.banks[0])
    K, V, _ = orc.banks[0].key_rows()
    bank._layer_keep = layer
    return bank, storage_to_f64(K, "bf16"), storage_to_f64(V, "bf16")


def _weights(n_layers, seed):
    ws = make_stack_weights(CFG.C, CFG.d_kv, F, n_layers, "bf16", seed=seed)
    f64 = [{k: (storage_to_f64(v, "bf16") if v.dtype == np.uint16 else v.astype(np.float64)) for k, v in w.items()}
           for w in ws]
    return ws, f64


def _grid_x(seed):
    rng = np.random.default_rng([seed, 77])
    return to_storage(rng.standard_normal((CFG.mn, CFG.C), dtype=np.float32), "bf16")


def _sel(k, seed):
    rng = np.random.default_rng([seed, 78])
    return np.sort(rng.choice(CFG.mn, k, replace=False)).astype(np.int32)


def _run(stack, bank, Xs, sel, max_sel, y_fp32=1, in_place=False, n_splits=0):
    """The stack on the GPU; returns (Y host array, bank error word)."""
    mn = CFG.mn
    Xd = _dev(Xs)
    sel_full = np.zeros(max(mn, 1), np.int32)
    sel_full[:len(sel)] = sel
    sd, cd = _dev(sel_full), _dev(np.array([len(sel)], np.int32))
    if in_place:
        Y = Xd
    elif y_fp32:
        Y = torch.empty((mn, CFG.C), dtype=torch.float32, device="cuda")
    else:
        Y = torch.empty((mn, CFG.C), dtype=torch.bfloat16, device="cuda")
    ws = torch.empty(max(stack.workspace_size(max_sel, n_splits), 16), dtype=torch.uint8, device="cuda")
    stack.readout((CFG.m, CFG.n, CFG.s), Xd, bank, sd, cd, max_sel, Y, y_fp32, ws, n_splits)
    torch.cuda.synchronize()
    return _host(Y), bank.error(clear=True)


def _check(case, Y, Xs, sel, want, y_fp32):
    X64 = storage_to_f64(Xs, "bf16")
    drop = np.setdiff1d(np.arange(CFG.mn), sel)
    if y_fp32:
        assert np.array_equal(Y[drop].astype(np.float64), X64[drop]), case
        got = Y[sel].astype(np.float64)
        bound = np.full(want.shape, STACK_TOL)
    else:
        assert np.array_equal(Y[drop], Xs[drop]), case
        got = storage_to_f64(Y[sel], "bf16")
        bound = STACK_TOL + np.abs(want) * 2.0 ** -8
    err = np.abs(got - want)
    worst = float((err / bound).max()) if err.size else 0.0
    record_margin(case, len(sel), float(err.max()) if err.size else 0.0, STACK_TOL)
    _log(case, "rows", len(sel), "max err %.4g" % (err.max() if err.size else 0.0), "worst err/bound %.3f" % worst)
    assert worst <= 1.0, (case, worst)


@pytest.fixture(scope="module")
def bank7():
    return _bank(7)


@pytest.mark.parametrize("L,H_s,rho,extra,y_fp32", [
    (4, 1, "0.25", 37, 1),     # the workload's layer count, one head of 256, ragged tail
    (4, 4, "0.15", 0, 0),      # four heads of 64, bf16 output
    (2, 8, "0.30", 100, 1),    # eight heads of 32
])
def test_stack_matches_oracle(bank7, L, H_s, rho, extra, y_fp32):
    import paper_2608_22526_amd as P
    bank, K, V = bank7
    ws, wf = _weights(L, seed=L * 10 + H_s)
    stack = P.Stack(ws, H_s=H_s, F=F)
    k = k_from_rho(rho, CFG.mn)
    Xs = _grid_x(L + H_s)
    sel = _sel(k, L + H_s)
    _log("stack L=%d H_s=%d k=%d max_sel=%d bank keys=%d" % (L, H_s, k, k + extra, K.shape[0]))
    Y, err = _run(stack, bank, Xs, sel, k + extra, y_fp32)
    assert err == 0
    want = ostack.stack_dense(storage_to_f64(Xs, "bf16")[sel], K, V, wf, H_s, 1)
    _check("L%d_Hs%d_k%d" % (L, H_s, k), Y, Xs, sel, want, y_fp32)


def test_stack_row_by_row_oracle_small(bank7):
    """A keep-set small enough for the row-by-row definition itself."""
    import paper_2608_22526_amd as P
    bank, K, V = bank7
    ws, wf = _weights(2, seed=5)
    stack = P.Stack(ws, H_s=2, F=F)
    Xs = _grid_x(5)
    sel = _sel(150, 5)
    Y, err = _run(stack, bank, Xs, sel, 150, 1)
    assert err == 0
    want = ostack.stack(storage_to_f64(Xs, "bf16"), sel, K, V, wf, 2, 1)[sel]
    _check("rowwise_k150", Y, Xs, sel, want, 1)


def test_stack_keep_all_equals_dense(bank7):
    """Every cell kept: the whole grid through the whole-matrix layers (the
    keep-all limit at the end of Sec. 3.1)."""
    import paper_2608_22526_amd as P
    bank, K, V = bank7
    ws, wf = _weights(2, seed=6)
    stack = P.Stack(ws, H_s=1, F=F)
    Xs = _grid_x(6)
    sel = np.arange(CFG.mn, dtype=np.int32)
    Y, err = _run(stack, bank, Xs, sel, CFG.mn, 1)
    assert err == 0
    want = ostack.stack_dense(storage_to_f64(Xs, "bf16"), K, V, wf, 1, 1)
    _check("keep_all", Y, Xs, sel, want, 1)


@pytest.mark.parametrize("k", [1, 64, 65])
def test_stack_tile_edges(bank7, k):
    """One row, exactly one 64-row tile, one row past it."""
    import paper_2608_22526_amd as P
    bank, K, V = bank7
    ws, wf = _weights(1, seed=7)
    stack = P.Stack(ws, H_s=4, F=F)
    Xs = _grid_x(7)
    sel = _sel(k, 7 + k)
    Y, err = _run(stack, bank, Xs, sel, k, 1)
    assert err == 0
    want = ostack.stack(storage_to_f64(Xs, "bf16"), sel, K, V, wf, 4, 1)[sel]
    _check("edge_k%d" % k, Y, Xs, sel, want, 1)


def test_stack_empty_bank_and_empty_keep_set():
    import paper_2608_22526_amd as P
    bank, K, V = _bank(0)
    assert K.shape[0] == 0
    ws, wf = _weights(2, seed=8)
    stack = P.Stack(ws, H_s=1, F=F)
    Xs = _grid_x(8)
    sel = _sel(300, 8)
    Y, err = _run(stack, bank, Xs, sel, 400, 1)
    assert err == 0
    want = ostack.stack(storage_to_f64(Xs, "bf16"), sel, K, V, wf, 1, 1)[sel]
    _check("empty_bank", Y, Xs, sel, want, 1)
    # no kept row: Y is X everywhere (bf16 out of place and fp32)
    for y32 in (0, 1):
        Y, err = _run(stack, bank, Xs, sel[:0], 400, y32)
        assert err == 0
        if y32:
            assert np.array_equal(Y.astype(np.float64), storage_to_f64(Xs, "bf16"))
        else:
            assert np.array_equal(Y, Xs)


def test_stack_in_place_and_workspace_reuse(bank7):
    """Y = X (bf16), and a second call with fewer kept rows on the same
    workspace sizes."""
    import paper_2608_22526_amd as P
    bank, K, V = bank7
    ws, wf = _weights(2, seed=9)
    stack = P.Stack(ws, H_s=2, F=F)
    Xs = _grid_x(9)
    X64 = storage_to_f64(Xs, "bf16")
    for k in (700, 129):
        sel = _sel(k, 9 + k)
        Y, err = _run(stack, bank, Xs, sel, 700, 0, in_place=True)
        assert err == 0
        want = ostack.stack_dense(X64[sel], K, V, wf, 2, 1)
        _check("in_place_k%d" % k, Y, Xs, sel, want, 0)


def test_stack_bank_is_read_only(bank7):
    import paper_2608_22526_amd as P
    bank, K, V = bank7
    before = bank.export()
    ws, _ = _weights(1, seed=10)
    stack = P.Stack(ws, H_s=1, F=F)
    Xs = _grid_x(10)
    _run(stack, bank, Xs, _sel(500, 10), 500, 1)
    after = bank.export()
    for key in ("hdr", "frames", "K", "V", "pos"):
        assert np.array_equal(before[key], after[key]), key


def test_stack_reports_invalid_lists(bank7):
    """Entries out of order and a count past max_sel set the bank's error
    word; the dropped rows still come back as X."""
    import paper_2608_22526_amd as P
    bank, K, V = bank7
    ws, _ = _weights(1, seed=11)
    stack = P.Stack(ws, H_s=1, F=F)
    Xs = _grid_x(11)
    sel = _sel(200, 11)
    bad = sel.copy()
    bad[[50, 51]] = bad[[51, 50]]
    Y, err = _run(stack, bank, Xs, bad, 200, 0)
    assert err == P.RS3_E_INVALID
    drop = np.setdiff1d(np.arange(CFG.mn), sel)
    assert np.array_equal(Y[drop], Xs[drop])
    # count past max_sel
    mn = CFG.mn
    sel_full = np.zeros(mn, np.int32)
    sel_full[:200] = sel
    Xd = _dev(Xs)
    Yd = torch.empty((mn, CFG.C), dtype=torch.bfloat16, device="cuda")
    w = torch.empty(stack.workspace_size(100), dtype=torch.uint8, device="cuda")
    stack.readout((CFG.m, CFG.n, CFG.s), Xd, bank, _dev(sel_full), _dev(np.array([200], np.int32)), 100, Yd, 0, w)
    torch.cuda.synchronize()
    assert bank.error(clear=True) == P.RS3_E_INVALID
