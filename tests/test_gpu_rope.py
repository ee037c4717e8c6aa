"""Parity of the rotary readout (Sec. 3.1, "RoPE on the sparse subset", Eq. 7)
through the C ABI against the fp64 oracle.

Each selected query is turned by the table row of the cell it was gathered
from and each bank key by the row of the cell it was kept from.  Every checked
row is also compared with the oracle's dense layer told the row's cell, which
holds only with the gather (row independence); index lists and banks stay
bit-exact, outputs within 2e-2 (bf16) or 1e-4 (fp32).  The axial table is
built by the library on the device and by the oracle in fp64; the random
table is one seeded input handed to both."""
from dataclasses import replace

import numpy as np
import pytest

import oracle
from test_gpu_parity import Runner
from workloads import CONFIGS, make_frame, make_rope_table, make_sequence, make_weights

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


def _run(cfg, n_frames, first_read, rope_theta=None, rope_table=None, rows=None, y_fp32=0, tol=None, **kw):
    r = Runner(cfg, n_frames, rope_theta=rope_theta, rope_table=rope_table, **kw)
    if rope_table is not None:
        r.orc.rope = oracle.table_from_pairs(rope_table)
    else:
        r.orc.rope = oracle.axial_table(cfg.m, cfg.n, cfg.d_h, rope_theta)
    r.commit(0, True)
    for t in range(1, n_frames):
        if t >= first_read:
            r.select_readout(t, rows_per_obj=None if t == n_frames - 1 else rows, dense_check=True, y_fp32=y_fp32,
                             tol=tol)
        r.commit(t, False)
    return r


@pytest.mark.parametrize("d_kv", [32, 96])
def test_tiny_f32_axial(d_kv):
    # d_kv 96 takes the unstaged fp32 projection of the commit
    cfg = replace(CONFIGS["tiny_f32"], d_kv=d_kv)
    r = _run(cfg, 8, 1, rope_theta=100.0)
    print("tiny_f32 rope stats", r.stats)


def test_sam2_single_axial():
    cfg = CONFIGS["sam2_single"]
    r = _run(cfg, 10, 7, rope_theta=10000.0, rows=48, max_sel=1228)
    print("sam2 rope stats", r.stats)


@pytest.mark.parametrize("cfg_name", ["sam2_single", "heads32"])
def test_rotary_fp32_delta(cfg_name):
    # fp32 output keeps the attention update unrounded: 4e-3 is well below
    # the 0.09 by which these rows move when the rotation is dropped, turned
    # the wrong way or taken from the prefix rows
    cfg = CONFIGS["sam2_single"] if cfg_name == "sam2_single" else \
        replace(CONFIGS["highres"], m=48, n=48, f_max=6, cap_frames=7)
    r = _run(cfg, 8, 7, rope_theta=10000.0, rows=96, y_fp32=1, tol=4e-3)
    print("rope fp32-Y stats", r.stats)


def test_heads_of_32_axial():
    # eight heads of width 32 (the high-resolution layer) on a 48x48 grid
    cfg = replace(CONFIGS["highres"], m=48, n=48, f_max=6, cap_frames=7)
    r = _run(cfg, 8, 5, rope_theta=10000.0, rows=64)
    print("heads32 rope stats", r.stats)


def test_keep_all_with_rotary_equals_dense():
    # prior = whole grid and rho = 1: every cell is gathered (the identity)
    cfg = replace(CONFIGS["highres"], m=24, n=24, f_max=4, cap_frames=5)
    r = _run(cfg, 5, 3, rope_theta=10000.0, rho_override=1.0)
    assert all(n == cfg.mn for (_, _, n, _, _) in r.stats)


def test_random_table_many_objects():
    # an arbitrary table (not axial), eight objects with their own keep-sets
    cfg = replace(CONFIGS["multi_obj8"], m=32, n=32, cap_frames=8)
    r = _run(cfg, 8, 6, rope_table=make_rope_table(cfg), rows=40)
    print("multi rope stats", r.stats)


def test_rotary_argument_errors():
    import paper_2608_22526_amd as rs3
    from paper_2608_22526_amd.session import Session, to_device

    cfg = replace(CONFIGS["sam2_single"], m=16, n=16, f_max=3, cap_frames=3)
    W = make_weights(cfg)
    # absorbed layers run on the raw rows and cannot take a table
    L = rs3.Layer(cfg.C, cfg.H, cfg.d_kv, rs3.RS3_BF16, W.Wq, W.Wk, W.Wv, W.Wo, absorb=True)
    with pytest.raises(rs3.Rs3Error) as ei:
        L.set_rope_axial(cfg.m, cfg.n, 10000.0)
    assert ei.value.status == rs3.RS3_E_INVALID
    P = rs3.Layer(cfg.C, cfg.H, cfg.d_kv, rs3.RS3_BF16, W.Wq, W.Wk, W.Wv, W.Wo)
    for bad in ((0, 16, 10000.0), (16, 16, 1.0), (300, 300, 10000.0)):
        with pytest.raises(rs3.Rs3Error):
            P.set_rope_axial(*bad)
    with pytest.raises(rs3.Rs3Error):
        P.set_rope(16, 16, None)   # no table with a nonzero grid
    P.set_rope(cfg.m, cfg.n, make_rope_table(cfg))
    P.set_rope(0, 0, None)          # removed
    P.set_rope_axial(cfg.m, cfg.n, 10000.0)
    # with a bank alive the table cannot change
    bank = rs3.Bank(P, cfg.cap, cfg.f_max, cfg.n_pin)
    with pytest.raises(rs3.Rs3Error):
        P.set_rope_axial(cfg.m, cfg.n, 500.0)
    with pytest.raises(rs3.Rs3Error):
        P.set_rope(0, 0, None)
    del bank
    P.set_rope_axial(cfg.m, cfg.n, 500.0)   # allowed again once it is gone
    # a grid other than the table's is refused by readout and commit
    sess = Session(m=cfg.m, n=cfg.n, s=cfg.s, C=cfg.C, H=cfg.H, d_kv=cfg.d_kv, dtype=cfg.dtype, n_obj=1,
                   shared_x=True, union_objects=True, cap=cfg.cap, f_max=cfg.f_max, n_pin=cfg.n_pin, weights=W,
                   rope_theta=10000.0)
    other = rs3.Grid(cfg.m, cfg.n * 2, 1)
    seq = make_sequence(cfg, n_frames=1)
    fr = make_frame(cfg, 0)
    with pytest.raises(rs3.Rs3Error) as ei:
        rs3.commit(sess.banks, other, to_device(fr.Kmem), to_device(fr.Vmem), cfg.mn * cfg.d_kv,
                   to_device(np.zeros((1, cfg.m, 2 * cfg.n), np.uint8)), 0, 1, 0, 2 * cfg.mn, None, None)
    assert ei.value.status == rs3.RS3_E_INVALID
    sess.commit(to_device(fr.Kmem), to_device(fr.Vmem), to_device(seq.masks[0]), 0, True)
    torch.cuda.synchronize()
    assert sess.banks[0].error() == 0
