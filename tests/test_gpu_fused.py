"""rs3_readout_commit (a frame's readout and commit in one call, the split
merge and the commit sharing one launch) through the C ABI against the fp64
oracle: outputs within 2e-2 (bf16) or 1e-4 (fp32), unselected rows
bit-identical, banks bit-exact after every fused call, for one object in
both layer modes, eight objects with per-object lists and out-of-place
outputs (past 1,024 work-groups, where the merge and the commit run as two
launches), fp32 outputs, a rotary layer, the fp32 path (no merge launch), a frame
with an empty selection, and forced key-split counts from 1 to 100."""
from dataclasses import replace

import numpy as np
import pytest

import oracle
from test_gpu_parity import Runner
from workloads import CONFIGS

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


def _fused_run(cfg, n_frames, first, rows=None, y_fp32=0, tol=None, rope=None, **kw):
    r = Runner(cfg, n_frames, rope_theta=rope, **kw)
    if rope:
        r.orc.rope = oracle.axial_table(cfg.m, cfg.n, cfg.d_h, rope)
    r.commit(0, True)
    for t in range(1, n_frames):
        if t < first:
            r.commit(t, False)
        else:
            r.select_readout(t, rows_per_obj=None if t == n_frames - 1 else rows, y_fp32=y_fp32, tol=tol,
                             fused=True)
    return r


@pytest.mark.parametrize("absorb", [False, True])
def test_sam2_single_fused(absorb):
    _fused_run(CONFIGS["sam2_single"], 10, 4, rows=48, max_sel=1228, absorb=absorb)


def test_multi_obj8_fused():
    _fused_run(CONFIGS["multi_obj8"], 9, 6, rows=24, max_sel=1228, absorb=True)


def test_fused_fp32_output_and_rotary():
    cfg = CONFIGS["sam2_single"]
    _fused_run(cfg, 9, 7, rows=64, y_fp32=1, tol=4e-3, max_sel=1228)
    _fused_run(replace(cfg, m=32, n=32, f_max=4, cap_frames=4), 7, 2, rows=64, rope=10000.0)


def test_fused_fp32_layer_and_small_banks():
    # the fp32 path has no merge launch: the call runs readout then commit;
    # a small ring wraps and evicts during the fused calls
    _fused_run(CONFIGS["tiny_f32"], 8, 1)
    _fused_run(replace(CONFIGS["sam2_single"], m=16, n=16, f_max=3, cap_frames=2), 9, 1, absorb=True)


def test_fused_empty_selection():
    cfg = CONFIGS["sam2_single"]
    r = Runner(replace(cfg, m=32, n=32, f_max=4, cap_frames=4), 5, rho_override="0.0")
    r.commit(0, True)
    for t in range(1, 5):
        r.select_readout(t, fused=True)


@pytest.mark.parametrize("absorb", [True, False])
@pytest.mark.parametrize("n_splits", [1, 3, 9, 40, 100])
def test_fused_forced_splits(absorb, n_splits):
    # forced key-split counts: one split, fewer splits than a merge batch,
    # several merge batches per thread group (S > 8 NG), and more splits
    # than resident tiles (empty splits with l = 0, whose O is never written)
    cfg = replace(CONFIGS["sam2_single"], m=32, n=32, f_max=4, cap_frames=4)
    _fused_run(cfg, 6, 2, rows=64, absorb=absorb, n_splits=n_splits)


@pytest.mark.parametrize("n_obj,two", [(1, False), (2, False), (8, True)])
def test_fused_launch_shape(n_obj, two):
    # The merge and the commit share one launch while the two parts come to
    # at most 1,024 work-groups, else run as the readout's merge launch and
    # the commit launch; both shapes against the oracle, banks bit-exact.
    # At max_sel 1228 on 64x64 grids: 77 merge blocks (16 rows) and 65 commit
    # blocks per object, 1,136 at eight objects.
    import paper_2608_22526_amd as rs3
    cfg = CONFIGS["sam2_single"] if n_obj == 1 else replace(CONFIGS["multi_obj8"], n_obj=n_obj)
    rs3.profile_enable(True, 256)
    rs3.profile_reset()
    try:
        _fused_run(cfg, 9, 7, rows=24, max_sel=1228, absorb=True)
        rep = rs3.profile_report()
    finally:
        rs3.profile_enable(False)
    fused, merge, commit = rep["merge_commit"][1], rep["combine"][1], rep["commit"][1]
    calls = 2   # frames 7 and 8 in one call each; frames 0-6 by rs3_commit
    assert (fused, merge, commit) == ((0, calls, 7 + calls) if two else (calls, 0, 7))
