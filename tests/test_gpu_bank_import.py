"""Bank snapshot restore (rs3_bank_import) through the C ABI.

A bank exported after a sequence of commits (ring wrap-around included) is
imported into a fresh bank of the same layer: the re-export must be identical,
the readout against the restored bank must be bit-identical to the readout
against the original (its attention tiles are recomputed from the raw rows),
and later commits must continue exactly as the oracle's ring does.  Invalid
snapshots are rejected without changing the bank."""
from dataclasses import replace

import numpy as np
import pytest

from harness import OraclePipeline, compare_bank
from workloads import CONFIGS, make_frame, make_sequence, make_weights

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


def _snap_equal(a, b):
    assert a["n_frames"] == b["n_frames"] and a["pin_end"] == b["pin_end"]
    assert a["err"] == b["err"] and a["n_keys"] == b["n_keys"]
    for key in ("frames", "K", "V", "pos"):
        assert np.array_equal(a[key], b[key]), key


@pytest.mark.parametrize("name,absorb,rope_theta", [("sam2_single", False, None), ("sam2_single", True, None),
                                                   ("tiny_f32", False, None), ("sam2_single", False, 10000.0),
                                                   ("tiny_f32", False, 100.0)])
def test_export_import_round_trip(name, absorb, rope_theta):
    """With a rotary table the restored keys are turned again from the
    snapshot's stored cells, so the readout stays bit-identical."""
    import paper_2608_22526_amd as rs3
    from paper_2608_22526_amd.session import Session, to_device, to_host

    base = CONFIGS[name]
    # a ring of one grid of rows wraps within a few commits
    cfg = replace(base, m=32, n=32, f_max=4, cap_frames=1) if base.m > 16 else base
    W = make_weights(cfg)
    seq = make_sequence(cfg, n_frames=9)
    sess = Session(m=cfg.m, n=cfg.n, s=cfg.s, C=cfg.C, H=cfg.H, d_kv=cfg.d_kv, dtype=cfg.dtype, n_obj=1,
                   shared_x=True, union_objects=True, cap=cfg.cap, f_max=cfg.f_max, n_pin=cfg.n_pin, weights=W,
                   max_sel=cfg.mn, absorb=absorb, rope_theta=rope_theta)
    orc = OraclePipeline(cfg, W)
    for t in range(7):
        fr = make_frame(cfg, t)
        sess.commit(to_device(fr.Kmem), to_device(fr.Vmem), to_device(seq.masks[t]), t, t == 0)
        orc.commit(fr.Kmem, fr.Vmem, seq.masks[t], t, t == 0)
    torch.cuda.synchronize()
    snap = sess.banks[0].export()
    compare_bank(snap, orc.banks[0])

    restored = rs3.Bank(sess.layer, cfg.cap, cfg.f_max, cfg.n_pin)
    restored.import_snapshot(snap)
    _snap_equal(restored.export(), snap)

    # readout against the original and the restored bank: bit-identical
    fr = make_frame(cfg, 7)
    X = to_device(fr.X)
    sess.select(to_device(seq.read_mask(cfg, 7)), X, seq.k[7])
    Y1 = X.clone()
    sess.readout(Y1, Y1)
    original = sess.banks[0]
    sess.banks[0] = restored
    Y2 = X.clone()
    sess.readout(Y2, Y2)
    torch.cuda.synchronize()
    assert np.array_equal(to_host(Y1), to_host(Y2))

    # the restored bank keeps committing like the oracle's ring
    sess.commit(to_device(fr.Kmem), to_device(fr.Vmem), to_device(seq.masks[7]), 7, False)
    orc.commit(fr.Kmem, fr.Vmem, seq.masks[7], 7, False)
    torch.cuda.synchronize()
    compare_bank(restored.export(), orc.banks[0])
    # pin bookkeeping follows the snapshot: unpinned frames exist, so pin is refused
    with pytest.raises(rs3.Rs3Error):
        sess.commit(to_device(fr.Kmem), to_device(fr.Vmem), to_device(seq.masks[7]), 8, True)
    sess.banks[0] = original


def test_invalid_snapshots_rejected():
    import paper_2608_22526_amd as rs3
    from paper_2608_22526_amd.session import Session, to_device

    cfg = replace(CONFIGS["sam2_single"], m=16, n=16, f_max=4, cap_frames=3)
    W = make_weights(cfg)
    seq = make_sequence(cfg, n_frames=4)
    sess = Session(m=cfg.m, n=cfg.n, s=cfg.s, C=cfg.C, H=cfg.H, d_kv=cfg.d_kv, dtype=cfg.dtype, n_obj=1,
                   shared_x=True, union_objects=True, cap=cfg.cap, f_max=cfg.f_max, n_pin=cfg.n_pin, weights=W)
    for t in range(4):
        fr = make_frame(cfg, t)
        sess.commit(to_device(fr.Kmem), to_device(fr.Vmem), to_device(seq.masks[t]), t, t == 0)
    torch.cuda.synchronize()
    snap = sess.banks[0].export()
    assert snap["n_frames"] >= 3
    target = rs3.Bank(sess.layer, cfg.cap, cfg.f_max, cfg.n_pin)
    empty = target.export()

    def bad(mutate):
        s = {k: (v.copy() if isinstance(v, np.ndarray) else v) for k, v in snap.items()}
        mutate(s)
        with pytest.raises(rs3.Rs3Error) as ei:
            target.import_snapshot(s)
        assert ei.value.status == rs3.RS3_E_INVALID
        _snap_equal(target.export(), empty)   # unchanged

    def overlap(s):
        s["frames"][2, 0] = s["frames"][1, 0]

    def keys_sum(s):
        s["hdr"][3] += 1

    def pinned_not_first(s):
        s["frames"][1, 3] = 1

    def past_capacity(s):
        s["frames"][1, 0] = cfg.cap - 1

    def too_many_frames(s):
        s["hdr"][0] = cfg.f_max + 1

    for m in (overlap, keys_sum, pinned_not_first, past_capacity, too_many_frames):
        bad(m)
