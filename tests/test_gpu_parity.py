"""Parity of the HIP path (through the C ABI) against the fp64 oracle.

Index lists, counts, prior bitmaps, tracker state and bank contents must be
bit-exact; selected output rows must agree within 2e-2 max-abs (bf16 inputs,
fp32 accumulation) or 1e-4 (fp32 mode); unselected rows must be bit-identical
to the input."""
import numpy as np
import pytest

from harness import OraclePipeline, TOL, compare_bank, grid_masks, max_abs, record_margin, sample_rows
from workloads import CONFIGS, Config, make_frame, make_sequence, make_weights, storage_to_f64
from dataclasses import replace

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


def _session(cfg, W, **kw):
    from paper_2608_22526_amd.session import Session
    return Session(m=cfg.m, n=cfg.n, s=cfg.s, C=cfg.C, H=cfg.H, d_kv=cfg.d_kv, dtype=cfg.dtype,
                   n_obj=cfg.n_obj, shared_x=cfg.shared_x, union_objects=cfg.union_objects, cap=cfg.cap,
                   f_max=cfg.f_max, n_pin=cfg.n_pin, weights=W, r_s=cfg.r_s, c=cfg.c, **kw)


def _dev(a):
    from paper_2608_22526_amd.session import to_device
    return to_device(a)


def _host(t):
    from paper_2608_22526_amd.session import to_host
    return to_host(t)


class Runner:
    """Runs one seeded sequence on both sides and checks every step."""

    def __init__(self, cfg: Config, n_frames: int, logit_scale=1.0, rho_override=None, **kw):
        self.cfg = cfg
        self.W = make_weights(cfg, logit_scale)
        self.seq = make_sequence(cfg, n_frames=n_frames, rho_override=rho_override)
        self.sess = _session(cfg, self.W, **kw)
        self.orc = OraclePipeline(cfg, self.W)
        self.stats = []

    def commit(self, t, pin):
        cfg = self.cfg
        fr = make_frame(cfg, t)
        masks = self.seq.masks[t]
        self.sess.commit(_dev(fr.Kmem), _dev(fr.Vmem), _dev(masks), t, pin)
        counts = self.orc.commit(fr.Kmem, fr.Vmem, masks, t, pin)
        torch.cuda.synchronize()
        assert _host(self.sess.kept_count).tolist() == counts
        for o in range(cfg.n_obj):
            compare_bank(self.sess.banks[o].export(), self.orc.banks[o])

    def select_readout(self, t, rows_per_obj=None, in_place=None, y_fp32=0, dense_check=False, tol=None,
                       fused=False, dense_oracle=False, check_bank=True, max_sel=None):
        """fused: the readout and frame t's commit run as one rs3_readout_commit
        call; the bank is then checked against the oracle's after its commit
        (check_bank).  dense_oracle: the expected rows come from the oracle's
        whole-matrix evaluation in row blocks (large banks and row counts)
        instead of its row loop."""
        cfg, sess = self.cfg, self.sess
        fr = make_frame(cfg, t)
        rmask = self.seq.read_mask(cfg, t)
        k = self.seq.k[t]
        Xd = _dev(fr.X)
        prior = torch.zeros((sess.n_groups, cfg.mn), dtype=torch.uint8, device="cuda")
        sess.select(_dev(rmask), Xd, k, prior_out=prior)
        sel, priors = self.orc.select(rmask, fr.X, k)
        torch.cuda.synchronize()
        cnt = _host(sess.sel_count)
        idx = _host(sess.sel_idx)
        for g in range(sess.n_groups):
            assert cnt[g] == len(sel[g]), (g, cnt[g], len(sel[g]))
            assert np.array_equal(idx[g, :cnt[g]], sel[g])
        assert np.array_equal(_host(prior).astype(bool), priors)
        exp_tracks = np.array([tr.as_list() for tr in self.orc.tracks], dtype=np.int32)
        assert np.array_equal(sess.track.export(), exp_tracks)
        # readout
        if in_place is None:
            in_place = cfg.n_obj == 1 and not y_fp32
        if fused:
            fk = (_dev(fr.Kmem), _dev(fr.Vmem), _dev(self.seq.masks[t]), t, False)
            run = lambda Xi, Yo, **k: sess.readout_commit(Xi, Yo, *fk, **k)
        else:
            run = sess.readout
        if in_place:
            Y = Xd.clone()
            run(Y, Y, max_sel=max_sel)
        else:
            dt = torch.float32 if (y_fp32 or cfg.dtype == "f32") else torch.bfloat16
            Y = torch.empty((cfg.n_obj, cfg.mn, cfg.C), dtype=dt, device="cuda")
            run(Xd, Y, y_fp32=y_fp32, max_sel=max_sel)
        torch.cuda.synchronize()
        Yh = _host(Y).reshape(cfg.n_obj if not in_place else 1, cfg.mn, cfg.C)
        tol = TOL[cfg.dtype] if tol is None else tol
        for o in range(cfg.n_obj):
            g = 0 if cfg.union_objects else o
            xi = 0 if fr.X.shape[0] == 1 else o
            Yo = Yh[o if not in_place else 0]
            Xo = fr.X[xi]
            s_all = sel[g]
            unsel = np.setdiff1d(np.arange(cfg.mn), s_all)
            if y_fp32:
                assert np.array_equal(Yo[unsel], storage_to_f64(Xo[unsel], cfg.dtype).astype(np.float32))
            else:
                assert np.array_equal(Yo[unsel].view(np.uint8), Xo[unsel].view(np.uint8))
            rows = s_all if rows_per_obj is None else sample_rows(s_all, rows_per_obj, 1000 * t + o)
            if len(rows) == 0:
                continue
            if dense_oracle:
                exp = self.orc.readout_dense_blocked(fr.X, o, rows)
            else:
                exp = self.orc.readout_rows(fr.X, o, rows)
            got = storage_to_f64(Yo[rows], cfg.dtype if not y_fp32 else "f32")
            err = max_abs(got, exp)
            delta = exp - storage_to_f64(Xo[rows], cfg.dtype)
            self.stats.append((t, o, len(rows), err, float(np.abs(delta).max())))
            record_margin("%s t=%d o=%d" % (cfg.name, t, o), len(rows), err, tol)
            assert err <= tol, (t, o, err)
            if dense_check:
                dense = self.orc.readout_dense_rows(fr.X, o, rows)
                err_d = max_abs(got, dense)
                record_margin("%s t=%d o=%d dense" % (cfg.name, t, o), len(rows), err_d, tol)
                assert err_d <= tol
        if fused:
            counts = self.orc.commit(fr.Kmem, fr.Vmem, self.seq.masks[t], t, False)
            assert _host(sess.kept_count).tolist() == counts
            if check_bank:
                for o in range(cfg.n_obj):
                    compare_bank(sess.banks[o].export(), self.orc.banks[o])
        self.last_Y = Yh
        return sel


@pytest.mark.parametrize("absorb", [False, True])
def test_tiny_f32_sequence(absorb):
    cfg = CONFIGS["tiny_f32"]
    r = Runner(cfg, 8, absorb=absorb)
    r.commit(0, True)
    for t in range(1, 8):
        r.select_readout(t)
        r.commit(t, False)
    print("tiny_f32 stats", r.stats)


@pytest.mark.parametrize("absorb", [False, True])
def test_sam2_single_steady_state(absorb):
    cfg = CONFIGS["sam2_single"]
    r = Runner(cfg, 11, max_sel=1228, absorb=absorb)
    r.commit(0, True)
    for t in range(1, 11):
        if t >= 7:
            r.select_readout(t, rows_per_obj=None if t == 10 else 48)
        r.commit(t, False)
    print("sam2 stats", r.stats)


@pytest.mark.parametrize("absorb", [False, True])
def test_sam2_y_fp32_delta(absorb):
    """fp32 output exposes the attention update itself (no final rounding)."""
    cfg = CONFIGS["sam2_single"]
    r = Runner(cfg, 9, max_sel=1228, absorb=absorb)
    r.commit(0, True)
    for t in range(1, 8):
        r.commit(t, False)
    r.select_readout(8, rows_per_obj=96, y_fp32=1, tol=4e-3)
    print("sam2 fp32-Y stats", r.stats)


@pytest.mark.parametrize("absorb", [False, True])
def test_multi_obj8_one_launch(absorb):
    cfg = CONFIGS["multi_obj8"]
    r = Runner(cfg, 10, max_sel=1228, absorb=absorb)
    r.commit(0, True)
    for t in range(1, 10):
        if t >= 8:
            # every selected row of every object on the last frame
            r.select_readout(t, rows_per_obj=None if t == 9 else 24, dense_oracle=t == 9)
        r.commit(t, False)
    print("multi stats", r.stats)


@pytest.mark.parametrize("absorb", [False, True])
def test_keep_all_is_dense(absorb):
    cfg = replace(CONFIGS["sam2_single"], m=32, n=32, full_prior=True, rho=1.0, rho_lo=None, rho_hi=None,
                  cap_frames=4, f_max=3)
    r = Runner(cfg, 5, max_sel=cfg.mn, absorb=absorb)
    r.commit(0, True)
    for t in range(1, 4):
        r.commit(t, False)
    sel = r.select_readout(4, rows_per_obj=64, dense_check=True)
    assert len(sel[0]) == cfg.mn


def test_empty_bank_returns_input():
    cfg = replace(CONFIGS["sam2_single"], m=16, n=16)
    r = Runner(cfg, 3, max_sel=cfg.mn)
    # no commit at all: every row passes through bit for bit
    r.select_readout(1)
    r.select_readout(2, y_fp32=1)


def test_determinism():
    cfg = CONFIGS["sam2_single"]
    outs = []
    for _ in range(2):
        r = Runner(cfg, 9, max_sel=1228)
        r.commit(0, True)
        for t in range(1, 8):
            r.sess.commit(_dev(make_frame(cfg, t).Kmem), _dev(make_frame(cfg, t).Vmem), _dev(r.seq.masks[t]), t, False)
        fr = make_frame(cfg, 8)
        Xd = _dev(fr.X)
        r.sess.select(_dev(r.seq.masks[7]), Xd, r.seq.k[8])
        Y = Xd.clone()
        r.sess.readout(Y, Y)
        torch.cuda.synchronize()
        outs.append(_host(Y))
    assert np.array_equal(outs[0], outs[1])


@pytest.mark.parametrize("C,H,d_kv,rope", [(40, 4, 16, True), (24, 8, 16, False), (256, 2, 64, False),
                                           (64, 4, 32, True)])
def test_f32_layer_shapes(C, H, d_kv, rope):
    """fp32 layers whose heads are not 16-byte multiples (widths 10 and 3),
    heads wider than the 64 lanes of a wave (128), several heads, with and
    without a rotary table: every selected row within 1e-4 of the oracle."""
    import oracle
    from workloads import make_rope_table
    cfg = replace(CONFIGS["tiny_f32"], C=C, H=H, d_h=C // H, d_kv=d_kv)
    tbl = make_rope_table(cfg, seed=3) if rope else None
    r = Runner(cfg, 6, rope_table=tbl)
    if rope:
        r.orc.rope = oracle.table_from_pairs(tbl)
    r.commit(0, True)
    for t in range(1, 6):
        r.select_readout(t)
        r.commit(t, False)
    print("f32 shapes", C, H, d_kv, rope, r.stats)
