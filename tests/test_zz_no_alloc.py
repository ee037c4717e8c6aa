"""rs3_readout_noalloc (the readout for callers that cannot allocate) through
the C ABI against rs3_readout on the same inputs: two calls in a row, the
second with a smaller selection and a smaller max_sel, in both layer forms.
With the same key-split count the two entry points run the same kernels on
the same data, so their outputs must match bit for bit; where the automatic
count had to shrink to fit the fixed scratch, both must stay within the bf16
tolerance of the fp64 oracle.  A layout that cannot fit is refused before
any launch."""
from dataclasses import replace

import numpy as np
import pytest

from harness import TOL, max_abs, record_margin
from test_gpu_parity import Runner, _dev, _host
from workloads import CONFIGS, k_from_rho, make_frame, storage_to_f64

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


def _both(r, t, k, max_sel, n_splits=0):
    """select frame t with budget k, then rs3_readout and rs3_readout_noalloc
    on copies of X; returns (selected list, Y of readout, Y of noalloc)."""
    import paper_2608_22526_amd as rs3
    cfg, sess = r.cfg, r.sess
    fr = make_frame(cfg, t)
    Xd = _dev(fr.X)
    sess.select(_dev(r.seq.read_mask(cfg, t)), Xd, [k])
    torch.cuda.synchronize()
    cnt = int(_host(sess.sel_count)[0])
    sel = _host(sess.sel_idx)[0, :cnt].copy()
    Y1, Y2 = Xd.clone(), Xd.clone()
    rs3.readout(sess.layer, sess.grid, 1, Y1, 0, sess.banks, sess.sel_idx, sess.sel_count, 0, max_sel, n_splits,
                Y1, 0, 0, sess.ws_read)
    rs3.readout_noalloc(sess.layer, sess.grid, 1, Y2, 0, sess.banks, sess.sel_idx, sess.sel_count, 0, max_sel,
                        n_splits, Y2, 0, 0)
    torch.cuda.synchronize()
    return fr, sel, _host(Y1)[0], _host(Y2)[0]


def _prefill(cfg, absorb, n):
    r = Runner(cfg, n, max_sel=cfg.mn, absorb=absorb)
    r.commit(0, True)
    for t in range(1, cfg.f_max):
        r.commit(t, False)
    return r


@pytest.mark.parametrize("absorb", [True, False])
def test_noalloc_matches_readout_two_calls(absorb):
    cfg = CONFIGS["sam2_single"]
    r = _prefill(cfg, absorb, cfg.f_max + 2)
    t = cfg.f_max
    # first call: the benchmark's budget; second: a smaller selection and a
    # smaller max_sel (fewer query tiles)
    for k, max_sel in ((k_from_rho("0.3", cfg.mn), k_from_rho("0.3", cfg.mn)), (300, 512)):
        fr, sel, Y1, Y2 = _both(r, t, k, max_sel)
        assert len(sel) == min(k, len(sel)) and len(sel) > 0
        assert np.array_equal(Y1.view(np.uint16), Y2.view(np.uint16)), (k, max_sel)
        unsel = np.setdiff1d(np.arange(cfg.mn), sel)
        assert np.array_equal(Y2[unsel], fr.X[0][unsel])
        exp = r.orc.readout_dense_blocked(fr.X, 0, sel)
        err = max_abs(storage_to_f64(Y2[sel], cfg.dtype), exp)
        record_margin("noalloc absorb=%d k=%d" % (absorb, k), len(sel), err, TOL["bf16"])
        assert err <= TOL["bf16"]
        t += 1


def test_noalloc_fits_splits_and_refuses_oversize():
    """At 128x128 with eight heads of 32 the automatic split count of the
    workspace form needs more than the fixed scratch at rho = 0.1: the
    allocation-free form runs fewer splits (same results within the
    tolerance); a forced count that cannot fit is refused."""
    import paper_2608_22526_amd as rs3
    cfg = replace(CONFIGS["highres"], f_max=4, cap_frames=17)
    r = _prefill(cfg, False, cfg.f_max + 2)
    k = k_from_rho("0.1", cfg.mn)
    need = rs3.readout_workspace_size(r.sess.layer, 1, k, 0)
    assert need > rs3.RS3_NOALLOC_SCRATCH_BYTES   # the automatic count does not fit as it is
    for t, (kk, ms) in ((cfg.f_max, (k, k)), (cfg.f_max + 1, (400, 512))):
        fr, sel, Y1, Y2 = _both(r, t, kk, ms)
        unsel = np.setdiff1d(np.arange(cfg.mn), sel)
        assert np.array_equal(Y2[unsel], fr.X[0][unsel])
        got1 = storage_to_f64(Y1[sel], cfg.dtype)
        got2 = storage_to_f64(Y2[sel], cfg.dtype)
        exp = r.orc.readout_dense_blocked(fr.X, 0, sel)
        e1, e2 = max_abs(got1, exp), max_abs(got2, exp)
        record_margin("noalloc highres k=%d" % kk, len(sel), e2, TOL["bf16"])
        assert e1 <= TOL["bf16"] and e2 <= TOL["bf16"], (e1, e2)
    # 32 forced splits of 1638 rows x 256 wide partials: about 27 MB
    Y = _dev(make_frame(cfg, 0).X)
    before = _host(Y).copy()
    with pytest.raises(rs3.Rs3Error) as ei:
        rs3.readout_noalloc(r.sess.layer, r.sess.grid, 1, Y, 0, r.sess.banks, r.sess.sel_idx, r.sess.sel_count, 0,
                            k, 32, Y, 0, 0)
    assert ei.value.status == rs3.RS3_E_INVALID
    torch.cuda.synchronize()
    assert np.array_equal(_host(Y), before)
