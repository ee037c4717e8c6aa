"""rs3_frame (select + readout + commit of one frame in one call) through the
C ABI: for every layer form it must give, bit for bit, what the separate
calls rs3_select_queries and rs3_readout_commit give on the same inputs
(selected lists and counts, priors, tracker state, outputs, kept counts and
banks), including the form whose energy launch projects the query of every
cell for the attention (one head of 64 at d_model 256); and over a sequence
it must match the fp64 oracle (Eq. 6 within 2e-2, everything else bit-exact)."""
from dataclasses import replace

import numpy as np
import pytest

import oracle
from harness import OraclePipeline, TOL, compare_bank, max_abs, record_margin
from test_gpu_parity import _dev, _host, _session
from workloads import CONFIGS, k_from_rho, make_frame, make_sequence, make_weights, storage_to_f64

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

CASES = {
    "sam2_absorbed": (CONFIGS["sam2_single"], dict(absorb=True), None),        # projection in the energy launch
    "sam2_projected": (CONFIGS["sam2_single"], dict(absorb=False), None),
    "multi8_absorbed": (CONFIGS["multi_obj8"], dict(absorb=True), None),       # shared grid, per-object groups
    "own_grids_absorbed": (replace(CONFIGS["multi_obj8"], n_obj=3, shared_x=False), dict(absorb=True), None),
    "four_heads_64": (replace(CONFIGS["sam2_single"], H=4, d_h=64), {}, None),
    "rope_projected": (replace(CONFIGS["sam2_single"], m=32, n=32, f_max=4, cap_frames=4), {}, 10000.0),
    "tiny_f32": (CONFIGS["tiny_f32"], {}, None),
    "highres_8x32": (replace(CONFIGS["highres"], f_max=3, cap_frames=4), {}, None),
}


@pytest.mark.parametrize("case", list(CASES))
def test_frame_equals_separate_calls(case):
    cfg, kw, rope = CASES[case]
    n = cfg.f_max + 4
    W = make_weights(cfg)
    seq = make_sequence(cfg, n_frames=n)
    max_sel = max(max(ks) for ks in seq.k)
    a = _session(cfg, W, max_sel=max_sel, rope_theta=rope, **kw)
    b = _session(cfg, W, max_sel=max_sel, rope_theta=rope, **kw)
    for t in range(cfg.f_max):
        fr = make_frame(cfg, t)
        for sess in (a, b):
            sess.commit(_dev(fr.Kmem), _dev(fr.Vmem), _dev(seq.masks[t]), t, t < cfg.n_pin)
    in_place = cfg.n_obj == 1
    for t in range(cfg.f_max, n):
        fr = make_frame(cfg, t)
        rm, cm = _dev(seq.read_mask(cfg, t)), _dev(seq.masks[t])
        K, V = _dev(fr.Kmem), _dev(fr.Vmem)
        outs, priors = [], []
        for sess, use_frame in ((a, False), (b, True)):
            X = _dev(fr.X)
            Y = X if in_place else torch.empty((cfg.n_obj, cfg.mn, cfg.C), dtype=X.dtype, device="cuda")
            pr = torch.zeros((sess.n_groups, cfg.mn), dtype=torch.uint8, device="cuda")
            if use_frame:
                sess.frame(rm, X, seq.k[t], Y, K, V, cm, t, False, max_sel=max(seq.k[t]), prior_out=pr)
            else:
                sess.select(rm, X, seq.k[t], prior_out=pr)
                sess.readout_commit(X, Y, K, V, cm, t, False, max_sel=max(seq.k[t]))
            torch.cuda.synchronize()
            outs.append(_host(Y))
            priors.append(_host(pr))
        assert np.array_equal(_host(a.sel_count), _host(b.sel_count)), t
        assert np.array_equal(_host(a.sel_idx), _host(b.sel_idx)), t
        assert np.array_equal(priors[0], priors[1]), t
        assert np.array_equal(a.track.export(), b.track.export()), t
        assert np.array_equal(outs[0].view(np.uint8), outs[1].view(np.uint8)), t
        assert np.array_equal(_host(a.kept_count), _host(b.kept_count)), t
        for o in range(cfg.n_obj):
            ea, eb = a.banks[o].export(), b.banks[o].export()
            for key in ("frames", "K", "V", "pos"):
                assert np.array_equal(ea[key], eb[key]), (t, o, key)
            assert (ea["n_frames"], ea["pin_end"], ea["err"]) == (eb["n_frames"], eb["pin_end"], eb["err"])


def test_frame_sequence_matches_oracle():
    """The benchmark workload driven by rs3_frame alone for 12 frames against
    the oracle: bit-exact lists, tracker and bank, every selected row within
    2e-2, unselected rows bit-identical."""
    cfg = CONFIGS["sam2_single"]
    n = 19
    W = make_weights(cfg)
    seq = make_sequence(cfg, n_frames=n)
    sess = _session(cfg, W, max_sel=k_from_rho("0.3", cfg.mn), absorb=True)
    orc = OraclePipeline(cfg, W)
    for t in range(cfg.f_max):
        fr = make_frame(cfg, t)
        sess.commit(_dev(fr.Kmem), _dev(fr.Vmem), _dev(seq.masks[t]), t, t == 0)
        orc.commit(fr.Kmem, fr.Vmem, seq.masks[t], t, t == 0)
    for t in range(cfg.f_max, n):
        fr = make_frame(cfg, t)
        rmask = seq.read_mask(cfg, t)
        X = _dev(fr.X)
        sess.frame(_dev(rmask), X, seq.k[t], X, _dev(fr.Kmem), _dev(fr.Vmem), _dev(seq.masks[t]), t,
                   max_sel=max(seq.k[t]))
        sel, _ = orc.select(rmask, fr.X, seq.k[t])
        exp = orc.readout_dense_blocked(fr.X, 0, sel[0])
        orc.commit(fr.Kmem, fr.Vmem, seq.masks[t], t, False)
        torch.cuda.synchronize()
        cnt = int(_host(sess.sel_count)[0])
        assert np.array_equal(_host(sess.sel_idx)[0, :cnt], sel[0])
        assert np.array_equal(sess.track.export(), np.array([tr.as_list() for tr in orc.tracks], np.int32))
        Y = _host(X)[0]
        err = max_abs(storage_to_f64(Y[sel[0]], cfg.dtype), exp)
        record_margin("frame sam2 t=%d" % t, len(sel[0]), err, TOL["bf16"])
        assert err <= TOL["bf16"], (t, err)
        unsel = np.setdiff1d(np.arange(cfg.mn), sel[0])
        assert np.array_equal(Y[unsel], fr.X[0][unsel])
        compare_bank(sess.banks[0].export(), orc.banks[0])
