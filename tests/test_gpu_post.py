"""Closure of the decoded masks and the palette argmax (Sec. 3.3; the end of
Algorithm 1) through the C ABI against the fp64 oracle: closed masks and
palettes bit-exact for 1 to 8 overlapping objects with salt-and-pepper and
block holes, structuring elements 1 to 15, bf16 and fp32 logits, ragged,
tall and 4096-wide images; the closed masks then drive the next selection
(the tracker update) exactly as the oracle's do."""
import numpy as np
import pytest

import oracle
from test_gpu_parity import Runner, _dev, _host
from workloads import CONFIGS, make_decoder_logits, make_frame, storage_to_f64

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


def _close_gpu(L_store, dtype, k, want_closed=True, want_palette=True):
    import paper_2608_22526_amd as rs3
    n_obj, H, W = L_store.shape
    ws = torch.zeros(rs3.close_workspace_size(n_obj, H, W), dtype=torch.uint8, device="cuda")
    closed = torch.full((n_obj, H, W), 9, dtype=torch.uint8, device="cuda") if want_closed else None
    pal = torch.full((H, W), 99, dtype=torch.uint8, device="cuda") if want_palette else None
    rs3.close_masks(n_obj, H, W, _dev(L_store), rs3.RS3_BF16 if dtype == "bf16" else rs3.RS3_F32, k, closed, pal,
                    ws)
    torch.cuda.synchronize()
    return (None if closed is None else _host(closed)), (None if pal is None else _host(pal))


@pytest.mark.parametrize("n_obj,H,W,k,dtype", [
    (1, 64, 64, 9, "bf16"), (3, 100, 130, 9, "bf16"), (4, 256, 256, 9, "bf16"), (2, 37, 300, 15, "f32"),
    (8, 128, 192, 3, "f32"), (5, 64, 65, 1, "bf16"), (2, 3, 4096, 9, "bf16"), (1, 2000, 8, 9, "f32"),
    (2, 70, 64, 13, "bf16")])
def test_close_and_palette_bit_exact(n_obj, H, W, k, dtype):
    L = make_decoder_logits(n_obj, H, W, seed=H * 31 + W + k, dtype=dtype)
    closed, pal = _close_gpu(L, dtype, k)
    exp_closed, exp_pal = oracle.close_masks(storage_to_f64(L, dtype), k)
    assert np.array_equal(closed, exp_closed)
    assert np.array_equal(pal, exp_pal)
    # the holes the closing fills are exercised, also under no positive logit
    pos = (storage_to_f64(L, dtype) > 0).any(axis=0)
    if k > 1 and H > 8 and W > 8:
        assert (exp_closed.astype(bool) & ~(storage_to_f64(L, dtype) > 0)).any()
        assert ((exp_pal > 0) & ~pos).any()


def test_optional_outputs_and_argument_errors():
    import paper_2608_22526_amd as rs3
    L = make_decoder_logits(3, 50, 70, seed=5)
    exp_closed, exp_pal = oracle.close_masks(storage_to_f64(L, "bf16"), 9)
    closed, _ = _close_gpu(L, "bf16", 9, want_palette=False)
    assert np.array_equal(closed, exp_closed)
    _, pal = _close_gpu(L, "bf16", 9, want_closed=False)
    assert np.array_equal(pal, exp_pal)
    ws = torch.zeros(rs3.close_workspace_size(3, 50, 70), dtype=torch.uint8, device="cuda")
    small = ws[:-1]
    for bad in (dict(k=8), dict(k=17), dict(ws=small)):
        args = dict(k=9, ws=ws)
        args.update(bad)
        with pytest.raises(rs3.Rs3Error) as ei:
            rs3.close_masks(3, 50, 70, _dev(L), rs3.RS3_BF16, args["k"], None, None, args["ws"])
        assert ei.value.status == rs3.RS3_E_INVALID
    with pytest.raises(rs3.Rs3Error):
        rs3.close_workspace_size(3, 50, 5000)


def test_closed_masks_drive_the_next_selection():
    # decoded logits of frame t-1 -> closed masks -> the prior and tracker
    # update of frame t, on both sides
    cfg = CONFIGS["multi_obj8"]
    r = Runner(cfg, 3)
    L = make_decoder_logits(cfg.n_obj, cfg.m * cfg.s, cfg.n * cfg.s, seed=17, area=(0.03, 0.15))
    closed, _ = _close_gpu(L, "bf16", 9, want_palette=False)
    exp_closed, _ = oracle.close_masks(storage_to_f64(L, "bf16"), 9)
    assert np.array_equal(closed, exp_closed)
    fr = make_frame(cfg, 1)
    k = r.seq.k[1]
    prior = torch.zeros((r.sess.n_groups, cfg.mn), dtype=torch.uint8, device="cuda")
    r.sess.select(_dev(closed), _dev(fr.X), k, prior_out=prior)
    sel, priors = r.orc.select(exp_closed, fr.X, k)
    torch.cuda.synchronize()
    cnt, idx = _host(r.sess.sel_count), _host(r.sess.sel_idx)
    for g in range(r.sess.n_groups):
        assert np.array_equal(idx[g, :cnt[g]], sel[g])
    assert np.array_equal(_host(prior).astype(bool), priors)
    exp_tracks = np.array([tr.as_list() for tr in r.orc.tracks], dtype=np.int32)
    assert np.array_equal(r.sess.track.export(), exp_tracks)
