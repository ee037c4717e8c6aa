"""Edge cases of the HIP path against the oracle: empty and full masks, the
lost-object streak, k = 0 and k = mn, tied energies, stride-2 masks, the
write fall-through, capacity errors, zero-length frames and invalid
selection lists."""
from dataclasses import replace

import numpy as np
import pytest

from harness import OraclePipeline, compare_bank
from workloads import CONFIGS, make_weights, storage_to_f64, to_storage
import oracle

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


def _dev(a):
    from paper_2608_22526_amd.session import to_device
    return to_device(a)


def _host(t):
    from paper_2608_22526_amd.session import to_host
    return to_host(t)


def _session(cfg, W, **kw):
    from paper_2608_22526_amd.session import Session
    return Session(m=cfg.m, n=cfg.n, s=cfg.s, C=cfg.C, H=cfg.H, d_kv=cfg.d_kv, dtype=cfg.dtype,
                   n_obj=cfg.n_obj, shared_x=cfg.shared_x, union_objects=cfg.union_objects, cap=cfg.cap,
                   f_max=cfg.f_max, n_pin=cfg.n_pin, weights=W, r_s=cfg.r_s, c=cfg.c, **kw)


SMALL = replace(CONFIGS["sam2_single"], m=24, n=20, C=64, H=1, d_h=64, d_kv=16, f_max=4, cap_frames=3)


def _check_select(sess, orc, masks, X, k, seed_box=False):
    prior = torch.zeros((sess.n_groups, sess.mn), dtype=torch.uint8, device="cuda")
    sess.select(_dev(masks), _dev(X), k, seed_box=seed_box, prior_out=prior)
    sel, pri = orc.select(masks, X, k, seed_box=seed_box)
    torch.cuda.synchronize()
    cnt, idx = _host(sess.sel_count), _host(sess.sel_idx)
    for g in range(sess.n_groups):
        assert cnt[g] == len(sel[g])
        assert np.array_equal(idx[g, :cnt[g]], sel[g])
    assert np.array_equal(_host(prior).astype(bool), pri)
    exp_tracks = np.array([t.as_list() for t in orc.tracks], dtype=np.int32)
    assert np.array_equal(sess.track.export(), exp_tracks)
    return sel


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_streak_empty_full_and_k_extremes(dtype):
    cfg = replace(SMALL, dtype=dtype)
    W = make_weights(cfg)
    sess, orc = _session(cfg, W), OraclePipeline(cfg, W)
    rng = np.random.default_rng(0)
    X = to_storage(rng.standard_normal((1, cfg.mn, cfg.C)).astype(np.float32), dtype)
    m0 = np.zeros((1, cfg.m, cfg.n), np.uint8)
    m0[0, 5:9, 3:12] = 1
    empty = np.zeros_like(m0)
    full = np.ones_like(m0)
    _check_select(sess, orc, m0, X, [50])
    for t in range(20):                   # streak grows to the cap and stays
        _check_select(sess, orc, empty, X, [cfg.mn])
    _check_select(sess, orc, full, X, [0])          # k = 0
    _check_select(sess, orc, full, X, [cfg.mn])     # keep everything
    _check_select(sess, orc, m0, X, [7], seed_box=True)
    one = np.zeros_like(m0)
    one[0, 0, cfg.n - 1] = 1
    _check_select(sess, orc, one, X, [3])


def test_tied_energies():
    cfg = SMALL
    W = make_weights(cfg)
    sess, orc = _session(cfg, W), OraclePipeline(cfg, W)
    rng = np.random.default_rng(1)
    base = rng.standard_normal((4, cfg.C)).astype(np.float32)
    X = to_storage(base[rng.integers(0, 4, size=cfg.mn)][None], "bf16")   # four distinct energies
    full = np.ones((1, cfg.m, cfg.n), np.uint8)
    for k in (1, 13, 100, 333, cfg.mn - 1):
        _check_select(sess, orc, full, X, [k])


def test_stride2_masks_and_groups():
    cfg = replace(SMALL, s=2, n_obj=3, union_objects=False)
    W = make_weights(cfg)
    sess, orc = _session(cfg, W), OraclePipeline(cfg, W)
    rng = np.random.default_rng(2)
    X = to_storage(rng.standard_normal((1, cfg.mn, cfg.C)).astype(np.float32), "bf16")
    masks = (rng.random((3, cfg.m * 2, cfg.n * 2)) < 0.05).astype(np.uint8)
    masks[1] = 0
    for t in range(3):
        _check_select(sess, orc, masks, X, [40, 60, 80])
        masks = np.roll(masks, 1, axis=0)
    cfgu = replace(cfg, union_objects=True)
    sess2, orc2 = _session(cfgu, W), OraclePipeline(cfgu, W)
    _check_select(sess2, orc2, masks, X, [90])


def test_commit_ring_rules_fall_through_and_capacity():
    cfg = replace(SMALL, m=8, n=8, cap_frames=2, f_max=4)   # cap = 128 rows
    W = make_weights(cfg)
    sess, orc = _session(cfg, W), OraclePipeline(cfg, W)
    rng = np.random.default_rng(3)
    npdt = np.uint16
    sizes = [10, 30, 0, 64, 25, 40, 64, 64, 3, 0, 50]
    for t, L in enumerate(sizes):
        K = to_storage(rng.standard_normal((1, cfg.mn, cfg.d_kv)).astype(np.float32), "bf16")
        V = to_storage(rng.standard_normal((1, cfg.mn, cfg.d_kv)).astype(np.float32), "bf16")
        mask = np.zeros((1, cfg.m, cfg.n), np.uint8)
        mask.reshape(-1)[rng.choice(cfg.mn, L, replace=False)] = 1
        fmin, fmax = (4, 60) if t % 3 == 2 else (0, cfg.mn)
        pin = t == 0
        sess.commit(_dev(K), _dev(V), _dev(mask), t, pin, fmin, fmax)
        counts = orc.commit(K, V, mask, t, pin, fmin, fmax)
        torch.cuda.synchronize()
        assert _host(sess.kept_count).tolist() == counts
        compare_bank(sess.banks[0].export(), orc.banks[0])
    # a frame longer than cap - pin_end is a capacity error; the bank stays
    cfg2 = replace(cfg, cap_frames=1)
    sess2, orc2 = _session(cfg2, W), OraclePipeline(cfg2, W)
    K = to_storage(rng.standard_normal((1, cfg.mn, cfg.d_kv)).astype(np.float32), "bf16")
    m_half = np.zeros((1, cfg.m, cfg.n), np.uint8)
    m_half[0, :2] = 1
    full = np.ones_like(m_half)
    for t, (mk, pin) in enumerate([(m_half, True), (full, False), (m_half, False)]):
        sess2.commit(_dev(K), _dev(K), _dev(mk), t, pin)
        orc2.commit(K, K, mk, t, pin)
        torch.cuda.synchronize()
        compare_bank(sess2.banks[0].export(), orc2.banks[0])
    assert sess2.banks[0].error() == oracle.RS3_E_CAPACITY


def test_pin_misuse_rejected_on_host():
    from paper_2608_22526_amd import Rs3Error
    cfg = replace(SMALL, m=8, n=8)
    W = make_weights(cfg)
    sess = _session(cfg, W)
    K = _dev(np.zeros((1, cfg.mn, cfg.d_kv), np.uint16))
    mask = _dev(np.ones((1, cfg.m, cfg.n), np.uint8))
    sess.commit(K, K, mask, 0, False)
    with pytest.raises(Rs3Error):
        sess.commit(K, K, mask, 1, True)


def test_invalid_selection_sets_error_and_skips_rows():
    cfg = SMALL
    W = make_weights(cfg)
    sess = _session(cfg, W)
    rng = np.random.default_rng(4)
    K = to_storage(rng.standard_normal((1, cfg.mn, cfg.d_kv)).astype(np.float32), "bf16")
    sess.commit(_dev(K), _dev(K), _dev(np.ones((1, cfg.m, cfg.n), np.uint8)), 0, True)
    X = _dev(to_storage(rng.standard_normal((1, cfg.mn, cfg.C)).astype(np.float32), "bf16"))
    sess.sel_idx[0, :4] = torch.tensor([3, 2, 7, cfg.mn + 5], dtype=torch.int32)   # not ascending, out of range
    sess.sel_count[0] = 4
    Y = X.clone()
    sess.readout(Y, Y)
    torch.cuda.synchronize()
    assert sess.banks[0].error(clear=True) == oracle.RS3_E_INVALID
    assert sess.banks[0].error() == 0
    Yh, Xh = _host(Y), _host(X)
    # rows 2 (non-ascending) and the out-of-range entry are skipped
    assert np.array_equal(Yh[0, 2], Xh[0, 2])


def test_tall_grid_byte_path_and_max_cells():
    """8192 x 4 grid: too many rows for the row-bitmask prior (byte path) and
    32 cells per select thread (the largest grid, mn = 32768)."""
    cfg = replace(SMALL, m=8192, n=4, C=64, d_kv=16, cap_frames=1, f_max=2)
    W = make_weights(cfg)
    sess, orc = _session(cfg, W), OraclePipeline(cfg, W)
    rng = np.random.default_rng(5)
    X = to_storage(rng.standard_normal((1, cfg.mn, cfg.C)).astype(np.float32), "bf16")
    masks = (rng.random((1, cfg.m, cfg.n)) < 0.002).astype(np.uint8)
    sel = _check_select(sess, orc, masks, X, [1000])
    assert len(sel[0]) == 1000
    _check_select(sess, orc, np.zeros_like(masks), X, [100])     # box fallback of the cached box


def test_wide_grid_multiword_rows():
    """Rows of 200 cells span four 64-bit words in the bitmask prior."""
    cfg = replace(SMALL, m=40, n=200, C=64, d_kv=16, cap_frames=1, f_max=2, r_s=9)
    W = make_weights(cfg)
    sess, orc = _session(cfg, W), OraclePipeline(cfg, W)
    rng = np.random.default_rng(6)
    X = to_storage(rng.standard_normal((1, cfg.mn, cfg.C)).astype(np.float32), "bf16")
    masks = (rng.random((1, cfg.m, cfg.n)) < 0.004).astype(np.uint8)
    masks[0, 7, 63] = masks[0, 7, 64] = masks[0, 30, 127] = masks[0, 2, 199] = masks[0, 39, 0] = 1
    _check_select(sess, orc, masks, X, [2000])


# (grid rows, grid columns, channels, objects, dtype): each call takes the
# wide energy form (at least 256 blocks of 256 rows): fp32 rows of 72
# channels (18 chunks: a short last column slice) on 4,100-cell grids (a
# short last row block) through the energy launch without the prior; 64x64
# bf16 grids of 64 channels through the launch with the prior beside; and
# the batch shape of 64 grids of 64x64 x 256 channels (four slices).
WIDE_ENERGY = {
    "f32_c72_100x41_obj64": (100, 41, 72, 64, "f32"),
    "bf16_c64_64x64_obj16": (64, 64, 64, 16, "bf16"),
    "bf16_c256_64x64_obj64": (64, 64, 256, 64, "bf16"),
}


@pytest.mark.parametrize("case", sorted(WIDE_ENERGY))
def test_energy_wide_batches(case):
    """Energies (Eq. 4) of large batches, bit-exact: the fp64 sums and the
    per-64-cell minimum/maximum words in the selection workspace, the
    selected lists, priors and tracker states of two frames."""
    m, n, C, nobj, dt = WIDE_ENERGY[case]
    cfg = replace(SMALL, m=m, n=n, C=C, d_h=C, n_obj=nobj, shared_x=False, union_objects=False, dtype=dt,
                  cap_frames=1, f_max=2)
    W = make_weights(cfg)
    sess, orc = _session(cfg, W), OraclePipeline(cfg, W)
    rng = np.random.default_rng(17)
    mn = cfg.mn
    nb = (mn + 63) // 64
    for frame in range(2):
        X = to_storage(rng.standard_normal((nobj, mn, C)).astype(np.float32), dt)
        masks = (rng.random((nobj, m, n)) < 0.01).astype(np.uint8)
        k = [int(x) for x in rng.integers(1, mn // 3, nobj)]
        _check_select(sess, orc, masks, X, k)
        ws = _host(sess.ws_sel)
        e = ws[:nobj * mn * 8].view(np.float64).reshape(nobj, mn)
        r0 = (nobj * mn * 8 + 255) // 256 * 256
        rng_words = ws[r0:r0 + nobj * nb * 16].view(np.uint64).reshape(nobj, nb, 2)
        Xf = storage_to_f64(X, dt)
        for o in range(nobj):
            eo = oracle.energy(Xf[o])
            assert np.array_equal(e[o].view(np.uint64), eo.view(np.uint64)), (case, frame, o)
            bits = np.zeros(nb * 64, np.uint64)
            bits[:mn] = eo.view(np.uint64)
            lo = np.where(np.arange(nb * 64) < mn, bits, np.uint64(~np.uint64(0))).reshape(nb, 64).min(axis=1)
            hi = bits.reshape(nb, 64).max(axis=1)
            assert np.array_equal(rng_words[o, :, 0], lo) and np.array_equal(rng_words[o, :, 1], hi), (case, o)
