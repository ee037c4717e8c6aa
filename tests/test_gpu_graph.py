"""The hot calls under HIP stream capture.

Four frames of select + readout + commit are captured into one graph and
replayed several times, with eager work and synchronisations between the
replays.  A second session runs the same frames eagerly; after every replay
the outputs, the last selection, the tracker state and the bank must equal
the eager ones bit for bit (the kernels are deterministic, so the two
sessions walk through identical states)."""
import numpy as np
import pytest

from workloads import CONFIGS, make_frame, make_sequence, make_weights

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


def _session(cfg, W, absorb):
    from paper_2608_22526_amd.session import Session
    return Session(m=cfg.m, n=cfg.n, s=cfg.s, C=cfg.C, H=cfg.H, d_kv=cfg.d_kv, dtype=cfg.dtype, n_obj=cfg.n_obj,
                   shared_x=cfg.shared_x, union_objects=cfg.union_objects, cap=cfg.cap, f_max=cfg.f_max,
                   n_pin=cfg.n_pin, weights=W, r_s=cfg.r_s, c=cfg.c, max_sel=cfg.mn, absorb=absorb)


@pytest.mark.parametrize("absorb", [False, True])
def test_graph_replay_matches_eager(absorb):
    from paper_2608_22526_amd.session import to_device, to_host

    cfg = CONFIGS["sam2_single"]
    n_pre, n_cap = cfg.f_max, 4
    W = make_weights(cfg)
    seq = make_sequence(cfg, n_frames=n_pre + n_cap)
    frames = []
    for t in range(n_pre + n_cap):
        fr = make_frame(cfg, t)
        frames.append(dict(X=to_device(fr.X), K=to_device(fr.Kmem), V=to_device(fr.Vmem),
                           mask=to_device(seq.masks[t]), rmask=to_device(seq.read_mask(cfg, t)), k=seq.k[t]))
    eager, graphed = _session(cfg, W, absorb), _session(cfg, W, absorb)
    for sess in (eager, graphed):
        for t in range(n_pre):
            f = frames[t]
            sess.commit(f["K"], f["V"], f["mask"], t, t < cfg.n_pin)
    Y = {id(s): [torch.empty_like(frames[0]["X"]) for _ in range(n_cap)] for s in (eager, graphed)}

    def run(sess):
        for j in range(n_cap):
            t = n_pre + j
            f = frames[t]
            sess.select(f["rmask"], f["X"], f["k"])
            sess.readout(f["X"], Y[id(sess)][j])
            sess.commit(f["K"], f["V"], f["mask"], t, False)

    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        run(graphed)
    torch.cuda.synchronize()
    for rep in range(3):
        g.replay()
        torch.cuda.synchronize()
        run(eager)
        torch.cuda.synchronize()
        for j in range(n_cap):
            assert torch.equal(Y[id(eager)][j], Y[id(graphed)][j]), (rep, j)
        assert np.array_equal(to_host(eager.sel_count), to_host(graphed.sel_count)), rep
        assert np.array_equal(to_host(eager.sel_idx), to_host(graphed.sel_idx)), rep
        assert np.array_equal(eager.track.export(), graphed.track.export()), rep
        a, b = eager.banks[0].export(), graphed.banks[0].export()
        for key in ("n_frames", "pin_end", "err", "n_keys"):
            assert a[key] == b[key], (rep, key)
        for key in ("frames", "K", "V", "pos"):
            assert np.array_equal(a[key], b[key]), (rep, key)
        assert a["err"] == 0
    del g
