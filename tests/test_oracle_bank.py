"""Pins for write compaction and the ring bank (Sec. 3.2, Eq. 8)."""
import json
import os

import numpy as np
import pytest

import oracle
from oracle import RingBank, FrameListBank
from workloads import fall_counts


def test_compact_counts_and_order():
    rng = np.random.default_rng(0)
    for _ in range(20):
        mask = (rng.random(300) < rng.random()).astype(np.uint8)
        kept = oracle.compact(mask)
        assert len(kept) == int(mask.sum())
        assert np.all(np.diff(kept) > 0)
        assert np.all(mask[kept] == 1)


def test_fall_through_thresholds():
    mn = 400
    fmin, fmax = fall_counts("0.05", "0.95", mn)
    assert (fmin, fmax) == (20, 380)
    for cnt, falls in [(19, True), (20, False), (380, False), (381, True), (0, True), (400, True)]:
        mask = np.zeros(mn, np.uint8)
        mask[:cnt] = 1
        kept = oracle.compact(mask, fmin, fmax)
        assert len(kept) == (mn if falls else cnt)
    # off: (0, 1) keeps exactly the mask, including empty and full
    fmin, fmax = fall_counts(0, 1, mn)
    assert len(oracle.compact(np.zeros(mn, np.uint8), fmin, fmax)) == 0
    assert len(oracle.compact(np.ones(mn, np.uint8), fmin, fmax)) == mn


def test_ring_hand_trace(golden_dir):
    g = json.load(open(os.path.join(golden_dir, "ring_trace.json")))
    b = RingBank(g["cap"], g["f_max"], g["n_pin"], 1, np.float64)
    for st in g["steps"]:
        mask = np.zeros(20, np.uint8)
        mask[:st["L"]] = 1
        src = np.arange(20, dtype=np.float64).reshape(20, 1) + 100 * st["t"]
        b.commit(src, -src, mask, st["t"], bool(st["pin"]))
        assert b.frame_table().tolist() == st["frames"], st
        assert b.err == st["err"]
        K, V, pos = b.key_rows()
        exp_rows = np.concatenate([np.arange(f[1]) + 100 * f[2] for f in st["frames"]]) if st["frames"] else []
        assert K[:, 0].tolist() == list(exp_rows)
        assert V[:, 0].tolist() == [-v for v in exp_rows]


def test_ring_matches_frame_list_when_roomy():
    rng = np.random.default_rng(1)
    mn, f_max, n_pin = 64, 5, 1
    cap = mn + (f_max - n_pin + 1) * mn
    ring = RingBank(cap, f_max, n_pin, 3, np.float32)
    lst = FrameListBank(f_max, n_pin)
    commits = []
    for t in range(40):
        mask = (rng.random(mn) < rng.random()).astype(np.uint8)
        K = rng.standard_normal((mn, 3)).astype(np.float32)
        V = rng.standard_normal((mn, 3)).astype(np.float32)
        pin = t == 0
        ring.commit(K, V, mask, t, pin)
        lst.commit(K, V, mask, t, pin)
        commits.append(t)
        assert ring.err == 0
        assert [int(x) for x in ring.frame_table()[:, 2]] == lst.resident_times()
        exp = [0] + commits[1:][-(f_max - n_pin):]
        assert lst.resident_times() == exp
        Kr, Vr, pr = ring.key_rows()
        assert np.array_equal(Kr, np.concatenate([f[2] for f in lst.frames]))
        assert np.array_equal(pr, np.concatenate([f[4] for f in lst.frames]))


def test_ring_small_cap_invariants():
    rng = np.random.default_rng(2)
    mn, f_max, n_pin, cap = 50, 6, 2, 130
    ring = RingBank(cap, f_max, n_pin, 1, np.float64)
    seen = []
    for t in range(200):
        mask = (rng.random(mn) < rng.uniform(0, 0.9)).astype(np.uint8)
        src = np.full((mn, 1), float(t))
        before = ring.frame_table().tolist()
        L = ring.commit(src, src, mask, t, t < n_pin)
        ft = ring.frame_table()
        if L > cap - ring.pin_end and t >= n_pin:
            assert ft.tolist() == before and ring.err == oracle.RS3_E_CAPACITY
            continue
        seen.append(t)
        # resident frames are disjoint, inside the ring, and in commit order
        spans = sorted((s, s + l) for s, l, _, _ in ft.tolist() if l > 0)
        for (a0, a1), (b0, b1) in zip(spans, spans[1:]):
            assert a1 <= b0
        assert all(0 <= s and s + l <= cap for s, l, _, _ in ft.tolist())
        ts = ft[:, 2].tolist()
        assert ts == sorted(ts) and ts[-1] == t
        assert len(ts) <= f_max
        # unpinned residents are a suffix of the unpinned commits (FIFO)
        unp = [x for x in ts if x >= n_pin]
        unp_seen = [x for x in seen if x >= n_pin]
        assert unp == unp_seen[len(unp_seen) - len(unp):]
        K, _, _ = ring.key_rows()
        exp = np.concatenate([np.full(l, float(tt)) for _, l, tt, _ in ft.tolist()])
        assert np.array_equal(K[:, 0], exp)


def test_pin_misuse_rejected():
    b = RingBank(100, 3, 1, 1, np.float64)
    m = np.ones(4, np.uint8)
    s = np.zeros((4, 1))
    b.commit(s, s, m, 0, True)
    with pytest.raises(ValueError):
        b.commit(s, s, m, 1, True)
    b2 = RingBank(100, 3, 1, 1, np.float64)
    b2.commit(s, s, m, 0, False)
    with pytest.raises(ValueError):
        b2.commit(s, s, m, 1, True)
    with pytest.raises(ValueError):
        RingBank(100, 2, 2, 1, np.float64)
