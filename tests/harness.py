"""Test-side drivers: the fp64 oracle pipeline and the HIP session run on the
same seeded inputs (test infrastructure)."""
from __future__ import annotations

import json
import math
import os
from typing import List

import numpy as np

import oracle
from workloads import Config, storage_to_f64

TOL = {"bf16": 2e-2, "f32": 1e-4}

# Largest error seen by each parity check, next to its tolerance: written as
# JSON at the end of the session when RS3_MARGINS_OUT names a file.
MARGINS: List[dict] = []


def record_margin(case: str, n_rows: int, err: float, tol: float):
    test = os.environ.get("PYTEST_CURRENT_TEST", "").split(" ")[0]
    MARGINS.append(dict(test=test, case=case, rows=int(n_rows), max_abs_err=float(err), tol=float(tol),
                        margin=float(tol - err)))


def write_margins():
    path = os.environ.get("RS3_MARGINS_OUT")
    if not path or not MARGINS:
        return
    worst = {}
    for r in MARGINS:
        w = worst.get(r["test"])
        if w is None or r["max_abs_err"] / r["tol"] > w["max_abs_err"] / w["tol"]:
            worst[r["test"]] = dict(r, checks=0, rows_total=0)
    for r in MARGINS:
        worst[r["test"]]["checks"] += 1
        worst[r["test"]]["rows_total"] += r["rows"]
    os.makedirs(os.path.dirname(os.path.abspath(path)), exist_ok=True)
    with open(path, "w") as fh:
        json.dump({"per_test_worst": sorted(worst.values(), key=lambda r: r["test"]), "all": MARGINS}, fh, indent=1)


def grid_masks(cfg: Config, masks_px: np.ndarray) -> np.ndarray:
    """Pixel masks [n_obj][m*s][n*s] -> token-grid masks [n_obj][mn] (down_s)."""
    return np.stack([oracle.down_s(masks_px[o], cfg.s).reshape(-1).astype(np.uint8)
                     for o in range(masks_px.shape[0])])


class OraclePipeline:
    """rope: optional complex rotary table [mn][d_h/2] (Eq. 7) applied to the
    selected queries and to the bank keys by their stored cells."""

    def __init__(self, cfg: Config, W, rope=None):
        self.cfg = cfg
        self.rope = rope
        self.W = {k: storage_to_f64(getattr(W, k), cfg.dtype) for k in ("Wq", "Wk", "Wv", "Wo")}
        npdt = np.uint16 if cfg.dtype == "bf16" else np.float32
        self.tracks: List[oracle.Track] = [oracle.Track() for _ in range(cfg.n_obj)]
        self.banks = [oracle.RingBank(cfg.cap, cfg.f_max, cfg.n_pin, cfg.d_kv, npdt) for _ in range(cfg.n_obj)]

    def select(self, masks_px, X_store, k, seed_box=False):
        cfg = self.cfg
        X = storage_to_f64(X_store, cfg.dtype)
        sel, priors, self.tracks = oracle.select_queries(masks_px, cfg.s, cfg.m, cfg.n, self.tracks, X, k,
                                                         cfg.r_s, cfg.c, seed_box, cfg.union_objects)
        return sel, priors

    def commit(self, K_store, V_store, masks_px, t, pin, fall_min=0, fall_max=None):
        gm = grid_masks(self.cfg, masks_px)
        return [self.banks[o].commit(K_store[o], V_store[o], gm[o], t, pin, fall_min, fall_max)
                for o in range(self.cfg.n_obj)]

    def readout_rows(self, X_store, o, rows):
        """Oracle y for cell indices `rows` of object o (float64 [len][C])."""
        cfg = self.cfg
        xi = 0 if X_store.shape[0] == 1 else o
        X = storage_to_f64(X_store[xi], cfg.dtype)
        K, V, pos = self.banks[o].key_rows()
        Kf, Vf = storage_to_f64(K, cfg.dtype), storage_to_f64(V, cfg.dtype)
        Y = oracle.readout(X, rows, Kf, Vf, self.W["Wq"], self.W["Wk"], self.W["Wv"], self.W["Wo"], cfg.H,
                           rope=self.rope, kpos=pos)
        return Y[np.asarray(rows, dtype=np.int64)]

    def projected_bank(self, o):
        """(K^, V^, key cells) of object o's resident keys in key order, the
        keys turned by their cells when there is a table; cached until the
        bank changes."""
        cfg = self.cfg
        bank = self.banks[o]
        sig = (len(bank.frames), tuple(tuple(f) for f in bank.frame_table().tolist()), bank.err)
        cache = getattr(self, "_proj", {})
        if cache.get(o, (None,))[0] != sig:
            K, V, pos = bank.key_rows()
            Kh, Vh = oracle.project_bank(storage_to_f64(K, cfg.dtype), storage_to_f64(V, cfg.dtype),
                                         self.W["Wk"], self.W["Wv"])
            Kh = oracle.rotate_keys(Kh, self.rope, pos, cfg.H)
            cache[o] = (sig, Kh, Vh)
            self._proj = cache
        return cache[o][1], cache[o][2]

    def readout_dense_blocked(self, X_store, o, rows, block=256):
        """Oracle y for cells `rows` of object o by the whole-matrix
        evaluation, in row blocks against one projection of the bank."""
        cfg = self.cfg
        xi = 0 if X_store.shape[0] == 1 else o
        rows = np.asarray(rows, dtype=np.int64)
        X = storage_to_f64(X_store[xi], cfg.dtype)
        Kh, Vh = self.projected_bank(o)
        out = np.empty((len(rows), cfg.C))
        for b0 in range(0, len(rows), block):
            r = rows[b0:b0 + block]
            out[b0:b0 + block] = oracle.readout_dense_projected(X[r], Kh, Vh, self.W["Wq"], self.W["Wo"], cfg.H,
                                                                rope=self.rope, qpos=r)
        return out

    def readout_dense_rows(self, X_store, o, rows):
        cfg = self.cfg
        xi = 0 if X_store.shape[0] == 1 else o
        rows = np.asarray(rows, dtype=np.int64)
        X = storage_to_f64(X_store[xi], cfg.dtype)[rows]
        K, V, pos = self.banks[o].key_rows()
        Kf, Vf = storage_to_f64(K, cfg.dtype), storage_to_f64(V, cfg.dtype)
        return oracle.readout_dense(X, Kf, Vf, self.W["Wq"], self.W["Wk"], self.W["Wv"], self.W["Wo"], cfg.H,
                                    rope=self.rope, kpos=pos, qpos=rows)


def compare_bank(gpu_export: dict, ring: oracle.RingBank):
    ft = ring.frame_table()
    assert gpu_export["n_frames"] == len(ring.frames), (gpu_export["n_frames"], len(ring.frames))
    assert gpu_export["pin_end"] == ring.pin_end
    assert gpu_export["err"] == ring.err
    assert np.array_equal(gpu_export["frames"], ft), (gpu_export["frames"], ft)
    K, V, pos = ring.key_rows()
    assert gpu_export["n_keys"] == K.shape[0]
    assert np.array_equal(gpu_export["pos"], pos)
    assert np.array_equal(gpu_export["K"].view(np.uint8), np.ascontiguousarray(K).view(np.uint8))
    assert np.array_equal(gpu_export["V"].view(np.uint8), np.ascontiguousarray(V).view(np.uint8))


def sample_rows(sel: np.ndarray, n: int, seed: int) -> np.ndarray:
    if len(sel) <= n:
        return np.asarray(sel)
    rng = np.random.default_rng(seed)
    return np.sort(rng.choice(np.asarray(sel), n, replace=False))


def max_abs(a, b) -> float:
    if a.size == 0:
        return 0.0
    return float(np.max(np.abs(np.asarray(a, np.float64) - np.asarray(b, np.float64))))
