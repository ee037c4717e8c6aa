"""Synthetic workloads for the read-sparse readout and store-sparse commit.

The paper measures whole video-object-segmentation pipelines on public VOS
datasets with trained networks.  Neither is available here, so seeded random
tensors of the same shapes stand in: Gaussian tokens, Gaussian weights scaled
by 1/fan_in, and rotated-ellipse object masks whose areas follow the ranges of
the five workload configurations.  No dataset item is reproduced.

Random-number streams: every array is drawn from
``numpy.random.default_rng([seed, frame, stream_id])`` (PCG64 seeded through
SeedSequence), so any single frame can be regenerated on its own.  Values are
drawn in float32 and rounded once to bfloat16 (round to nearest even) when the
configuration is bf16; both sides consume those stored bits.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from fractions import Fraction
from typing import List, Optional

import numpy as np

# stream ids for default_rng([seed, frame, stream])
_S_X, _S_K, _S_V, _S_MASK, _S_RHO, _S_W, _S_ROPE, _S_STACK = 1, 2, 3, 4, 5, 6, 7, 8


# ----------------------------------------------------------------------------
# dtype plumbing (storage conversion only)
# ----------------------------------------------------------------------------
def bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bfloat16 bit patterns (uint16), round to nearest even.

    Inputs here are finite, so no NaN handling is needed.
    """
    # finite values: u + 0x7FFF + lsb stays below 2^32, so uint32 suffices
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    u = u + (np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1)))
    return (u >> np.uint32(16)).astype(np.uint16)


def bits_to_f32(b: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns -> exact float32 values."""
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def to_storage(x32: np.ndarray, dtype: str) -> np.ndarray:
    """Store float32 draws in the configuration dtype ('bf16' -> uint16 bits)."""
    if dtype == "bf16":
        return bf16_bits(x32)
    if dtype == "f32":
        return np.ascontiguousarray(x32, dtype=np.float32)
    raise ValueError(dtype)


def storage_to_f64(a: np.ndarray, dtype: str) -> np.ndarray:
    """Exact widening of stored values to float64."""
    if dtype == "bf16":
        return bits_to_f32(a).astype(np.float64)
    return np.asarray(a, dtype=np.float32).astype(np.float64)


# ----------------------------------------------------------------------------
# configurations
# ----------------------------------------------------------------------------
@dataclass(frozen=True)
class Config:
    name: str
    m: int
    n: int
    C: int            # query token width (d_model)
    H: int            # heads
    d_h: int          # head width; D = H * d_h = C
    d_kv: int         # width of the bank's raw key/value tokens
    dtype: str        # 'bf16' or 'f32'
    n_obj: int
    shared_x: bool    # one query grid shared by all objects
    union_objects: bool
    f_max: int        # bank frames
    n_pin: int
    cap_frames: int   # bank capacity in units of mn tokens
    area_lo: float    # ellipse area fraction range per frame
    area_hi: float
    rho_lo: Optional[float]   # per-frame keep ratio range (None: rho fixed)
    rho_hi: Optional[float]
    rho: Optional[float]
    seed: int
    drift: bool = False       # one drifting ellipse (long-video workload)
    full_prior: bool = False  # read prior = whole grid
    s: int = 1                # encoder stride of the masks
    r_s: int = 4
    c: int = 14
    n_frames: int = 8

    @property
    def mn(self) -> int:
        return self.m * self.n

    @property
    def D(self) -> int:
        return self.H * self.d_h

    @property
    def cap(self) -> int:
        return self.cap_frames * self.mn


CONFIGS = {
    # 16x16 grid, fp32, one head of 64, k/v width 32, two-frame bank
    "tiny_f32": Config("tiny_f32", 16, 16, 64, 1, 64, 32, "f32", 1, True, True,
                       2, 1, 3, 0.30, 0.30, None, None, 0.25, 0, n_frames=8),
    # SAM2-like single object: 64x64 grid, bf16, d_model 256, one head, k/v 64,
    # 1 conditioning + 6 recent frames
    "sam2_single": Config("sam2_single", 64, 64, 256, 1, 256, 64, "bf16", 1, True, True,
                          7, 1, 8, 0.10, 0.40, 0.15, 0.30, None, 1, n_frames=227),
    # eight objects on one shared grid, per-object banks and keep-sets
    "multi_obj8": Config("multi_obj8", 64, 64, 256, 1, 256, 64, "bf16", 8, True, False,
                         7, 1, 8, 0.05, 0.25, 0.15, 0.30, None, 2, n_frames=227),
    # long video: bank grows to 64 frames, drifting ellipse, rho = 0.3
    "long_video": Config("long_video", 64, 64, 256, 1, 256, 64, "bf16", 1, True, True,
                         64, 1, 65, 0.10, 0.30, None, None, 0.3, 3, drift=True, n_frames=300),
    # high-res: 128x128 grid, 8 heads of 32, 16-frame bank, prior = whole grid
    "highres": Config("highres", 128, 128, 256, 8, 32, 64, "bf16", 1, True, True,
                      16, 1, 17, 0.05, 0.50, None, None, 0.25, 4, full_prior=True, n_frames=76),
}


def k_from_rho(rho, mn: int) -> int:
    """k = floor(rho * mn) evaluated exactly (rho given as a decimal string,
    Fraction or float; a float is taken at its exact binary value)."""
    if isinstance(rho, str):
        fr = Fraction(rho)
    else:
        fr = Fraction(rho)
    return int(math.floor(fr * mn))


def fall_counts(lo, hi, mn: int):
    """Integer thresholds for the write fall-through: a frame falls through
    when count < fall_min or count > fall_max; (lo, hi) = (0, 1) is off."""
    # floats go through their shortest decimal form (0.05 -> 1/20, not the
    # binary value just above it)
    flo, fhi = (Fraction(repr(v)) if isinstance(v, float) else Fraction(v) for v in (lo, hi))
    fall_min = int(math.ceil(flo * mn))
    fall_max = int(math.floor(fhi * mn))
    return fall_min, fall_max


# ----------------------------------------------------------------------------
# masks
# ----------------------------------------------------------------------------
def _ellipse_cells(m, n, cy, cx, A, B, theta):
    yy, xx = np.meshgrid(np.arange(m) + 0.5, np.arange(n) + 0.5, indexing="ij")
    dy, dx = yy - cy, xx - cx
    ct, st = math.cos(theta), math.sin(theta)
    u = (dx * ct + dy * st) / A
    v = (-dx * st + dy * ct) / B
    return ((u * u + v * v) <= 1.0).astype(np.uint8)


def _ellipse_params(rng, m, n, area):
    kappa = math.exp(rng.uniform(-math.log(2.0), math.log(2.0)))
    A = math.sqrt(area * m * n * kappa / math.pi)
    B = math.sqrt(area * m * n / (math.pi * kappa))
    theta = rng.uniform(0.0, math.pi)
    ex = math.sqrt((A * math.cos(theta)) ** 2 + (B * math.sin(theta)) ** 2)
    ey = math.sqrt((A * math.sin(theta)) ** 2 + (B * math.cos(theta)) ** 2)
    cx = rng.uniform(ex, n - ex) if 2 * ex < n else n / 2.0
    cy = rng.uniform(ey, m - ey) if 2 * ey < m else m / 2.0
    return cy, cx, A, B, theta, kappa


def ellipse_mask(rng, m, n, area) -> np.ndarray:
    """Rotated ellipse of target area fraction `area`; cell (y, x) is set iff
    its centre (y + 1/2, x + 1/2) lies inside.  Returns uint8 [m][n]."""
    cy, cx, A, B, theta, _ = _ellipse_params(rng, m, n, area)
    return _ellipse_cells(m, n, cy, cx, A, B, theta)


# ----------------------------------------------------------------------------
# tensors
# ----------------------------------------------------------------------------
@dataclass
class Weights:
    Wq: np.ndarray   # [C][D]
    Wk: np.ndarray   # [d_kv][D]
    Wv: np.ndarray   # [d_kv][D]
    Wo: np.ndarray   # [D][C]


def make_weights(cfg: Config, logit_scale: float = 1.0) -> Weights:
    """Gaussian weights N(0, 1/fan_in) in the configuration dtype.

    `logit_scale` multiplies W_q (used by tests that want peaked softmax)."""
    rng = np.random.default_rng([cfg.seed, 0, _S_W])
    D = cfg.D
    wq = rng.standard_normal((cfg.C, D), dtype=np.float32) / np.float32(math.sqrt(cfg.C))
    wk = rng.standard_normal((cfg.d_kv, D), dtype=np.float32) / np.float32(math.sqrt(cfg.d_kv))
    wv = rng.standard_normal((cfg.d_kv, D), dtype=np.float32) / np.float32(math.sqrt(cfg.d_kv))
    wo = rng.standard_normal((D, cfg.C), dtype=np.float32) / np.float32(math.sqrt(D))
    wq = wq * np.float32(logit_scale)
    return Weights(*(to_storage(w, cfg.dtype) for w in (wq, wk, wv, wo)))


STACK_MATRICES = ("Wqs", "Wks", "Wvs", "Wos", "Wq", "Wk", "Wv", "Wo", "W1", "W2")
STACK_NORMS = ("ln1_g", "ln1_b", "ln2_g", "ln2_b", "ln3_g", "ln3_b")


def make_stack_weights(C: int, d_kv: int, F: int, n_layers: int, dtype: str = "bf16", seed: int = 0,
                       branch_scale: float = 0.5) -> List[dict]:
    """Synthetic weights of an L-layer memory-attention stack (no trained
    weights exist for it).  Per layer: Gaussian matrices N(0, 1/fan_in)
    W_qs, W_ks, W_vs, W_os [C][C], W_q [C][C], W_k, W_v [d_kv][C],
    W_o [C][C], W_1 [C][F], W_2 [F][C] in the storage dtype, the three
    output maps of the residual branches (W_os, W_o, W_2) times
    `branch_scale` so that each layer changes the stream by a fraction of
    its size; norm gains 1 + 0.1 N(0, 1) and shifts 0.1 N(0, 1) in float32.
    Layer l draws from default_rng([seed, l, stream])."""
    shapes = {"Wqs": (C, C), "Wks": (C, C), "Wvs": (C, C), "Wos": (C, C), "Wq": (C, C), "Wk": (d_kv, C),
              "Wv": (d_kv, C), "Wo": (C, C), "W1": (C, F), "W2": (F, C)}
    out = []
    for layer in range(n_layers):
        rng = np.random.default_rng([seed, layer, _S_STACK])
        w = {}
        for name in STACK_MATRICES:
            r, c = shapes[name]
            a = rng.standard_normal((r, c), dtype=np.float32) / np.float32(math.sqrt(r))
            if name in ("Wos", "Wo", "W2"):
                a = a * np.float32(branch_scale)
            w[name] = to_storage(a, dtype)
        for name in STACK_NORMS:
            v = rng.standard_normal(C, dtype=np.float32) * np.float32(0.1)
            w[name] = (v + np.float32(1.0)) if name.endswith("_g") else v
        out.append(w)
    return out


def make_rope_table(cfg: Config, seed: int = 0) -> np.ndarray:
    """A random rotary table of unit factors, float32 [mn][d_h/2][2] holding
    (cos, sin) of angles drawn uniformly from [0, 2 pi): an arbitrary table
    for the gather of Eq. 7, passed to both sides as it is."""
    rng = np.random.default_rng([cfg.seed, seed, _S_ROPE])
    ang = rng.uniform(0.0, 2.0 * math.pi, (cfg.mn, cfg.d_h // 2))
    return np.stack([np.cos(ang), np.sin(ang)], axis=-1).astype(np.float32)


def make_decoder_logits(n_obj: int, H: int, W: int, seed: int, dtype: str = "bf16",
                        area=(0.05, 0.3), hole_p: float = 0.04, n_blobs: int = 6) -> np.ndarray:
    """Synthetic mask-decoder logits [n_obj][H][W]: per object a seeded
    rotated ellipse with logits ~ +|N(2, 1)| inside and -|N(2, 1)| outside,
    salt-and-pepper holes (inside pixels turned negative with probability
    hole_p) and n_blobs square holes of side 1..12 inside it.  Objects
    overlap where their ellipses do."""
    rng = np.random.default_rng([seed, H, W, _S_MASK])
    out = np.empty((n_obj, H, W), dtype=np.float32)
    for o in range(n_obj):
        inside = ellipse_mask(rng, H, W, float(rng.uniform(*area))).astype(bool)
        mag = np.abs(rng.normal(2.0, 1.0, (H, W))).astype(np.float32)
        lo = np.where(inside, mag, -mag)
        flip = inside & (rng.random((H, W)) < hole_p)
        lo[flip] = -lo[flip]
        ys, xs = np.nonzero(inside)
        for _ in range(n_blobs if len(ys) else 0):
            j = int(rng.integers(len(ys)))
            side = int(rng.integers(1, 13))
            blk = lo[ys[j]:ys[j] + side, xs[j]:xs[j] + side]
            blk[...] = -np.abs(blk)
        out[o] = lo
    return to_storage(out, dtype)


@dataclass
class FrameInputs:
    X: np.ndarray       # [n_x][mn][C] (n_x = 1 when the grid is shared)
    Kmem: np.ndarray    # [n_obj][mn][d_kv]
    Vmem: np.ndarray    # [n_obj][mn][d_kv]


def make_frame(cfg: Config, frame: int) -> FrameInputs:
    """Fresh N(0,1) query tokens and memory-encoder tokens for one frame."""
    n_x = 1 if cfg.shared_x else cfg.n_obj
    rx = np.random.default_rng([cfg.seed, frame, _S_X])
    rk = np.random.default_rng([cfg.seed, frame, _S_K])
    rv = np.random.default_rng([cfg.seed, frame, _S_V])
    X = rx.standard_normal((n_x, cfg.mn, cfg.C), dtype=np.float32)
    K = rk.standard_normal((cfg.n_obj, cfg.mn, cfg.d_kv), dtype=np.float32)
    V = rv.standard_normal((cfg.n_obj, cfg.mn, cfg.d_kv), dtype=np.float32)
    return FrameInputs(*(to_storage(a, cfg.dtype) for a in (X, K, V)))


@dataclass
class Sequence:
    """Per-frame masks and keep budgets of one seeded video.

    masks[t] is uint8 [n_obj][m*s][n*s]; read_masks[t] is the mask the read
    prior of frame t is built from (masks[t-1], or all ones when the prior is
    the whole grid); k[t] is the per-group keep budget floor(rho_t * mn)."""
    masks: List[np.ndarray] = field(default_factory=list)
    k: List[List[int]] = field(default_factory=list)
    areas: List[List[float]] = field(default_factory=list)

    def read_mask(self, cfg: Config, t: int) -> np.ndarray:
        if cfg.full_prior:
            return np.ones_like(self.masks[t])
        return self.masks[max(t - 1, 0)]


def make_sequence(cfg: Config, n_frames: Optional[int] = None,
                  rho_override=None) -> Sequence:
    n_frames = cfg.n_frames if n_frames is None else n_frames
    seq = Sequence()
    n_groups = 1 if cfg.union_objects else cfg.n_obj
    drift_state = None
    for t in range(n_frames):
        rm = np.random.default_rng([cfg.seed, t, _S_MASK])
        rr = np.random.default_rng([cfg.seed, t, _S_RHO])
        frame_masks, frame_areas = [], []
        for o in range(cfg.n_obj):
            if cfg.drift:
                if drift_state is None:
                    r0 = np.random.default_rng([cfg.seed, 0, _S_MASK, 99])
                    area = r0.uniform(cfg.area_lo, cfg.area_hi)
                    cy, cx, A, B, theta, kappa = _ellipse_params(r0, cfg.m, cfg.n, area)
                    ang = r0.uniform(0.0, 2 * math.pi)
                    drift_state = dict(area=area, cy=cy, cx=cx, theta=theta, kappa=kappa,
                                       vy=0.5 * math.sin(ang), vx=0.5 * math.cos(ang))
                else:
                    st = drift_state
                    st["area"] = float(np.clip(st["area"] + rm.uniform(-0.01, 0.01),
                                               cfg.area_lo, cfg.area_hi))
                    st["theta"] += rm.uniform(-0.05, 0.05)
                    for ax, vel, lim in (("cy", "vy", cfg.m), ("cx", "vx", cfg.n)):
                        p = st[ax] + st[vel]
                        if p < 0 or p > lim:
                            st[vel] = -st[vel]
                            p = st[ax] + st[vel]
                        st[ax] = p
                st = drift_state
                A = math.sqrt(st["area"] * cfg.mn * st["kappa"] / math.pi)
                B = math.sqrt(st["area"] * cfg.mn / (math.pi * st["kappa"]))
                grid = _ellipse_cells(cfg.m, cfg.n, st["cy"], st["cx"], A, B, st["theta"])
                area = st["area"]
            else:
                area = rm.uniform(cfg.area_lo, cfg.area_hi)
                grid = ellipse_mask(rm, cfg.m, cfg.n, area)
            if cfg.s > 1:
                grid = np.repeat(np.repeat(grid, cfg.s, axis=0), cfg.s, axis=1)
            frame_masks.append(grid)
            frame_areas.append(area)
        seq.masks.append(np.stack(frame_masks).astype(np.uint8))
        seq.areas.append(frame_areas)
        ks = []
        for g in range(n_groups):
            if rho_override is not None:
                ks.append(k_from_rho(rho_override, cfg.mn))
            elif cfg.rho is not None:
                ks.append(k_from_rho(repr(cfg.rho), cfg.mn))
            else:
                ks.append(k_from_rho(rr.uniform(cfg.rho_lo, cfg.rho_hi), cfg.mn))
        seq.k.append(ks)
    return seq
