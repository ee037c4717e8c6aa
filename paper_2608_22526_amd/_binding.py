"""ctypes binding of librs3.so (argument marshalling only).

Tensors are torch tensors on the GPU (their data_ptr() is passed); host-side
arrays are numpy.  `stream=None` means torch's current stream.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import numpy as np

RS3_OK, RS3_E_INVALID, RS3_E_CAPACITY, RS3_E_DEVICE, RS3_E_OOM = 0, 1, 2, 3, 4
RS3_F32, RS3_BF16 = 0, 1
RS3_MAX_OBJ = 64
RS3_MAX_MN = 32768
RS3_TRACK_WORDS = 6
RS3_BANK_HDR_WORDS = 8
RS3_NOALLOC_SCRATCH_BYTES = 16 << 20

lib_path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "librs3.so")

c_i32, c_i64, c_sz, c_vp = ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t, ctypes.c_void_p
P_i32 = ctypes.POINTER(ctypes.c_int32)


class Grid(ctypes.Structure):
    _fields_ = [("m", c_i32), ("n", c_i32), ("s", c_i32)]


class SelectParams(ctypes.Structure):
    _fields_ = [("r_s", c_i32), ("c", c_i32), ("seed_box", c_i32), ("union_objects", c_i32)]


class FrameIO(ctypes.Structure):
    """rs3_frame_io: the arguments of one frame (select, readout, commit)."""
    _fields_ = [("read_masks", c_vp), ("X", c_vp), ("x_obj_stride", c_i64), ("k", c_vp), ("params", SelectParams),
                ("sel_idx", c_vp), ("sel_count", c_vp), ("prior_out", c_vp), ("max_sel", c_i32),
                ("n_splits", c_i32), ("Y", c_vp), ("y_obj_stride", c_i64), ("y_fp32", c_i32), ("Kmem", c_vp),
                ("Vmem", c_vp), ("kv_obj_stride", c_i64), ("commit_masks", c_vp), ("t", c_i32), ("pin", c_i32),
                ("fall_min", c_i32), ("fall_max", c_i32), ("kept_count", c_vp)]


class StackWeights(ctypes.Structure):
    """rs3_stack_weights: one layer's host arrays (see rs3.h)."""
    _fields_ = [(n, c_vp) for n in ("ln1_g", "ln1_b", "Wqs", "Wks", "Wvs", "Wos", "ln2_g", "ln2_b", "Wq", "Wk",
                                    "Wv", "Wo", "ln3_g", "ln3_b", "W1", "W2")]


class Rs3Error(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__("%s failed: %s (%d)" % (what, _status_str(status), status))


_SIGS = {
    "rs3_status_str": (ctypes.c_char_p, [c_i32]),
    "rs3_track_create": (c_i32, [c_i32, ctypes.POINTER(c_vp)]),
    "rs3_track_destroy": (None, [c_vp]),
    "rs3_track_export": (c_i32, [c_vp, c_vp]),
    "rs3_track_import": (c_i32, [c_vp, c_vp]),
    "rs3_layer_create": (c_i32, [c_i32, c_i32, c_i32, c_i32, c_i32, c_vp, c_vp, c_vp, c_vp, ctypes.POINTER(c_vp)]),
    "rs3_layer_destroy": (None, [c_vp]),
    "rs3_layer_set_rope": (c_i32, [c_vp, c_i32, c_i32, c_vp]),
    "rs3_layer_set_rope_axial": (c_i32, [c_vp, c_i32, c_i32, ctypes.c_double]),
    "rs3_bank_create": (c_i32, [c_vp, c_i32, c_i32, c_i32, ctypes.POINTER(c_vp)]),
    "rs3_bank_destroy": (None, [c_vp]),
    "rs3_bank_export": (c_i32, [c_vp, c_vp, c_vp, c_vp, c_vp, c_vp]),
    "rs3_bank_import": (c_i32, [c_vp, c_vp, c_vp, c_vp, c_vp, c_vp]),
    "rs3_attend_workspace_size": (c_i32, [c_i32, c_i32, c_i32, c_i32, c_i32, c_i32, ctypes.POINTER(c_sz)]),
    "rs3_attend": (c_i32, [c_vp, c_vp, c_vp, c_i32, c_i32, c_i32, c_i32, c_i32, c_i32, c_vp, c_vp, c_sz, c_vp]),
    "rs3_bank_error": (c_i32, [c_vp, c_vp, c_i32]),
    "rs3_select_workspace_size": (c_i32, [ctypes.POINTER(Grid), c_i32, c_i64, ctypes.POINTER(c_sz)]),
    "rs3_select_queries": (c_i32, [ctypes.POINTER(Grid), c_i32, c_vp, c_vp, c_vp, c_i64, c_i32, c_i32, c_vp,
                                   ctypes.POINTER(SelectParams), c_vp, c_sz, c_vp, c_vp, c_vp, c_vp]),
    "rs3_readout_workspace_size": (c_i32, [c_vp, c_i32, c_i32, c_i32, ctypes.POINTER(c_sz)]),
    "rs3_readout": (c_i32, [c_vp, ctypes.POINTER(Grid), c_i32, c_vp, c_i64, c_vp, c_vp, c_vp, c_i32, c_i32,
                            c_i32, c_vp, c_i64, c_i32, c_vp, c_sz, c_vp]),
    "rs3_readout_noalloc": (c_i32, [c_vp, ctypes.POINTER(Grid), c_i32, c_vp, c_i64, c_vp, c_vp, c_vp, c_i32, c_i32,
                                    c_i32, c_vp, c_i64, c_i32, c_vp]),
    "rs3_readout_commit": (c_i32, [c_vp, ctypes.POINTER(Grid), c_i32, c_vp, c_i64, c_vp, c_vp, c_vp, c_i32, c_i32,
                                   c_i32, c_vp, c_i64, c_i32, c_vp, c_sz, c_vp, c_vp, c_i64, c_vp, c_i32, c_i32,
                                   c_i32, c_i32, c_vp, c_vp]),
    "rs3_commit": (c_i32, [c_vp, c_i32, ctypes.POINTER(Grid), c_vp, c_vp, c_i64, c_vp, c_i32, c_i32, c_i32,
                           c_i32, c_vp, c_vp]),
    "rs3_frame_workspace_size": (c_i32, [c_vp, ctypes.POINTER(Grid), c_i32, c_i64, c_i32, c_i32,
                                         ctypes.POINTER(c_sz)]),
    "rs3_frame": (c_i32, [c_vp, ctypes.POINTER(Grid), c_i32, c_vp, c_vp, ctypes.POINTER(FrameIO), c_vp, c_sz, c_vp]),
    "rs3_write_keepset": (c_i32, [ctypes.POINTER(Grid), c_i32, c_vp, c_i32, c_i32, c_i32, c_i32, c_vp, c_vp, c_vp]),
    "rs3_close_workspace_size": (c_i32, [c_i32, c_i32, c_i32, ctypes.POINTER(c_sz)]),
    "rs3_close_masks": (c_i32, [c_i32, c_i32, c_i32, c_vp, c_i32, c_i32, c_vp, c_vp, c_vp, c_sz, c_vp]),
    "rs3_stack_create": (c_i32, [c_i32, c_i32, c_i32, c_i32, c_i32, c_i32, ctypes.POINTER(StackWeights),
                                 ctypes.POINTER(c_vp)]),
    "rs3_stack_destroy": (None, [c_vp]),
    "rs3_stack_workspace_size": (c_i32, [c_vp, c_i32, c_i32, ctypes.POINTER(c_sz)]),
    "rs3_stack_readout": (c_i32, [c_vp, ctypes.POINTER(Grid), c_vp, c_vp, c_vp, c_vp, c_i32, c_i32, c_vp, c_i32,
                                  c_vp, c_sz, c_vp]),
    "rs3_profile_enable": (c_i32, [c_i32, c_i32]),
    "rs3_profile_report": (c_i32, [c_vp, c_vp, c_vp]),
    "rs3_profile_reset": (c_i32, []),
    "rs3_stream_read": (c_i32, [c_vp, c_sz, c_vp, c_vp]),
}

RS3_STREAM_READ_THREADS = 1024 * 256

KERNEL_NAMES = ["energy", "select", "commit", "commit_append", "copy", "qproj", "attn", "combine",
                "readout_f32", "merge_commit", "stack_gemm", "stack_merge", "stack_mlp", "stack_rows"]

_lib = None


def lib():
    """Load librs3.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(lib_path):
            raise RuntimeError("librs3.so is not built; run `python -m paper_2608_22526_amd.build`")
        L = ctypes.CDLL(lib_path)
        for name, (res, args) in _SIGS.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def exported_symbols():
    return list(_SIGS)


def _status_str(s: int) -> str:
    try:
        return lib().rs3_status_str(int(s)).decode()
    except Exception:  # library not loadable
        return "status"


def _check(status: int, what: str):
    if status != RS3_OK:
        raise Rs3Error(status, what)


def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    if isinstance(t, np.ndarray):
        return t.ctypes.data
    return t.data_ptr()


def _stream(stream):
    if stream is not None:
        return stream
    import torch
    return torch.cuda.current_stream().cuda_stream


# ---------------------------------------------------------------------------
class Track:
    """rs3_track: per-object (box, streak, has_box) state."""

    def __init__(self, n_obj: int):
        h = c_vp()
        _check(lib().rs3_track_create(n_obj, ctypes.byref(h)), "rs3_track_create")
        self.h, self.n_obj = h, n_obj

    def export(self) -> np.ndarray:
        out = np.zeros((self.n_obj, RS3_TRACK_WORDS), np.int32)
        _check(lib().rs3_track_export(self.h, out.ctypes.data), "rs3_track_export")
        return out

    def import_(self, state: np.ndarray):
        st = np.ascontiguousarray(state, dtype=np.int32)
        _check(lib().rs3_track_import(self.h, st.ctypes.data), "rs3_track_import")

    def __del__(self):
        if getattr(self, "h", None) and _lib is not None:
            _lib.rs3_track_destroy(self.h)
            self.h = None


class Layer:
    """rs3_layer: W_q [C][D], W_k/W_v [d_kv][D], W_o [D][C] host arrays
    (uint16 bf16 bits or float32).  absorb=True runs the single-head
    attention on the raw bank rows (see rs3.h)."""

    def __init__(self, C: int, H: int, d_kv: int, dtype: int, Wq, Wk, Wv, Wo, absorb: bool = False):
        arrs = [np.ascontiguousarray(w) for w in (Wq, Wk, Wv, Wo)]
        h = c_vp()
        _check(lib().rs3_layer_create(C, H, d_kv, dtype, int(absorb), *(a.ctypes.data for a in arrs),
                                      ctypes.byref(h)), "rs3_layer_create")
        self.h, self.C, self.H, self.d_kv, self.dtype, self.absorb = h, C, H, d_kv, dtype, bool(absorb)

    def set_rope(self, m: int, n: int, table=None):
        """Attach a rotary table: float32 host array [m*n][d_h/2][2] of
        (cos, sin) pairs; table=None with m = n = 0 removes it."""
        t = None if table is None else np.ascontiguousarray(table, dtype=np.float32)
        _check(lib().rs3_layer_set_rope(self.h, m, n, None if t is None else t.ctypes.data), "rs3_layer_set_rope")

    def set_rope_axial(self, m: int, n: int, theta: float):
        """Attach the axial rotary table built on the device."""
        _check(lib().rs3_layer_set_rope_axial(self.h, m, n, float(theta)), "rs3_layer_set_rope_axial")

    def __del__(self):
        if getattr(self, "h", None) and _lib is not None:
            _lib.rs3_layer_destroy(self.h)
            self.h = None


class Bank:
    """rs3_bank: one object's ring bank for `layer`."""

    def __init__(self, layer: Layer, cap: int, f_max: int, n_pin: int):
        h = c_vp()
        _check(lib().rs3_bank_create(layer.h, cap, f_max, n_pin, ctypes.byref(h)), "rs3_bank_create")
        self.h, self.layer, self.cap, self.f_max, self.n_pin = h, layer, cap, f_max, n_pin

    def export(self):
        es = 2 if self.layer.dtype == RS3_BF16 else 4
        npdt = np.uint16 if es == 2 else np.float32
        hdr = np.zeros(RS3_BANK_HDR_WORDS, np.int32)
        frames = np.zeros((self.f_max, 4), np.int32)
        K = np.zeros((self.cap, self.layer.d_kv), npdt)
        V = np.zeros((self.cap, self.layer.d_kv), npdt)
        pos = np.zeros(self.cap, np.int32)
        _check(lib().rs3_bank_export(self.h, hdr.ctypes.data, frames.ctypes.data, K.ctypes.data,
                                     V.ctypes.data, pos.ctypes.data), "rs3_bank_export")
        nf, nk = int(hdr[0]), int(hdr[3])
        return dict(hdr=hdr, n_frames=nf, pin_end=int(hdr[1]), err=int(hdr[2]), n_keys=nk,
                    frames=frames[:nf].copy(), K=K[:nk].copy(), V=V[:nk].copy(), pos=pos[:nk].copy())

    def import_snapshot(self, snap: dict):
        """Restore from a dict in the format of export() (synchronises)."""
        es = 2 if self.layer.dtype == RS3_BF16 else 4
        npdt = np.uint16 if es == 2 else np.float32
        hdr = np.ascontiguousarray(snap["hdr"], dtype=np.int32)
        frames = np.ascontiguousarray(snap["frames"], dtype=np.int32).reshape(-1, 4)
        K = np.ascontiguousarray(snap["K"], dtype=npdt)
        V = np.ascontiguousarray(snap["V"], dtype=npdt)
        pos = np.ascontiguousarray(snap["pos"], dtype=np.int32)
        _check(lib().rs3_bank_import(self.h, hdr.ctypes.data, frames.ctypes.data, K.ctypes.data, V.ctypes.data,
                                     pos.ctypes.data), "rs3_bank_import")

    def info(self) -> dict:
        """Header only (n_frames, pin_end, err, n_keys); synchronises."""
        hdr = np.zeros(RS3_BANK_HDR_WORDS, np.int32)
        _check(lib().rs3_bank_export(self.h, hdr.ctypes.data, None, None, None, None), "rs3_bank_export")
        return dict(n_frames=int(hdr[0]), pin_end=int(hdr[1]), err=int(hdr[2]), n_keys=int(hdr[3]))

    def error(self, clear: bool = False) -> int:
        e = np.zeros(1, np.int32)
        _check(lib().rs3_bank_error(self.h, e.ctypes.data, int(clear)), "rs3_bank_error")
        return int(e[0])

    def __del__(self):
        if getattr(self, "h", None) and _lib is not None:
            _lib.rs3_bank_destroy(self.h)
            self.h = None


def _grid(g) -> Grid:
    if isinstance(g, Grid):
        return g
    m, n, s = g
    return Grid(m, n, s)


def select_workspace_size(grid, n_obj: int, x_obj_stride: int) -> int:
    out = c_sz()
    _check(lib().rs3_select_workspace_size(ctypes.byref(_grid(grid)), n_obj, x_obj_stride, ctypes.byref(out)),
           "rs3_select_workspace_size")
    return out.value


def select_queries(grid, n_obj: int, masks, track: Track, X, x_obj_stride: int, C: int, dtype: int,
                   k: Sequence[int], params: SelectParams, ws, sel_idx, sel_count, prior_out=None,
                   stream=None):
    karr = np.ascontiguousarray(np.asarray(k, dtype=np.int32))
    _check(lib().rs3_select_queries(ctypes.byref(_grid(grid)), n_obj, _ptr(masks), track.h, _ptr(X),
                                    x_obj_stride, C, dtype, karr.ctypes.data, ctypes.byref(params), _ptr(ws),
                                    ws.numel() * ws.element_size(), _ptr(sel_idx), _ptr(sel_count),
                                    _ptr(prior_out), _stream(stream)), "rs3_select_queries")


def readout_workspace_size(layer: Layer, n_obj: int, max_sel: int, n_splits: int = 0) -> int:
    out = c_sz()
    _check(lib().rs3_readout_workspace_size(layer.h, n_obj, max_sel, n_splits, ctypes.byref(out)),
           "rs3_readout_workspace_size")
    return out.value


def readout(layer: Layer, grid, n_obj: int, X, x_obj_stride: int, banks: Sequence[Bank], sel_idx, sel_count,
            sel_stride: int, max_sel: int, n_splits: int, Y, y_obj_stride: int, y_fp32: int = 0, ws=None,
            stream=None):
    harr = (c_vp * len(banks))(*[b.h for b in banks])
    ws_bytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check(lib().rs3_readout(layer.h, ctypes.byref(_grid(grid)), n_obj, _ptr(X), x_obj_stride,
                             ctypes.cast(harr, c_vp), _ptr(sel_idx), _ptr(sel_count), sel_stride, max_sel,
                             n_splits, _ptr(Y), y_obj_stride, y_fp32, _ptr(ws), ws_bytes, _stream(stream)),
           "rs3_readout")


def readout_noalloc(layer: Layer, grid, n_obj: int, X, x_obj_stride: int, banks: Sequence[Bank], sel_idx, sel_count,
                    sel_stride: int, max_sel: int, n_splits: int, Y, y_obj_stride: int, y_fp32: int = 0, stream=None):
    """rs3_readout without a workspace: the library's fixed per-GPU scratch
    holds the split partials (nothing is allocated)."""
    harr = (c_vp * len(banks))(*[b.h for b in banks])
    _check(lib().rs3_readout_noalloc(layer.h, ctypes.byref(_grid(grid)), n_obj, _ptr(X), x_obj_stride,
                                     ctypes.cast(harr, c_vp), _ptr(sel_idx), _ptr(sel_count), sel_stride, max_sel,
                                     n_splits, _ptr(Y), y_obj_stride, y_fp32, _stream(stream)), "rs3_readout_noalloc")


def commit(banks: Sequence[Bank], grid, Kmem, Vmem, kv_obj_stride: int, masks, t: int, pin: int,
           fall_min: int, fall_max: int, kept_count=None, stream=None):
    harr = (c_vp * len(banks))(*[b.h for b in banks])
    _check(lib().rs3_commit(ctypes.cast(harr, c_vp), len(banks), ctypes.byref(_grid(grid)), _ptr(Kmem),
                            _ptr(Vmem), kv_obj_stride, _ptr(masks), t, pin, fall_min, fall_max,
                            _ptr(kept_count), _stream(stream)), "rs3_commit")


def readout_commit(layer: Layer, grid, n_obj: int, X, x_obj_stride: int, banks: Sequence[Bank], sel_idx, sel_count,
                   sel_stride: int, max_sel: int, n_splits: int, Y, y_obj_stride: int, y_fp32: int, ws, Kmem, Vmem,
                   kv_obj_stride: int, masks, t: int, pin: int, fall_min: int, fall_max: int, kept_count=None,
                   stream=None):
    """rs3_readout followed by rs3_commit, merged into fewer launches."""
    harr = (c_vp * len(banks))(*[b.h for b in banks])
    ws_bytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check(lib().rs3_readout_commit(layer.h, ctypes.byref(_grid(grid)), n_obj, _ptr(X), x_obj_stride,
                                    ctypes.cast(harr, c_vp), _ptr(sel_idx), _ptr(sel_count), sel_stride, max_sel,
                                    n_splits, _ptr(Y), y_obj_stride, y_fp32, _ptr(ws), ws_bytes, _ptr(Kmem),
                                    _ptr(Vmem), kv_obj_stride, _ptr(masks), t, pin, fall_min, fall_max,
                                    _ptr(kept_count), _stream(stream)), "rs3_readout_commit")


def frame_workspace_size(layer: Layer, grid, n_obj: int, x_obj_stride: int, max_sel: int, n_splits: int = 0) -> int:
    out = c_sz()
    _check(lib().rs3_frame_workspace_size(layer.h, ctypes.byref(_grid(grid)), n_obj, x_obj_stride, max_sel, n_splits,
                                          ctypes.byref(out)), "rs3_frame_workspace_size")
    return out.value


def frame(layer: Layer, grid, n_obj: int, track: Track, banks: Sequence[Bank], io: FrameIO, ws, stream=None):
    """One frame: rs3_select_queries then rs3_readout_commit in one call
    (`io` holds the arguments of both)."""
    harr = (c_vp * len(banks))(*[b.h for b in banks])
    _check(lib().rs3_frame(layer.h, ctypes.byref(_grid(grid)), n_obj, track.h, ctypes.cast(harr, c_vp),
                           ctypes.byref(io), _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)), "rs3_frame")


def write_keepset(grid, n_obj: int, seed_masks, D_w: int, fall_min: int, fall_max: int, n_copies: int, keep,
                  counts=None, stream=None):
    """The fixed write keep-set K_w (u8 [n_copies][m*n]) from the seed masks."""
    _check(lib().rs3_write_keepset(ctypes.byref(_grid(grid)), n_obj, _ptr(seed_masks), D_w, fall_min, fall_max,
                                   n_copies, _ptr(keep), _ptr(counts), _stream(stream)), "rs3_write_keepset")


def close_workspace_size(n_obj: int, H: int, W: int) -> int:
    out = c_sz()
    _check(lib().rs3_close_workspace_size(n_obj, H, W, ctypes.byref(out)), "rs3_close_workspace_size")
    return out.value


def close_masks(n_obj: int, H: int, W: int, logits, dtype: int, k: int, closed=None, palette=None, ws=None,
                stream=None):
    """k x k closure of each object's decoded mask and the palette argmax."""
    ws_bytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check(lib().rs3_close_masks(n_obj, H, W, _ptr(logits), dtype, k, _ptr(closed), _ptr(palette), _ptr(ws),
                                 ws_bytes, _stream(stream)), "rs3_close_masks")


def attend_workspace_size(n_q: int, n_kv: int, H: int, d_h: int, dtype: int, n_splits: int = 0) -> int:
    out = c_sz()
    _check(lib().rs3_attend_workspace_size(n_q, n_kv, H, d_h, dtype, n_splits, ctypes.byref(out)),
           "rs3_attend_workspace_size")
    return out.value


def attend(Q, K, V, n_q: int, n_kv: int, H: int, d_h: int, dtype: int, O, ws=None, n_splits: int = 0,
           stream=None):
    """Bare attention core: O [n_q][H*d_h] fp32 from projected Q, K, V."""
    ws_bytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check(lib().rs3_attend(_ptr(Q), _ptr(K), _ptr(V), n_q, n_kv, H, d_h, dtype, n_splits, _ptr(O), _ptr(ws),
                            ws_bytes, _stream(stream)), "rs3_attend")


class Stack:
    """rs3_stack: the L-layer memory-attention stack on the kept queries.
    layers: one dict per layer with the keys of StackWeights (matrices uint16
    bf16 bits, row-major input dimension first; norm gains/shifts float32)."""

    def __init__(self, layers: Sequence[dict], C: int = 256, H_s: int = 1, d_kv: int = 64, F: int = 2048,
                 dtype: int = RS3_BF16):
        keep = []
        arr = (StackWeights * len(layers))()
        for i, w in enumerate(layers):
            for name, _ in StackWeights._fields_:
                a = np.ascontiguousarray(w[name], dtype=np.float32 if name.startswith("ln") else np.uint16)
                keep.append(a)
                setattr(arr[i], name, a.ctypes.data)
        h = c_vp()
        _check(lib().rs3_stack_create(len(layers), C, H_s, d_kv, F, dtype, arr, ctypes.byref(h)), "rs3_stack_create")
        self.h, self.n_layers, self.C, self.H_s, self.d_kv, self.F = h, len(layers), C, H_s, d_kv, F

    def workspace_size(self, max_sel: int, n_splits: int = 0) -> int:
        out = c_sz()
        _check(lib().rs3_stack_workspace_size(self.h, max_sel, n_splits, ctypes.byref(out)),
               "rs3_stack_workspace_size")
        return out.value

    def readout(self, grid, X, bank: Bank, sel_idx, sel_count, max_sel: int, Y, y_fp32: int = 0, ws=None,
                n_splits: int = 0, stream=None):
        ws_bytes = 0 if ws is None else ws.numel() * ws.element_size()
        _check(lib().rs3_stack_readout(self.h, ctypes.byref(_grid(grid)), _ptr(X), bank.h, _ptr(sel_idx),
                                       _ptr(sel_count), max_sel, n_splits, _ptr(Y), y_fp32, _ptr(ws), ws_bytes,
                                       _stream(stream)), "rs3_stack_readout")

    def __del__(self):
        if getattr(self, "h", None) and _lib is not None:
            _lib.rs3_stack_destroy(self.h)
            self.h = None


def profile_enable(on: bool, max_launches: int = 65536):
    _check(lib().rs3_profile_enable(int(on), max_launches), "rs3_profile_enable")


def profile_reset():
    _check(lib().rs3_profile_reset(), "rs3_profile_reset")


def stream_read(src, nbytes: int, out, stream=None):
    """rs3_stream_read: reads nbytes of device memory at src once; out
    (RS3_STREAM_READ_THREADS uint32) receives one xor word per thread."""
    _check(lib().rs3_stream_read(_ptr(src), nbytes, _ptr(out), _stream(stream)), "rs3_stream_read")


def profile_report() -> dict:
    """{kernel name: (total ms, launches)} accumulated since the last reset."""
    n = len(KERNEL_NAMES)
    ms = np.zeros(n, np.float64)
    cnt = np.zeros(n, np.int64)
    dropped = np.zeros(1, np.int64)
    _check(lib().rs3_profile_report(ms.ctypes.data, cnt.ctypes.data, dropped.ctypes.data), "rs3_profile_report")
    out = {KERNEL_NAMES[i]: (float(ms[i]), int(cnt[i])) for i in range(n)}
    out["_dropped"] = (0.0, int(dropped[0]))
    return out
