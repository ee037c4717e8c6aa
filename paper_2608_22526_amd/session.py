"""Convenience owner of the handles and device buffers for one stream of
frames (argument marshalling only; all work runs in librs3.so).

The per-frame calls keep their argument objects (grid and parameter structs,
the bank handle array, the keep-budget array and the bound C functions)
across calls, so that a frame costs the host two foreign calls and little
else."""
from __future__ import annotations

import ctypes
from typing import Optional, Sequence

import numpy as np

from . import _binding as B


def to_device(a: np.ndarray, device="cuda"):
    """Host array -> torch tensor on the GPU.  uint16 arrays are bf16 bits."""
    import torch
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).to(device).view(torch.bfloat16)
    return torch.from_numpy(a).to(device)


def to_host(t) -> np.ndarray:
    """torch tensor -> numpy (bf16 -> uint16 bits)."""
    import torch
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return t.cpu().numpy()


class Session:
    def __init__(self, *, m: int, n: int, s: int, C: int, H: int, d_kv: int, dtype: str, n_obj: int,
                 shared_x: bool, union_objects: bool, cap: int, f_max: int, n_pin: int, weights,
                 r_s: int = 4, c: int = 14, max_sel: Optional[int] = None, n_splits: int = 0,
                 absorb: bool = False, rope_theta: Optional[float] = None, rope_table=None,
                 device: str = "cuda"):
        import torch
        self.torch = torch
        self.m, self.n, self.s, self.mn = m, n, s, m * n
        self.C, self.H, self.d_kv = C, H, d_kv
        self.dt = B.RS3_BF16 if dtype == "bf16" else B.RS3_F32
        self.n_obj, self.shared_x, self.union_objects = n_obj, shared_x, union_objects
        self.n_groups = 1 if union_objects else n_obj
        self.grid = B.Grid(m, n, s)
        self.params = B.SelectParams(r_s, c, 0, 1 if union_objects else 0)
        self.layer = B.Layer(C, H, d_kv, self.dt, weights.Wq, weights.Wk, weights.Wv, weights.Wo, absorb)
        if rope_table is not None:
            self.layer.set_rope(m, n, rope_table)
        elif rope_theta is not None:
            self.layer.set_rope_axial(m, n, rope_theta)
        self.banks = [B.Bank(self.layer, cap, f_max, n_pin) for _ in range(n_obj)]
        self.track = B.Track(n_obj)
        self.device = device
        self.x_stride = 0 if shared_x else self.mn * C
        self.max_sel = self.mn if max_sel is None else max_sel
        self.n_splits = n_splits
        i32 = torch.int32
        self.sel_idx = torch.zeros((self.n_groups, self.mn), dtype=i32, device=device)
        self.sel_count = torch.zeros(self.n_groups, dtype=i32, device=device)
        self.kept_count = torch.zeros(n_obj, dtype=i32, device=device)
        ws = B.select_workspace_size(self.grid, n_obj, self.x_stride)
        self.ws_sel = torch.zeros(max(ws, 8), dtype=torch.uint8, device=device)
        wr = B.readout_workspace_size(self.layer, n_obj, self.max_sel, n_splits)
        self.ws_read = torch.zeros(max(wr, 256), dtype=torch.uint8, device=device)
        wf = B.frame_workspace_size(self.layer, self.grid, n_obj, self.x_stride, self.max_sel, n_splits)
        self.ws_frame = torch.zeros(max(wf, 256), dtype=torch.uint8, device=device)
        # argument objects reused by every call
        L = B.lib()
        self._f_select, self._f_readout = L.rs3_select_queries, L.rs3_readout
        self._f_commit, self._f_readout_commit = L.rs3_commit, L.rs3_readout_commit
        self._f_frame = L.rs3_frame
        self._io = B.FrameIO()
        self._io_ref = ctypes.byref(self._io)
        self._grid_ref = ctypes.byref(self.grid)
        self._params_ref = ctypes.byref(self.params)
        self._harr_src = None
        self._k = (ctypes.c_int32 * self.n_groups)()
        self._k_addr = ctypes.addressof(self._k)
        self._ws_sel = (self.ws_sel.data_ptr(), self.ws_sel.numel())
        self._ws_read = (self.ws_read.data_ptr(), self.ws_read.numel())
        self._ws_frame = (self.ws_frame.data_ptr(), self.ws_frame.numel())
        io = self._io
        io.x_obj_stride, io.k, io.params = self.x_stride, self._k_addr, self.params
        io.sel_idx, io.sel_count = self.sel_idx.data_ptr(), self.sel_count.data_ptr()
        io.n_splits, io.y_obj_stride = n_splits, self.mn * C if n_obj > 1 else 0
        io.kv_obj_stride, io.kept_count = self.mn * d_kv, self.kept_count.data_ptr()
        self._p_sel_idx, self._p_sel_count = self.sel_idx.data_ptr(), self.sel_count.data_ptr()
        self._p_kept = self.kept_count.data_ptr()
        self._sel_stride = 0 if union_objects else self.mn
        self._y_stride = self.mn * C if n_obj > 1 else 0
        self._dev_index = torch.device(device).index or 0
        raw = getattr(torch._C, "_cuda_getCurrentRawStream", None)
        self._raw_stream = (lambda: raw(self._dev_index)) if raw is not None else \
            (lambda: torch.cuda.current_stream().cuda_stream)

    def _handles(self):
        """Device address of the bank handle array, rebuilt when the bank
        list has changed (a bank replaced by a restored one, say)."""
        if self.banks != self._harr_src:
            self._harr_keep = (B.c_vp * len(self.banks))(*[b.h for b in self.banks])
            self._harr = ctypes.cast(self._harr_keep, B.c_vp).value
            self._harr_src = list(self.banks)
        return self._harr

    def _stream(self, stream):
        return self._raw_stream() if stream is None else stream

    @staticmethod
    def _check(status, what):
        if status != B.RS3_OK:
            raise B.Rs3Error(status, what)

    # -- calls ---------------------------------------------------------------
    def select(self, masks, X, k: Sequence[int], seed_box: bool = False, prior_out=None, stream=None):
        if len(k) != self.n_groups:
            raise ValueError("select: %d keep budgets for %d groups" % (len(k), self.n_groups))
        self.params.seed_box = 1 if seed_box else 0
        kk = self._k
        for i, v in enumerate(k):
            kk[i] = v
        self._check(self._f_select(self._grid_ref, self.n_obj, masks.data_ptr(), self.track.h, X.data_ptr(),
                                   self.x_stride, self.C, self.dt, self._k_addr, self._params_ref, self._ws_sel[0],
                                   self._ws_sel[1], self._p_sel_idx, self._p_sel_count,
                                   None if prior_out is None else prior_out.data_ptr(), self._stream(stream)),
                    "rs3_select_queries")

    def readout(self, X, Y, max_sel: Optional[int] = None, y_fp32: int = 0, stream=None):
        ms = self.max_sel if max_sel is None else max_sel
        self._check(self._f_readout(self.layer.h, self._grid_ref, self.n_obj, X.data_ptr(), self.x_stride,
                                    self._handles(), self._p_sel_idx, self._p_sel_count, self._sel_stride, ms,
                                    self.n_splits, Y.data_ptr(), self._y_stride, y_fp32, self._ws_read[0],
                                    self._ws_read[1], self._stream(stream)), "rs3_readout")

    def readout_commit(self, X, Y, Kmem, Vmem, masks, t: int, pin: bool, max_sel: Optional[int] = None,
                       y_fp32: int = 0, fall_min: int = 0, fall_max: Optional[int] = None, stream=None):
        """readout(X, Y) then commit(Kmem, Vmem, masks, t, pin) in one call."""
        ms = self.max_sel if max_sel is None else max_sel
        fmax = self.mn if fall_max is None else fall_max
        self._check(self._f_readout_commit(
            self.layer.h, self._grid_ref, self.n_obj, X.data_ptr(), self.x_stride, self._handles(), self._p_sel_idx,
            self._p_sel_count, self._sel_stride, ms, self.n_splits, Y.data_ptr(), self._y_stride, y_fp32,
            self._ws_read[0], self._ws_read[1], Kmem.data_ptr(), Vmem.data_ptr(), self.mn * self.d_kv,
            masks.data_ptr(), t, int(pin), fall_min, fmax, self._p_kept, self._stream(stream)),
            "rs3_readout_commit")

    def frame(self, read_masks, X, k: Sequence[int], Y, Kmem, Vmem, commit_masks, t: int, pin: bool = False,
              max_sel: Optional[int] = None, y_fp32: int = 0, seed_box: bool = False, prior_out=None,
              fall_min: int = 0, fall_max: Optional[int] = None, stream=None):
        """select(read_masks, X, k), then readout_commit(X, Y, Kmem, Vmem,
        commit_masks, t, pin), as one rs3_frame call."""
        if len(k) != self.n_groups:
            raise ValueError("frame: %d keep budgets for %d groups" % (len(k), self.n_groups))
        kk = self._k
        for i, v in enumerate(k):
            kk[i] = v
        io = self._io
        io.params.seed_box = 1 if seed_box else 0
        io.read_masks, io.X, io.Y = read_masks.data_ptr(), X.data_ptr(), Y.data_ptr()
        io.prior_out = None if prior_out is None else prior_out.data_ptr()
        io.max_sel = self.max_sel if max_sel is None else max_sel
        io.y_fp32 = y_fp32
        io.Kmem, io.Vmem, io.commit_masks = Kmem.data_ptr(), Vmem.data_ptr(), commit_masks.data_ptr()
        io.t, io.pin, io.fall_min = t, int(pin), fall_min
        io.fall_max = self.mn if fall_max is None else fall_max
        self._check(self._f_frame(self.layer.h, self._grid_ref, self.n_obj, self.track.h, self._handles(),
                                  self._io_ref, self._ws_frame[0], self._ws_frame[1], self._stream(stream)),
                    "rs3_frame")

    def commit(self, Kmem, Vmem, masks, t: int, pin: bool, fall_min: int = 0, fall_max: Optional[int] = None,
               stream=None):
        fmax = self.mn if fall_max is None else fall_max
        self._check(self._f_commit(self._handles(), self.n_obj, self._grid_ref, Kmem.data_ptr(), Vmem.data_ptr(),
                                   self.mn * self.d_kv, masks.data_ptr(), t, int(pin), fall_min, fmax, self._p_kept,
                                   self._stream(stream)), "rs3_commit")
