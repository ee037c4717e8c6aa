"""Convenience owner of the handles and device buffers for one stream of
frames (argument marshalling only; all work runs in librs3.so)."""
from __future__ import annotations

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

    # -- calls ---------------------------------------------------------------
    def select(self, masks, X, k: Sequence[int], seed_box: bool = False, prior_out=None, stream=None):
        self.params.seed_box = 1 if seed_box else 0
        B.select_queries(self.grid, self.n_obj, masks, self.track, X, self.x_stride, self.C, self.dt, k,
                         self.params, self.ws_sel, self.sel_idx, self.sel_count, prior_out, stream)

    def readout(self, X, Y, max_sel: Optional[int] = None, y_fp32: int = 0, stream=None):
        ms = self.max_sel if max_sel is None else max_sel
        sel_stride = 0 if self.union_objects else self.mn
        y_stride = self.mn * self.C if self.n_obj > 1 else 0
        B.readout(self.layer, self.grid, self.n_obj, X, self.x_stride, self.banks, self.sel_idx, self.sel_count,
                  sel_stride, ms, self.n_splits, Y, y_stride, y_fp32, self.ws_read, stream)

    def readout_commit(self, X, Y, Kmem, Vmem, masks, t: int, pin: bool, max_sel: Optional[int] = None,
                       y_fp32: int = 0, fall_min: int = 0, fall_max: Optional[int] = None, stream=None):
        """readout(X, Y) then commit(Kmem, Vmem, masks, t, pin) in one call."""
        ms = self.max_sel if max_sel is None else max_sel
        sel_stride = 0 if self.union_objects else self.mn
        y_stride = self.mn * self.C if self.n_obj > 1 else 0
        fmax = self.mn if fall_max is None else fall_max
        B.readout_commit(self.layer, self.grid, self.n_obj, X, self.x_stride, self.banks, self.sel_idx,
                         self.sel_count, sel_stride, ms, self.n_splits, Y, y_stride, y_fp32, self.ws_read, Kmem,
                         Vmem, self.mn * self.d_kv, masks, t, int(pin), fall_min, fmax, self.kept_count, stream)

    def commit(self, Kmem, Vmem, masks, t: int, pin: bool, fall_min: int = 0, fall_max: Optional[int] = None,
               stream=None):
        fmax = self.mn if fall_max is None else fall_max
        B.commit(self.banks, self.grid, Kmem, Vmem, self.mn * self.d_kv, masks, t, int(pin), fall_min, fmax,
                 self.kept_count, stream)
