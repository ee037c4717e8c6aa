"""Write-side compaction and the ring memory bank (test infrastructure).

Sec. 3.2 admits into the bank only the memory-encoder tokens of the kept write
set (Eq. 8; Algorithm 1, sparse write): each stored frame holds |K_w| tokens
instead of mn, and the bank grows by that many rows per commit.  On the rare
frames whose footprint covers more than 95% or less than 5% of the grid the
write falls through to the original dense path.

Readings (the paper only says the rows are appended):
  * `compact` keeps the cells set in the mask passed in, ascending; the
    fall-through is expressed with integer thresholds (count < fall_min or
    count > fall_max -> keep all mn cells), computed exactly by the caller;
  * the bank has `cap` token rows and at most `f_max` frames; the first
    commits may be pinned (at most n_pin, all before any unpinned one): they
    are laid out from row 0 and never evicted; pin_end = their total length;
  * an unpinned frame of length L is placed as follows:
      1. L > cap - pin_end  -> capacity error, the bank is unchanged;
      2. while the bank holds f_max frames, evict the oldest unpinned frame;
      3. start = end of the newest unpinned frame (pin_end if none);
         if start + L > cap, start = pin_end (frames are never split);
      4. evict unpinned frames oldest first until none intersects
         [start, start + L);
      5. write the rows and record (start, L, t, pinned);
  * zero-length frames are recorded as frames;
  * key order for the readout: pinned frames, then unpinned oldest to newest;
  * the error word keeps the first error; a failing commit changes nothing.
`FrameListBank` is an independent model of the same rule without offsets,
used to cross-check which frames are resident.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import List, Optional

import numpy as np

RS3_OK, RS3_E_INVALID, RS3_E_CAPACITY = 0, 1, 2


def compact(mask: np.ndarray, fall_min: int = 0, fall_max: Optional[int] = None) -> np.ndarray:
    """Ascending list of set cells; all cells when the count falls outside
    [fall_min, fall_max]."""
    flat = np.asarray(mask).reshape(-1)
    mn = flat.shape[0]
    kept = [i for i in range(mn) if flat[i] != 0]
    if fall_max is None:
        fall_max = mn
    if len(kept) < fall_min or len(kept) > fall_max:
        kept = list(range(mn))
    return np.asarray(kept, dtype=np.int32)


@dataclass
class Frame:
    start: int
    length: int
    t: int
    pinned: int


class RingBank:
    """Offset-level model of one object's ring bank."""

    def __init__(self, cap: int, f_max: int, n_pin: int, d_kv: int, dtype):
        if cap <= 0 or f_max < 1 or not (0 <= n_pin < f_max):
            raise ValueError("invalid bank shape")
        self.cap, self.f_max, self.n_pin = cap, f_max, n_pin
        self.K = np.zeros((cap, d_kv), dtype=dtype)
        self.V = np.zeros((cap, d_kv), dtype=dtype)
        self.pos = np.zeros(cap, dtype=np.int32)
        self.frames: List[Frame] = []
        self.pin_end = 0
        self.err = RS3_OK
        self.pin_calls = 0
        self.unpinned_seen = False

    # -- placement -----------------------------------------------------------
    def _fail(self, code: int):
        if self.err == RS3_OK:
            self.err = code

    def _evict_oldest_unpinned(self):
        for idx, f in enumerate(self.frames):
            if not f.pinned:
                del self.frames[idx]
                return
        raise AssertionError("no unpinned frame to evict")

    @staticmethod
    def _overlaps(f: Frame, start: int, L: int) -> bool:
        return f.length > 0 and L > 0 and f.start < start + L and start < f.start + f.length

    def commit(self, Ksrc, Vsrc, mask, t: int, pin: bool, fall_min: int = 0,
               fall_max: Optional[int] = None) -> int:
        """Append one frame's kept rows.  Returns the kept count.  Raises
        ValueError for misuse that the host rejects before any device work."""
        if pin:
            if self.unpinned_seen or self.pin_calls >= self.n_pin:
                raise ValueError("pinned commit after an unpinned one or beyond n_pin")
            self.pin_calls += 1
        else:
            self.unpinned_seen = True
        kept = compact(mask, fall_min, fall_max)
        L = int(kept.shape[0])
        if pin:
            if self.pin_end + L > self.cap:
                self._fail(RS3_E_CAPACITY)
                return L
            start = self.pin_end
            self.pin_end += L
        else:
            if L > self.cap - self.pin_end:
                self._fail(RS3_E_CAPACITY)
                return L
            while len(self.frames) >= self.f_max:
                self._evict_oldest_unpinned()
            unpinned = [f for f in self.frames if not f.pinned]
            start = (unpinned[-1].start + unpinned[-1].length) if unpinned else self.pin_end
            if start + L > self.cap:
                start = self.pin_end
            while any((not f.pinned) and self._overlaps(f, start, L) for f in self.frames):
                self._evict_oldest_unpinned()
        self.K[start:start + L] = np.asarray(Ksrc)[kept]
        self.V[start:start + L] = np.asarray(Vsrc)[kept]
        self.pos[start:start + L] = kept
        self.frames.append(Frame(start, L, int(t), int(bool(pin))))
        return L

    # -- views ---------------------------------------------------------------
    def frame_table(self) -> np.ndarray:
        return np.asarray([[f.start, f.length, f.t, f.pinned] for f in self.frames],
                          dtype=np.int32).reshape(-1, 4)

    def header(self):
        return [len(self.frames), self.pin_end, self.err]

    def key_rows(self):
        """Resident rows (K, V, pos) concatenated in key order."""
        if not self.frames:
            d = self.K.shape[1]
            return (np.zeros((0, d), self.K.dtype), np.zeros((0, d), self.V.dtype),
                    np.zeros(0, np.int32))
        ks = [self.K[f.start:f.start + f.length] for f in self.frames]
        vs = [self.V[f.start:f.start + f.length] for f in self.frames]
        ps = [self.pos[f.start:f.start + f.length] for f in self.frames]
        return np.concatenate(ks), np.concatenate(vs), np.concatenate(ps)


class FrameListBank:
    """List-of-frames model: pinned frames plus a FIFO of unpinned frames
    bounded only by f_max (no offsets, no capacity)."""

    def __init__(self, f_max: int, n_pin: int):
        self.f_max, self.n_pin = f_max, n_pin
        self.frames = []   # (t, pinned, K rows, V rows, pos)

    def commit(self, Ksrc, Vsrc, mask, t: int, pin: bool, fall_min=0, fall_max=None):
        kept = compact(mask, fall_min, fall_max)
        if not pin:
            while len(self.frames) >= self.f_max:
                for idx, f in enumerate(self.frames):
                    if not f[1]:
                        del self.frames[idx]
                        break
        self.frames.append((int(t), int(bool(pin)), np.asarray(Ksrc)[kept],
                            np.asarray(Vsrc)[kept], kept))
        return int(kept.shape[0])

    def resident_times(self):
        return [f[0] for f in self.frames]
