// Host-side validation of caller-supplied state for the rs3 C ABI: plain
// C++ with no HIP dependency, so that it also builds and runs on its own
// (under the address and undefined-behaviour sanitizers in the CPU tests).
#pragma once

#include <stdint.h>

namespace rs3host {

// A bank snapshot as rs3_bank_import receives it: hdr[4] = {frames, pinned
// rows, error word, resident rows}, frames[4*nf] = {start, length, t,
// pinned} in key order.  Accepted only if it is a state the Eq. 8 ring
// placement can reach in a bank of `cap` rows, `f_max` frames and `n_pin`
// pinned frames: pinned frames first, packed from row 0; unpinned frames at
// or past the pinned rows; no two non-empty frames overlapping; lengths
// adding up to the resident rows; K, V and pos present when rows are.
// On success *n_pinned and *any_unpinned describe the frames.
bool bank_snapshot_ok(int32_t cap, int32_t f_max, int32_t n_pin, const int32_t* hdr, const int32_t* frames,
                      bool have_rows, int32_t* n_pinned, bool* any_unpinned);

// Tracker state as rs3_track_import receives it (n_obj x 6 words: y0, x0,
// y1, x1, streak, has_box): accepted only if every object's words are a
// state the tracker update reaches (has_box 0 or 1; streak in [0, 2^30];
// with a box, 0 <= y0 <= y1 < 2^30 and 0 <= x0 <= x1 < 2^30; without one,
// a zero box).
bool track_state_ok(int32_t n_obj, const int32_t* state);

}  // namespace rs3host
