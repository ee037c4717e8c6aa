#include "host_check.h"

namespace rs3host {

bool bank_snapshot_ok(int32_t cap, int32_t f_max, int32_t n_pin, const int32_t* hdr, const int32_t* frames,
                      bool have_rows, int32_t* n_pinned, bool* any_unpinned) {
  if (!hdr) return false;
  const int32_t nf = hdr[0], pin_end = hdr[1], keys = hdr[3];
  if (nf < 0 || nf > f_max || pin_end < 0 || pin_end > cap || keys < 0 || keys > cap) return false;
  if (nf > 0 && !frames) return false;
  if (keys > 0 && !have_rows) return false;
  int32_t pinned = 0;
  int64_t pinned_rows = 0, sum = 0;
  bool unpinned = false;
  for (int32_t f = 0; f < nf; ++f) {
    const int32_t st = frames[4 * f], len = frames[4 * f + 1], pin = frames[4 * f + 3];
    if (st < 0 || len < 0 || (int64_t)st + len > cap || (pin != 0 && pin != 1)) return false;
    if (pin) {
      if (unpinned || st != pinned_rows) return false;
      ++pinned;
      pinned_rows += len;
    } else {
      unpinned = true;
      if (len > 0 && st < pin_end) return false;
    }
    for (int32_t q = 0; q < f; ++q) {
      const int32_t qs = frames[4 * q], ql = frames[4 * q + 1];
      if (len > 0 && ql > 0 && (int64_t)qs < (int64_t)st + len && (int64_t)st < (int64_t)qs + ql) return false;
    }
    sum += len;
  }
  if (pinned > n_pin || pinned_rows != pin_end || sum != keys) return false;
  if (n_pinned) *n_pinned = pinned;
  if (any_unpinned) *any_unpinned = unpinned;
  return true;
}

bool track_state_ok(int32_t n_obj, const int32_t* state) {
  if (!state || n_obj < 0) return false;
  constexpr int32_t LIM = 1 << 30;
  for (int32_t o = 0; o < n_obj; ++o) {
    const int32_t* w = state + (int64_t)o * 6;
    const int32_t y0 = w[0], x0 = w[1], y1 = w[2], x1 = w[3], streak = w[4], has = w[5];
    if (has != 0 && has != 1) return false;
    if (streak < 0 || streak > LIM) return false;
    if (has) {
      if (y0 < 0 || x0 < 0 || y0 > y1 || x0 > x1 || y1 >= LIM || x1 >= LIM) return false;
    } else if (y0 != 0 || x0 != 0 || y1 != 0 || x1 != 0) {
      return false;
    }
  }
  return true;
}

}  // namespace rs3host
