// CPU fuzz of the host validators of the rs3 C ABI (host_check.cpp), built
// with the address and undefined-behaviour sanitizers by
// tests/test_host_sanitize.py.
//
// Bank snapshots (rs3_bank_import, Eq. 8 ring state):
//  * states built by a plain model of the ring (pinned frames packed from
//    row 0, unpinned frames at free places past them) must be accepted;
//  * every accepted snapshot, valid or mutated, must satisfy the placement
//    invariants, checked here on an occupancy array row by row;
//  * malformed snapshots (random words, extreme values, frame counts past
//    the table) must be rejected without reading outside the buffers: the
//    frame table is allocated with exactly the entries the header names.
// Tracker states (rs3_track_import, Eq. 5): random and extreme words are
// accepted exactly when an independent check of the reachable states holds.
#include <limits.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

#include <vector>

#include "host_check.h"

static uint64_t rng_state = 0x9e3779b97f4a7c15ull;
static uint64_t next_u64() {   // xorshift64*
  rng_state ^= rng_state >> 12;
  rng_state ^= rng_state << 25;
  rng_state ^= rng_state >> 27;
  return rng_state * 0x2545f4914f6cdd1dull;
}
static int32_t uni(int32_t lo, int32_t hi) {   // [lo, hi]
  return lo + (int32_t)(next_u64() % (uint64_t)((int64_t)hi - lo + 1));
}
static int32_t extreme() {
  static const int32_t v[] = {INT_MIN, INT_MIN + 1, -65536, -2, -1, 0, 1, 2, 63, 64, 65, 4095, 4096,
                              (1 << 30) - 1, 1 << 30, (1 << 30) + 1, INT_MAX - 1, INT_MAX};
  return v[next_u64() % (sizeof(v) / sizeof(v[0]))];
}

static int failures = 0;
#define CHECK(c, ...)                   \
  do {                                  \
    if (!(c)) {                         \
      fprintf(stderr, __VA_ARGS__);     \
      fprintf(stderr, "\n");            \
      ++failures;                       \
    }                                   \
  } while (0)

// The placement invariants, row by row.
static bool invariants(int32_t cap, int32_t f_max, int32_t n_pin, const int32_t* hdr, const int32_t* frames,
                       bool have_rows) {
  const int32_t nf = hdr[0], pin_end = hdr[1], keys = hdr[3];
  if (nf < 0 || nf > f_max || pin_end < 0 || pin_end > cap || keys < 0 || keys > cap) return false;
  if (keys > 0 && !have_rows) return false;
  std::vector<char> used((size_t)cap, 0);
  int32_t pinned = 0;
  int64_t next_pinned_row = 0, total = 0;
  bool seen_unpinned = false;
  for (int32_t f = 0; f < nf; ++f) {
    const int64_t st = frames[4 * f], len = frames[4 * f + 1];
    const int32_t pin = frames[4 * f + 3];
    if (pin != 0 && pin != 1) return false;
    if (st < 0 || len < 0 || st + len > cap) return false;
    if (pin == 1) {
      if (seen_unpinned || st != next_pinned_row) return false;
      next_pinned_row += len;
      ++pinned;
    } else {
      seen_unpinned = true;
      if (len > 0 && st < pin_end) return false;
    }
    for (int64_t r = st; r < st + len; ++r) {
      if (used[(size_t)r]) return false;
      used[(size_t)r] = 1;
    }
    total += len;
  }
  return pinned <= n_pin && next_pinned_row == pin_end && total == keys;
}

struct Snap {
  int32_t cap, f_max, n_pin;
  int32_t hdr[4];
  std::vector<int32_t> frames;   // 4 per frame
};

// A reachable state: up to n_pin pinned frames from row 0, then unpinned
// frames placed in free gaps past the pinned rows.
static Snap build_valid() {
  Snap s;
  s.cap = uni(1, 2048);
  s.f_max = uni(1, 64);
  s.n_pin = uni(0, s.f_max - 1);
  const int32_t npf = uni(0, s.n_pin < 3 ? s.n_pin : 3);
  int32_t row = 0, t = 0;
  for (int32_t i = 0; i < npf && (int32_t)(s.frames.size() / 4) < s.f_max; ++i) {
    const int32_t len = uni(0, (s.cap - row) / 4);
    s.frames.insert(s.frames.end(), {row, len, t++, 1});
    row += len;
  }
  const int32_t pin_end = row;
  std::vector<char> used((size_t)s.cap, 0);
  const int32_t nu = uni(0, s.f_max - (int32_t)(s.frames.size() / 4));
  for (int32_t i = 0; i < nu; ++i) {
    const int32_t len = uni(0, 96);
    const int32_t st = uni(pin_end, s.cap);
    bool ok = (int64_t)st + len <= s.cap;
    for (int32_t r = st; ok && r < st + len; ++r) ok = !used[(size_t)r];
    if (!ok) continue;
    for (int32_t r = st; r < st + len; ++r) used[(size_t)r] = 1;
    s.frames.insert(s.frames.end(), {st, len, t++, 0});
  }
  int32_t keys = 0;
  for (size_t f = 0; f < s.frames.size(); f += 4) keys += s.frames[f + 1];
  s.hdr[0] = (int32_t)(s.frames.size() / 4);
  s.hdr[1] = pin_end;
  s.hdr[2] = 0;
  s.hdr[3] = keys;
  return s;
}

static bool check_snapshot(const Snap& s, bool have_rows, bool must_accept) {
  // the frame table holds exactly the entries the header names (none when
  // that count is negative; a count past f_max, which must be rejected before
  // any entry is read, gets f_max + 3 entries): an over-read is a sanitizer
  // error
  const int32_t nf = s.hdr[0];
  const size_t n = nf > 0 ? (size_t)(nf <= s.f_max + 3 ? nf : s.f_max + 3) * 4 : 0;
  int32_t* fr = n ? (int32_t*)malloc(n * sizeof(int32_t)) : nullptr;
  for (size_t i = 0; i < n; ++i) fr[i] = i < s.frames.size() ? s.frames[i] : 0;
  int32_t np = -1;
  bool unp = false;
  const bool ok = rs3host::bank_snapshot_ok(s.cap, s.f_max, s.n_pin, s.hdr, fr, have_rows, &np, &unp);
  if (ok) {
    CHECK(invariants(s.cap, s.f_max, s.n_pin, s.hdr, fr, have_rows), "accepted an unreachable snapshot");
    int32_t cnt = 0;
    bool any = false;
    for (int32_t f = 0; f < nf; ++f) {   // (accepted: nf <= f_max)
      cnt += fr[4 * f + 3] == 1;
      any = any || fr[4 * f + 3] == 0;
    }
    CHECK(np == cnt && unp == any, "wrong frame summary");
  } else {
    CHECK(!invariants(s.cap, s.f_max, s.n_pin, s.hdr, fr, have_rows) || nf < 0,
          "rejected a reachable snapshot");
  }
  if (must_accept) CHECK(ok, "rejected a snapshot of the ring model");
  free(fr);
  return ok;
}

int main(int argc, char** argv) {
  const int iters = argc > 1 ? atoi(argv[1]) : 20000;
  if (argc > 2) {   // (a zero xorshift state would stay zero)
    rng_state = (strtoull(argv[2], nullptr, 10) + 1) * 0xd1b54a32d192ed03ull;
    if (rng_state == 0) rng_state = 1;
  }
  int accepted = 0, rejected = 0;
  for (int it = 0; it < iters; ++it) {
    Snap s = build_valid();
    check_snapshot(s, true, true);
    // rows missing while the header counts some
    if (s.hdr[3] > 0) {
      int32_t np;
      bool unp;
      CHECK(!rs3host::bank_snapshot_ok(s.cap, s.f_max, s.n_pin, s.hdr, s.frames.data(), false, &np, &unp),
            "accepted resident rows without K, V and pos");
    }
    // one to three mutated words of the header or the frame table
    const int nm = uni(1, 3);
    for (int k = 0; k < nm; ++k) {
      const int where = uni(0, 4 + (int)s.frames.size());
      const int32_t v = (next_u64() & 1) ? extreme() : uni(-70, 2100);
      if (where < 4)
        s.hdr[where] = v;
      else if (!s.frames.empty())
        s.frames[(size_t)(where - 4) % s.frames.size()] = v;
    }
    (check_snapshot(s, true, false) ? accepted : rejected)++;
    // a frame count past the frame table's capacity
    Snap t = build_valid();
    t.hdr[0] = t.f_max + uni(1, 3);
    check_snapshot(t, true, false);
    int32_t np;
    bool unp;
    const bool ok = rs3host::bank_snapshot_ok(s.cap, s.f_max, s.n_pin, s.hdr, nullptr, true, &np, &unp);
    CHECK(!ok || s.hdr[0] == 0, "accepted frames without a frame table");
  }
  // tracker states
  int t_acc = 0;
  for (int it = 0; it < iters; ++it) {
    const int n_obj = uni(1, 8);
    std::vector<int32_t> st((size_t)n_obj * 6);
    bool want = true;
    for (int o = 0; o < n_obj; ++o) {
      int32_t* w = &st[(size_t)o * 6];
      const int kind = uni(0, 3);
      if (kind == 0) {   // a reachable state with a box
        w[0] = uni(0, 4000);
        w[1] = uni(0, 4000);
        w[2] = w[0] + uni(0, 100);
        w[3] = w[1] + uni(0, 100);
        w[4] = uni(0, 30);
        w[5] = 1;
      } else if (kind == 1) {   // before any box
        w[0] = w[1] = w[2] = w[3] = 0;
        w[4] = uni(0, 30);
        w[5] = 0;
      } else {   // random or extreme words
        for (int j = 0; j < 6; ++j) w[j] = (next_u64() & 1) ? extreme() : uni(-5, 5);
      }
      const int32_t LIM = 1 << 30;
      const bool box_ok = w[0] >= 0 && w[1] >= 0 && w[0] <= w[2] && w[1] <= w[3] && w[2] < LIM && w[3] < LIM;
      const bool zero = w[0] == 0 && w[1] == 0 && w[2] == 0 && w[3] == 0;
      const bool ok = (w[5] == 1 && box_ok || w[5] == 0 && zero) && w[4] >= 0 && w[4] <= LIM;
      want = want && ok;
    }
    const bool got = rs3host::track_state_ok(n_obj, st.data());
    CHECK(got == want, "tracker state verdict %d, expected %d", (int)got, (int)want);
    t_acc += got;
  }
  CHECK(!rs3host::track_state_ok(1, nullptr), "accepted a null tracker state");
  CHECK(!rs3host::bank_snapshot_ok(10, 2, 1, nullptr, nullptr, true, nullptr, nullptr), "accepted a null header");
  printf("snapshots accepted %d rejected %d, tracker states accepted %d of %d, failures %d\n", accepted, rejected,
         t_acc, iters, failures);
  if (failures == 0) printf("ok\n");
  return failures ? 1 : 0;
}
