// Host side of the rs3 C ABI: handle management, argument validation and
// kernel launches.  Every check that can be made on the host runs before any
// HIP call, so a rejected call leaves all state untouched.
#include <math.h>
#include <stdlib.h>
#include <string.h>

#include <mutex>
#include <vector>

#include "host_check.h"
#include "rs3_internal.h"

using namespace rs3;

struct rs3_track {
  int32_t n_obj;
  int32_t* d_state;  // [n_obj][RS3_TRACK_WORDS]
};

struct rs3_layer {
  LayerDev dev;         // host copy holding device pointers
  mutable int n_banks;  // banks created from the layer and not yet destroyed
};

struct rs3_bank {
  const rs3_layer* L;
  BankDev host;     // host copy holding device pointers
  BankDev* d_desc;  // device copy of `host`
  int32_t pin_calls;
  int32_t unpinned_seen;
  uint32_t commits;   // commits launched; the parity selects the current frame table copy
};

namespace {

size_t dtype_size(int dt) { return dt == RS3_BF16 ? 2 : 4; }

rs3_status map_err(hipError_t e) {
  if (e == hipSuccess) return RS3_OK;
  if (e == hipErrorOutOfMemory) return RS3_E_OOM;
  return RS3_E_DEVICE;
}

bool setup_done = false;

rs3_status ensure_setup() {
  if (setup_done) return RS3_OK;
  hipError_t e = rs3_readout_setup();
  if (e == hipSuccess) e = rs3_select_setup();
  if (e == hipSuccess) e = rs3_commit_setup();
  if (e == hipSuccess) e = rs3_fused_setup();
  if (e == hipSuccess) e = rs3_stack_setup();
  if (e != hipSuccess) return RS3_E_DEVICE;
  setup_done = true;
  return RS3_OK;
}

bool grid_ok(const rs3_grid* g) {
  if (!g || g->m <= 0 || g->n <= 0 || g->s <= 0) return false;
  int64_t mn = (int64_t)g->m * g->n;
  if (mn > RS3_MAX_MN) return false;
  if ((int64_t)g->m * g->s * g->n * g->s > (1ll << 30)) return false;
  return true;
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Token tensors are read and written in 16-byte vectors: their base pointers
// must be 16-byte aligned and their per-object strides whole 16-byte units.
bool aligned16(const void* p) { return ((uintptr_t)p & 15) == 0; }
bool stride16(int64_t elems, size_t es) { return ((uint64_t)elems * es) % 16 == 0; }

// Transpose a row-major [rows][cols] host matrix of `es`-byte elements.
std::vector<uint8_t> transpose(const void* src, int rows, int cols, size_t es) {
  std::vector<uint8_t> out((size_t)rows * cols * es);
  const uint8_t* s = (const uint8_t*)src;
  for (int r = 0; r < rows; ++r)
    for (int c = 0; c < cols; ++c) memcpy(&out[((size_t)c * rows + r) * es], &s[((size_t)r * cols + c) * es], es);
  return out;
}

// Key splits per query tile.  The most splits whose attention launch
// (8*n_qt*ceil(n_obj*H*S/8) work-groups) still fits the 256 CUs once, and
// key ranges whose K^/V^ tiles (kv_bytes per object and head) fit an XCD's
// 4 MB L2 in slices of at most L2_SPLIT_BYTES: the query tiles of one key
// range run on one XCD and then share its cached tiles instead of each
// streaming the whole range from the memory side.
constexpr double L2_SPLIT_BYTES = 2.0 * 1024 * 1024;

int max_auto_splits(int H) {
  int S = 64;
  if (S * H > RS3_MAX_SPLITS_X_HEADS) S = RS3_MAX_SPLITS_X_HEADS / H;
  return S < 1 ? 1 : S;
}

int auto_splits(int n_obj, int H, int n_qt, double kv_bytes) {
  const int groups = n_qt <= 32 ? 8 * (32 / n_qt) : 0;   // key groups that fit one launch wave
  int S = groups / (n_obj * H);
  const double s_l2 = kv_bytes / L2_SPLIT_BYTES;
  if (s_l2 > S) S = s_l2 > 4096.0 ? 4096 : (int)s_l2 + 1;
  const int cap = max_auto_splits(H);
  if (S > cap) S = cap;
  if (S < 1) S = 1;
  return S;
}

}  // namespace

extern "C" {

const char* rs3_status_str(rs3_status s) {
  switch (s) {
    case RS3_OK: return "ok";
    case RS3_E_INVALID: return "invalid argument";
    case RS3_E_CAPACITY: return "bank capacity exceeded";
    case RS3_E_DEVICE: return "device error";
    case RS3_E_OOM: return "out of device memory";
  }
  return "unknown status";
}

// ---- tracker ---------------------------------------------------------------
rs3_status rs3_track_create(int32_t n_obj, rs3_track** out) {
  if (!out || n_obj <= 0 || n_obj > RS3_MAX_OBJ) return RS3_E_INVALID;
  *out = nullptr;
  rs3_track* t = new rs3_track();
  t->n_obj = n_obj;
  size_t bytes = (size_t)n_obj * RS3_TRACK_WORDS * 4;
  hipError_t e = hipMalloc((void**)&t->d_state, bytes);
  if (e == hipSuccess) e = hipMemset(t->d_state, 0, bytes);
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (e != hipSuccess) {
    if (t->d_state) (void)hipFree(t->d_state);
    delete t;
    return map_err(e);
  }
  *out = t;
  return RS3_OK;
}

void rs3_track_destroy(rs3_track* t) {
  if (!t) return;
  (void)hipFree(t->d_state);
  delete t;
}

rs3_status rs3_track_export(const rs3_track* t, int32_t* state) {
  if (!t || !state) return RS3_E_INVALID;
  hipError_t e = hipDeviceSynchronize();
  if (e == hipSuccess)
    e = hipMemcpy(state, t->d_state, (size_t)t->n_obj * RS3_TRACK_WORDS * 4, hipMemcpyDeviceToHost);
  return map_err(e);
}

rs3_status rs3_track_import(rs3_track* t, const int32_t* state) {
  if (!t || !state) return RS3_E_INVALID;
  // only states the tracker update reaches (host_check.h)
  if (!rs3host::track_state_ok(t->n_obj, state)) return RS3_E_INVALID;
  hipError_t e = hipDeviceSynchronize();
  if (e == hipSuccess)
    e = hipMemcpy(t->d_state, state, (size_t)t->n_obj * RS3_TRACK_WORDS * 4, hipMemcpyHostToDevice);
  return map_err(e);
}

}  // extern "C"

// ---- layer -----------------------------------------------------------------
namespace {

double load_elem(const void* p, size_t i, int dt) {
  if (dt == RS3_F32) return (double)((const float*)p)[i];
  uint32_t u = (uint32_t)((const uint16_t*)p)[i] << 16;
  float f;
  memcpy(&f, &u, 4);
  return (double)f;
}

// Rounds to the layer dtype (bf16: nearest even) and appends the bytes.
void store_elem(std::vector<uint8_t>& out, size_t i, double v, int dt) {
  float f = (float)v;
  if (dt == RS3_F32) {
    memcpy(&out[i * 4], &f, 4);
    return;
  }
  uint32_t u;
  memcpy(&u, &f, 4);
  u += 0x7fffu + ((u >> 16) & 1u);
  const uint16_t b = (uint16_t)(u >> 16);
  memcpy(&out[i * 2], &b, 2);
}

// (A B)^T for row-major A [r][k], B [k][c], accumulated in fp64, as [c][r].
std::vector<uint8_t> product_T(const void* A, const void* B, int r, int k, int c, int dt, bool b_transposed) {
  const size_t es = dtype_size(dt);
  std::vector<uint8_t> out((size_t)r * c * es);
  std::vector<double> a((size_t)r * k), bb((size_t)k * c);
  for (size_t i = 0; i < a.size(); ++i) a[i] = load_elem(A, i, dt);
  // b_transposed: B is given as [c][k] (row-major) and used as its transpose
  for (int kk = 0; kk < k; ++kk)
    for (int j = 0; j < c; ++j) bb[(size_t)kk * c + j] = load_elem(B, b_transposed ? (size_t)j * k + kk : (size_t)kk * c + j, dt);
  for (int i = 0; i < r; ++i)
    for (int j = 0; j < c; ++j) {
      double acc = 0.0;
      for (int kk = 0; kk < k; ++kk) acc += a[(size_t)i * k + kk] * bb[(size_t)kk * c + j];
      store_elem(out, (size_t)j * r + i, acc, dt);
    }
  return out;
}

}  // namespace

extern "C" {

rs3_status rs3_layer_create(int32_t C, int32_t H, int32_t d_kv, rs3_dtype dt, int32_t absorb, const void* Wq,
                            const void* Wk, const void* Wv, const void* Wo, rs3_layer** out) {
  if (!out || !Wq || !Wk || !Wv || !Wo) return RS3_E_INVALID;
  if (dt != RS3_BF16 && dt != RS3_F32) return RS3_E_INVALID;
  if (absorb != 0 && absorb != 1) return RS3_E_INVALID;
  if (C <= 0 || C > 1024 || H <= 0 || C % H != 0) return RS3_E_INVALID;
  const int d_h = C / H;
  if (d_kv <= 0 || d_kv > 256 || d_kv % 16 != 0) return RS3_E_INVALID;
  if (absorb && H != 1) return RS3_E_INVALID;
  const int Da = absorb ? d_kv : C;
  const int dah = absorb ? d_kv : d_h;
  if (dt == RS3_BF16) {
    if (dah != 32 && dah != 64 && dah != 128 && dah != 256) return RS3_E_INVALID;
    if (C % 64 != 0 || Da % 64 != 0) return RS3_E_INVALID;
  } else {
    if (dah > 256 || C % 8 != 0) return RS3_E_INVALID;
  }
  *out = nullptr;
  const size_t es = dtype_size(dt);
  const int D = C;
  rs3_layer* L = new rs3_layer();
  LayerDev& ld = L->dev;
  ld.C = C;
  ld.H = H;
  ld.d_h = d_h;
  ld.D = D;
  ld.d_kv = d_kv;
  ld.dtype = dt;
  ld.absorb = absorb;
  ld.Da = Da;
  ld.Ha = absorb ? 1 : H;
  ld.dah = dah;
  std::vector<uint8_t> wq, wk, wv, wo;
  if (absorb) {
    // W_qk = W_q W_k^T  [C][d_kv] -> stored transposed [d_kv][C]
    wq = product_T(Wq, Wk, C, D, d_kv, dt, true);
    // W_vo = W_v W_o    [d_kv][C] -> stored transposed [C][d_kv]
    wo = product_T(Wv, Wo, d_kv, D, C, dt, false);
  } else {
    wq = transpose(Wq, C, D, es);
    wk = transpose(Wk, d_kv, D, es);
    wv = transpose(Wv, d_kv, D, es);
    wo = transpose(Wo, D, C, es);
  }
  void** dst[4] = {&ld.WqT, &ld.WkT, &ld.WvT, &ld.WoT};
  std::vector<uint8_t>* src[4] = {&wq, &wk, &wv, &wo};
  hipError_t e = hipSuccess;
  for (int i = 0; i < 4 && e == hipSuccess; ++i) {
    if (src[i]->empty()) continue;
    e = hipMalloc(dst[i], src[i]->size());
    if (e == hipSuccess) e = hipMemcpy(*dst[i], src[i]->data(), src[i]->size(), hipMemcpyHostToDevice);
  }
  if (e != hipSuccess) {
    for (int i = 0; i < 4; ++i)
      if (*dst[i]) (void)hipFree(*dst[i]);
    delete L;
    return map_err(e);
  }
  *out = L;
  return RS3_OK;
}

void rs3_layer_destroy(rs3_layer* L) {
  if (!L) return;
  void* w[5] = {L->dev.WqT, L->dev.WkT, L->dev.WvT, L->dev.WoT, L->dev.rope};
  for (void* p : w)
    if (p) (void)hipFree(p);
  delete L;
}

// ---- rotary table ------------------------------------------------------------
namespace {

rs3_status rope_args_ok(const rs3_layer* L, int32_t m, int32_t n) {
  if (!L || L->dev.absorb || L->n_banks > 0 || L->dev.dah % 2 != 0) return RS3_E_INVALID;
  if (m <= 0 || n <= 0 || (int64_t)m * n > RS3_MAX_MN) return RS3_E_INVALID;
  return RS3_OK;
}

// Replaces the layer's table by a fresh uninitialised one of m x n rows.
rs3_status rope_alloc(rs3_layer* L, int32_t m, int32_t n, float** out) {
  const size_t bytes = (size_t)m * n * L->dev.dah * 4;   // d_h/2 pairs of two floats
  float* t = nullptr;
  hipError_t e = hipMalloc((void**)&t, bytes);
  if (e != hipSuccess) return map_err(e);
  *out = t;
  return RS3_OK;
}

void rope_install(rs3_layer* L, float* t, int32_t m, int32_t n) {
  if (L->dev.rope) (void)hipFree(L->dev.rope);
  L->dev.rope = t;
  L->dev.rope_m = m;
  L->dev.rope_n = n;
}

}  // namespace

rs3_status rs3_layer_set_rope(rs3_layer* L, int32_t m, int32_t n, const float* table) {
  if (!L) return RS3_E_INVALID;
  if (!table) {
    if (m != 0 || n != 0 || L->dev.absorb || L->n_banks > 0) return RS3_E_INVALID;
    rope_install(L, nullptr, 0, 0);
    return RS3_OK;
  }
  rs3_status st = rope_args_ok(L, m, n);
  if (st != RS3_OK) return st;
  float* t = nullptr;
  st = rope_alloc(L, m, n, &t);
  if (st != RS3_OK) return st;
  hipError_t e = hipMemcpy(t, table, (size_t)m * n * L->dev.dah * 4, hipMemcpyHostToDevice);
  if (e != hipSuccess) {
    (void)hipFree(t);
    return map_err(e);
  }
  rope_install(L, t, m, n);
  return RS3_OK;
}

rs3_status rs3_layer_set_rope_axial(rs3_layer* L, int32_t m, int32_t n, double theta) {
  rs3_status st = rope_args_ok(L, m, n);
  if (st != RS3_OK) return st;
  if (!(theta > 1.0) || L->dev.dah % 4 != 0) return RS3_E_INVALID;
  float* t = nullptr;
  st = rope_alloc(L, m, n, &t);
  if (st != RS3_OK) return st;
  hipError_t e = rs3_launch_rope_axial(t, m, n, L->dev.dah, theta, nullptr);
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (e != hipSuccess) {
    (void)hipFree(t);
    return map_err(e);
  }
  rope_install(L, t, m, n);
  return RS3_OK;
}

// ---- bank ------------------------------------------------------------------
rs3_status rs3_bank_create(const rs3_layer* L, int32_t cap, int32_t f_max, int32_t n_pin,
                           rs3_bank** out) {
  if (!out || !L) return RS3_E_INVALID;
  if (cap < 1 || cap > (1 << 26) || f_max < 1 || f_max > 256 || n_pin < 0 || n_pin >= f_max)
    return RS3_E_INVALID;
  *out = nullptr;
  rs3_status st = ensure_setup();
  if (st != RS3_OK) return st;
  const LayerDev& ld = L->dev;
  const size_t es = dtype_size(ld.dtype);
  rs3_bank* b = new rs3_bank();
  b->L = L;
  b->pin_calls = 0;
  b->unpinned_seen = 0;
  b->commits = 0;
  BankDev& h = b->host;
  memset(&h, 0, sizeof(h));
  h.cap = cap;
  h.f_max = f_max;
  h.n_pin = n_pin;
  h.d_kv = ld.d_kv;
  h.H = ld.Ha;
  h.d_h = ld.dah;
  h.dtype = ld.dtype;
  h.n_tiles_cap = (cap + KT - 1) / KT;
  const size_t raw = (size_t)cap * ld.d_kv * es;
  const size_t proj = (size_t)h.n_tiles_cap * KT * ld.Da * es;
  struct Alloc {
    void** p;
    size_t bytes;
  } allocs[] = {
      {&h.Kraw, raw},
      {&h.Vraw, raw},
      {(void**)&h.pos, (size_t)cap * 4},
      {&h.Khat, proj},
      {&h.Vhat, proj},
      {(void**)&h.hdr, HDR_WORDS * 4},
      {(void**)&h.frames, (size_t)2 * f_max * 16},
      {(void**)&h.tiles, (size_t)h.n_tiles_cap * sizeof(TileEnt)},
      {(void**)&b->d_desc, sizeof(BankDev)},
  };
  hipError_t e = hipSuccess;
  for (auto& a : allocs) {
    if (e != hipSuccess) break;
    e = hipMalloc(a.p, a.bytes);
    // zero fill: padding rows of the projected tiles must hold finite values
    if (e == hipSuccess) e = hipMemset(*a.p, 0, a.bytes);
  }
  if (e == hipSuccess) e = hipMemcpy(b->d_desc, &h, sizeof(BankDev), hipMemcpyHostToDevice);
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (e != hipSuccess) {
    for (auto& a : allocs)
      if (*a.p) (void)hipFree(*a.p);
    delete b;
    return map_err(e);
  }
  L->n_banks++;
  *out = b;
  return RS3_OK;
}

void rs3_bank_destroy(rs3_bank* b) {
  if (!b) return;
  b->L->n_banks--;
  BankDev& h = b->host;
  void* ptrs[] = {h.Kraw, h.Vraw, h.pos, h.Khat, h.Vhat, h.hdr, h.frames, h.tiles, b->d_desc};
  for (void* p : ptrs)
    if (p) (void)hipFree(p);
  delete b;
}

rs3_status rs3_bank_export(const rs3_bank* b, int32_t* hdr, int32_t* frames, void* K, void* V,
                           int32_t* pos) {
  if (!b || !hdr) return RS3_E_INVALID;
  const BankDev& h = b->host;
  const int p = b->commits & 1;   // current copy of the frame table
  hipError_t e = hipDeviceSynchronize();
  int32_t dh[HDR_WORDS];
  if (e == hipSuccess) e = hipMemcpy(dh, h.hdr, sizeof(dh), hipMemcpyDeviceToHost);
  if (e != hipSuccess) return map_err(e);
  const int nf = dh[HDR_NFRAMES + HDR_COPY * p];
  std::vector<int32_t> fr((size_t)h.f_max * 4, 0);
  e = hipMemcpy(fr.data(), h.frames + (size_t)4 * h.f_max * p, fr.size() * 4, hipMemcpyDeviceToHost);
  if (e != hipSuccess) return map_err(e);
  int keys = 0;
  for (int f = 0; f < nf; ++f) keys += fr[4 * f + 1];
  memset(hdr, 0, RS3_BANK_HDR_WORDS * 4);
  hdr[0] = nf;
  hdr[1] = dh[HDR_PINEND + HDR_COPY * p];
  hdr[2] = dh[HDR_ERR];
  hdr[3] = keys;
  if (frames) memcpy(frames, fr.data(), (size_t)nf * 16);
  const size_t es = dtype_size(h.dtype);
  const size_t row = (size_t)h.d_kv * es;
  size_t off = 0;
  for (int f = 0; f < nf && e == hipSuccess; ++f) {
    const int s = fr[4 * f], l = fr[4 * f + 1];
    if (l == 0) continue;
    if (K) e = hipMemcpy((uint8_t*)K + off * row, (uint8_t*)h.Kraw + (size_t)s * row, l * row, hipMemcpyDeviceToHost);
    if (V && e == hipSuccess)
      e = hipMemcpy((uint8_t*)V + off * row, (uint8_t*)h.Vraw + (size_t)s * row, l * row, hipMemcpyDeviceToHost);
    if (pos && e == hipSuccess)
      e = hipMemcpy(pos + off, h.pos + s, (size_t)l * 4, hipMemcpyDeviceToHost);
    off += l;
  }
  return map_err(e);
}

rs3_status rs3_bank_import(rs3_bank* b, const int32_t* hdr, const int32_t* frames, const void* K, const void* V,
                           const int32_t* pos) {
  if (!b || !hdr) return RS3_E_INVALID;
  BankDev& h = b->host;
  // the snapshot must be a state the placement rule can reach (host_check.h)
  int32_t n_pinned = 0;
  bool unpinned = false;
  if (!rs3host::bank_snapshot_ok(h.cap, h.f_max, h.n_pin, hdr, frames, K && V && pos, &n_pinned, &unpinned))
    return RS3_E_INVALID;
  const int nf = hdr[0], pin_end = hdr[1], err = hdr[2], keys = hdr[3];
  const rs3_layer* L = b->L;
  const int p = b->commits & 1;   // the restored state becomes the current copy
  hipError_t e = hipDeviceSynchronize();
  std::vector<int32_t> fr((size_t)h.f_max * 4, 0);
  if (nf > 0) memcpy(fr.data(), frames, (size_t)nf * 16);
  if (e == hipSuccess)
    e = hipMemcpy(h.frames + (size_t)4 * h.f_max * p, fr.data(), fr.size() * 4, hipMemcpyHostToDevice);
  int32_t dh[HDR_WORDS] = {};
  dh[HDR_NFRAMES + HDR_COPY * p] = nf;
  dh[HDR_PINEND + HDR_COPY * p] = pin_end;
  dh[HDR_ERR] = err;
  dh[HDR_PLEN] = -1;
  dh[HDR_NKEYS] = keys;
  if (e == hipSuccess) e = hipMemcpy(h.hdr, dh, sizeof(dh), hipMemcpyHostToDevice);
  const size_t row = (size_t)h.d_kv * dtype_size(h.dtype);
  size_t off = 0;
  for (int f = 0; f < nf && e == hipSuccess; ++f) {
    const int st = fr[4 * f], len = fr[4 * f + 1];
    if (len == 0) continue;
    e = hipMemcpy((uint8_t*)h.Kraw + (size_t)st * row, (const uint8_t*)K + off * row, len * row,
                  hipMemcpyHostToDevice);
    if (e == hipSuccess)
      e = hipMemcpy((uint8_t*)h.Vraw + (size_t)st * row, (const uint8_t*)V + off * row, len * row,
                    hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMemcpy(h.pos + st, pos + off, (size_t)len * 4, hipMemcpyHostToDevice);
    off += len;
  }
  if (e != hipSuccess) return map_err(e);
  rs3_status st0 = ensure_setup();
  if (st0 != RS3_OK) return st0;
  // attention tiles of every resident frame, projected from the raw ring
  Rs3CommitArgs a;
  memset(&a, 0, sizeof(a));
  a.banks[0] = b->d_desc;
  a.WkT = L->dev.WkT;
  a.WvT = L->dev.WvT;
  a.absorb = L->dev.absorb;
  a.rope = L->dev.rope;
  a.rope_mn = L->dev.rope_m * L->dev.rope_n;
  a.n_obj = 1;
  a.m = 1;
  a.s = 1;
  a.from_ring = 1;
  a.parity = (uint64_t)p;
  for (int f = 0; f < nf && e == hipSuccess; ++f) {
    const int span[2] = {fr[4 * f], fr[4 * f + 1]};
    if (span[1] == 0) continue;
    e = hipMemcpy(h.hdr + HDR_PSTART, span, sizeof(span), hipMemcpyHostToDevice);
    a.n = span[1];
    if (e == hipSuccess) e = rs3_launch_bank_restore(a, h.dtype, h.d_kv, 0, nullptr);
    if (e == hipSuccess) e = hipDeviceSynchronize();
  }
  if (e == hipSuccess) e = rs3_launch_bank_restore(a, h.dtype, h.d_kv, 1, nullptr);
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (e != hipSuccess) return map_err(e);
  b->pin_calls = n_pinned;
  b->unpinned_seen = unpinned ? 1 : 0;
  return RS3_OK;
}

rs3_status rs3_bank_error(rs3_bank* b, int32_t* err, int32_t clear) {
  if (!b || !err) return RS3_E_INVALID;
  hipError_t e = hipDeviceSynchronize();
  if (e == hipSuccess) e = hipMemcpy(err, b->host.hdr + HDR_ERR, 4, hipMemcpyDeviceToHost);
  if (e == hipSuccess && clear) e = hipMemset(b->host.hdr + HDR_ERR, 0, 4);
  if (e == hipSuccess && clear) e = hipDeviceSynchronize();
  return map_err(e);
}

// ---- select ----------------------------------------------------------------
rs3_status rs3_select_workspace_size(const rs3_grid* g, int32_t n_obj, int64_t x_obj_stride,
                                     size_t* bytes) {
  if (!bytes || !grid_ok(g) || n_obj <= 0 || n_obj > RS3_MAX_OBJ || x_obj_stride < 0) return RS3_E_INVALID;
  const int64_t mn = (int64_t)g->m * g->n;
  const int n_x = x_obj_stride ? n_obj : 1;
  // energies [n_x][mn] fp64, per-64-cell energy ranges [n_x][ceil(mn/64)][2],
  // then the priors computed beside the energies [n_obj][64][4] u64
  *bytes = align256((size_t)n_x * mn * 8) + align256((size_t)n_x * ((mn + 63) / 64) * 16) +
           (size_t)n_obj * 64 * 4 * 8;
  return RS3_OK;
}

// Validates a select call and fills its kernel arguments (no device work).
struct SelectLaunch {
  Rs3SelectArgs a;
  const void* X;
  int64_t x_stride;
  int n_x, mn, C, dtype, n_groups;
  double* e;
  unsigned long long* erange;
  uint64_t* pbits;
};

static rs3_status select_args(const rs3_grid* g, int32_t n_obj, const uint8_t* masks, rs3_track* tr, const void* X,
                              int64_t x_obj_stride, int32_t C, rs3_dtype dt, const int32_t* k,
                              const rs3_select_params* p, void* ws, size_t ws_bytes, int32_t* sel_idx,
                              int32_t* sel_count, uint8_t* prior_out, SelectLaunch& sl) {
  if (!grid_ok(g) || !masks || !tr || !X || !k || !p || !ws || !sel_idx || !sel_count) return RS3_E_INVALID;
  if (n_obj <= 0 || n_obj > RS3_MAX_OBJ || tr->n_obj != n_obj) return RS3_E_INVALID;
  if (dt != RS3_BF16 && dt != RS3_F32) return RS3_E_INVALID;
  if (C <= 0 || C % 8 != 0) return RS3_E_INVALID;
  const int mn = g->m * g->n;
  if (x_obj_stride < 0 || (x_obj_stride != 0 && x_obj_stride < (int64_t)mn * C)) return RS3_E_INVALID;
  if (x_obj_stride != 0 && p->union_objects && n_obj > 1) return RS3_E_INVALID;
  if (!aligned16(X) || !stride16(x_obj_stride, dtype_size(dt))) return RS3_E_INVALID;
  if (p->r_s < 0 || p->c < 0) return RS3_E_INVALID;
  const int n_groups = p->union_objects ? 1 : n_obj;
  for (int i = 0; i < n_groups; ++i)
    if (k[i] < 0 || k[i] > mn) return RS3_E_INVALID;
  size_t need;
  rs3_select_workspace_size(g, n_obj, x_obj_stride, &need);
  if (ws_bytes < need) return RS3_E_INVALID;
  const int n_x = x_obj_stride ? n_obj : 1;
  sl.e = (double*)ws;
  sl.erange = (unsigned long long*)((uint8_t*)ws + align256((size_t)n_x * mn * 8));
  sl.pbits = (uint64_t*)((uint8_t*)sl.erange + align256((size_t)n_x * ((mn + 63) / 64) * 16));
  Rs3SelectArgs& a = sl.a;
  memset(&a, 0, sizeof(a));
  a.masks = masks;
  a.track = tr->d_state;
  a.e = sl.e;
  a.erange = sl.erange;
  a.sel_idx = sel_idx;
  a.sel_count = sel_count;
  a.prior_out = prior_out;
  a.m = g->m;
  a.n = g->n;
  a.s = g->s;
  a.n_obj = n_obj;
  a.union_objects = p->union_objects ? 1 : 0;
  a.seed_box = p->seed_box ? 1 : 0;
  a.r_s = p->r_s;
  a.c = p->c;
  a.x_per_obj = n_x > 1;
  for (int i = 0; i < n_groups; ++i) a.k[i] = k[i];
  sl.X = X;
  sl.x_stride = x_obj_stride;
  sl.n_x = n_x;
  sl.mn = mn;
  sl.C = C;
  sl.dtype = dt;
  sl.n_groups = n_groups;
  return RS3_OK;
}

// Energies (and the priors beside them, and with qp every row's projected
// query), then the selection.
static hipError_t select_launch(SelectLaunch& sl, hipStream_t st, const Rs3QProjArgs* qp = nullptr) {
  Rs3SelectArgs& a = sl.a;
  hipError_t he;
  if (rs3_select_prior_beside(a.m, a.n, a.s)) {
    a.prior_bits = sl.pbits;
    he = rs3_launch_energy_prior(sl.X, sl.x_stride, sl.n_x, sl.mn, sl.C, sl.dtype, sl.e, sl.erange, a, sl.n_groups, st,
                                 qp);
  } else {
    he = rs3_launch_energy(sl.X, sl.x_stride, sl.n_x, sl.mn, sl.C, sl.dtype, sl.e, sl.erange, st, qp);
  }
  if (he != hipSuccess) return he;
  return rs3_launch_select(a, sl.n_groups, st);
}

rs3_status rs3_select_queries(const rs3_grid* g, int32_t n_obj, const uint8_t* masks, rs3_track* tr,
                              const void* X, int64_t x_obj_stride, int32_t C, rs3_dtype dt,
                              const int32_t* k, const rs3_select_params* p, void* ws, size_t ws_bytes,
                              int32_t* sel_idx, int32_t* sel_count, uint8_t* prior_out, void* stream) {
  SelectLaunch sl;
  rs3_status st = select_args(g, n_obj, masks, tr, X, x_obj_stride, C, dt, k, p, ws, ws_bytes, sel_idx, sel_count,
                              prior_out, sl);
  if (st != RS3_OK) return st;
  st = ensure_setup();
  if (st != RS3_OK) return st;
  return map_err(select_launch(sl, (hipStream_t)stream));
}

// ---- bare attention core ---------------------------------------------------
namespace {
struct AttendLayout {
  size_t desc, hdr, tiles, khat, vhat, qs, opart, ml, total;
  int ntile, S;
};

bool attend_shape(int32_t n_q, int32_t n_kv, int32_t H, int32_t d_h, rs3_dtype dt, int32_t n_splits,
                  AttendLayout* L) {
  if (n_q < 0 || n_q > RS3_MAX_MN || n_kv < 0 || n_kv > (1 << 26) || H <= 0 || n_splits < 0) return false;
  if (dt == RS3_BF16) {
    if (d_h != 32 && d_h != 64 && d_h != 128 && d_h != 256) return false;
    if (H * d_h > 1024 || n_splits * H > RS3_MAX_SPLITS_X_HEADS) return false;
  } else if (dt == RS3_F32) {
    if (d_h <= 0 || d_h > 256) return false;
  } else {
    return false;
  }
  memset(L, 0, sizeof(*L));
  if (dt != RS3_BF16) return true;
  const int D = H * d_h;
  L->ntile = (n_kv + KT - 1) / KT;
  const int n_qt = (n_q + 127) / 128;
  L->S = n_splits > 0 ? n_splits : auto_splits(1, H, n_qt > 0 ? n_qt : 1, (double)n_kv * d_h * 4);
  size_t off = 0;
  auto take = [&](size_t bytes) { const size_t at = off; off += align256(bytes); return at; };
  L->desc = take(sizeof(BankDev));
  L->hdr = take((HDR_WORDS + 8) * 4);
  L->tiles = take((size_t)L->ntile * sizeof(TileEnt));
  L->khat = take((size_t)L->ntile * H * KT * d_h * 2);
  L->vhat = take((size_t)L->ntile * H * d_h * KT * 2);
  L->qs = take((size_t)n_q * D * 2);
  L->opart = take((size_t)L->S * n_q * D * 2);
  L->ml = take((size_t)L->S * n_q * H * 8);
  L->total = off;
  return true;
}
}  // namespace

rs3_status rs3_attend_workspace_size(int32_t n_q, int32_t n_kv, int32_t H, int32_t d_h, rs3_dtype dt,
                                     int32_t n_splits, size_t* bytes) {
  AttendLayout L;
  if (!bytes || !attend_shape(n_q, n_kv, H, d_h, dt, n_splits, &L)) return RS3_E_INVALID;
  *bytes = L.total;
  return RS3_OK;
}

rs3_status rs3_attend(const void* Qh, const void* Kh, const void* Vh, int32_t n_q, int32_t n_kv, int32_t H,
                      int32_t d_h, rs3_dtype dt, int32_t n_splits, float* O, void* ws, size_t ws_bytes,
                      void* stream) {
  AttendLayout L;
  if (!attend_shape(n_q, n_kv, H, d_h, dt, n_splits, &L)) return RS3_E_INVALID;
  if ((n_q > 0 && (!Qh || !O)) || (n_kv > 0 && (!Kh || !Vh))) return RS3_E_INVALID;
  if (dt == RS3_BF16 && (!ws || ws_bytes < L.total)) return RS3_E_INVALID;
  if (!aligned16(Qh) || !aligned16(Kh) || !aligned16(Vh) || !aligned16(O) || !aligned16(ws)) return RS3_E_INVALID;
  rs3_status st0 = ensure_setup();
  if (st0 != RS3_OK) return st0;
  hipStream_t st = (hipStream_t)stream;
  const float qscale = (float)(1.4426950408889634 / sqrt((double)d_h));
  if (dt == RS3_F32)
    return map_err(rs3_launch_attend_f32((const float*)Qh, (const float*)Kh, (const float*)Vh, n_q, n_kv, H, d_h,
                                         qscale, O, st));
  if (n_q == 0) return RS3_OK;
  uint8_t* w = (uint8_t*)ws;
  AttendPrepArgs p;
  memset(&p, 0, sizeof(p));
  p.Q = (const bf16_t*)Qh;
  p.K = (const bf16_t*)Kh;
  p.V = (const bf16_t*)Vh;
  p.Qs = (bf16_t*)(w + L.qs);
  p.Khat = (bf16_t*)(w + L.khat);
  p.Vhat = (bf16_t*)(w + L.vhat);
  p.tiles = (TileEnt*)(w + L.tiles);
  p.desc = (BankDev*)(w + L.desc);
  p.hdr = (int32_t*)(w + L.hdr);
  p.count = p.hdr + HDR_WORDS;
  p.n_kv = n_kv;
  p.qscale = qscale;
  p.n_q = n_q;
  p.H = H;
  p.d_h = d_h;
  p.ntile = L.ntile;
  hipError_t e = rs3_launch_attend_prep(p, st);
  if (e != hipSuccess) return map_err(e);
  Rs3ReadoutArgs a;
  memset(&a, 0, sizeof(a));
  a.banks[0] = p.desc;
  a.sel_count = p.count;
  a.Q = p.Qs;
  a.Opart = w + L.opart;
  a.ML = (float*)(w + L.ml);
  a.qscale = qscale;
  a.mn = n_q;
  a.C = H * d_h;
  a.H = H;
  a.d_h = d_h;
  a.D = H * d_h;
  a.n_obj = 1;
  a.max_sel = n_q;
  a.S = L.S;
  a.n_qt = (n_q + 127) / 128;
  Rs3AttnBanks ab;
  memset(&ab, 0, sizeof(ab));
  ab.hdr[0] = p.hdr;
  ab.tiles[0] = p.tiles;
  ab.kh[0] = p.Khat;
  ab.vh[0] = p.Vhat;
  ab.ntcap[0] = L.ntile;
  e = rs3_launch_attn(a, ab, st, false);
  if (e != hipSuccess) return map_err(e);
  const int SA = L.ntile > 0 ? active_splits(L.ntile, L.S) : 0;
  return map_err(rs3_launch_attend_merge(a, SA, O, st));
}

// ---- readout ---------------------------------------------------------------
static void readout_shape(const rs3_layer* L, int32_t n_obj, int32_t max_sel, int32_t S, size_t* q_bytes,
                          size_t* o_bytes, size_t* ml_bytes) {
  const LayerDev& ld = L->dev;
  *q_bytes = align256((size_t)n_obj * max_sel * ld.Da * 2);
  *o_bytes = align256((size_t)n_obj * S * max_sel * ld.Da * 2);
  *ml_bytes = align256((size_t)n_obj * S * max_sel * ld.Ha * 8);
}

// kv_bytes < 0: the largest automatic choice (workspace sizing, where the
// banks are not known).
static int splits_for(const rs3_layer* L, int32_t n_obj, int32_t max_sel, int32_t n_splits, double kv_bytes) {
  if (n_splits > 0) return n_splits;
  if (kv_bytes < 0) return max_auto_splits(L->dev.Ha);
  const int n_qt = (max_sel + 127) / 128;
  return auto_splits(n_obj, L->dev.Ha, n_qt > 0 ? n_qt : 1, kv_bytes);
}

rs3_status rs3_readout_workspace_size(const rs3_layer* L, int32_t n_obj, int32_t max_sel, int32_t n_splits,
                                      size_t* bytes) {
  if (!L || !bytes || n_obj <= 0 || n_obj > RS3_MAX_OBJ || max_sel < 0 || n_splits < 0 ||
      n_splits * L->dev.Ha > RS3_MAX_SPLITS_X_HEADS)
    return RS3_E_INVALID;
  if (L->dev.dtype == RS3_F32) {
    *bytes = 0;
    return RS3_OK;
  }
  // The split count depends on max_sel, so take the largest layout over every
  // max_sel' <= max_sel (within a 128-row tile count the largest max_sel'
  // needs the most).
  size_t best = 0;
  const int n_qt_max = (max_sel + 127) / 128;
  for (int qt = 0; qt <= n_qt_max; ++qt) {
    const int ms = qt == n_qt_max ? max_sel : qt * 128;
    if (ms > max_sel) continue;
    const int S = splits_for(L, n_obj, ms, n_splits, -1.0);
    size_t q, o, ml;
    readout_shape(L, n_obj, ms, S, &q, &o, &ml);
    if (q + o + ml > best) best = q + o + ml;
  }
  *bytes = best;
  return RS3_OK;
}

// Validates a readout call and fills its kernel arguments (no device work).
static rs3_status readout_args(const rs3_layer* L, const rs3_grid* g, int32_t n_obj, const void* X,
                               int64_t x_obj_stride, rs3_bank* const* banks, const int32_t* sel_idx,
                               const int32_t* sel_count, int32_t sel_stride, int32_t max_sel, int32_t n_splits,
                               void* Y, int64_t y_obj_stride, int32_t y_fp32, void* ws, size_t ws_bytes,
                               Rs3ReadoutArgs& a, Rs3AttnBanks& ab, bool fit_splits = false) {
  if (!L || !grid_ok(g) || !X || !banks || !sel_idx || !sel_count || !Y) return RS3_E_INVALID;
  if (n_obj <= 0 || n_obj > RS3_MAX_OBJ) return RS3_E_INVALID;
  const LayerDev& ld = L->dev;
  const int mn = g->m * g->n;
  if (max_sel < 0 || max_sel > mn || n_splits < 0 || n_splits * ld.Ha > RS3_MAX_SPLITS_X_HEADS)
    return RS3_E_INVALID;
  if (sel_stride != 0 && sel_stride != mn) return RS3_E_INVALID;
  const int64_t grid_elems = (int64_t)mn * ld.C;
  if (x_obj_stride < 0 || (x_obj_stride != 0 && x_obj_stride < grid_elems)) return RS3_E_INVALID;
  if (n_obj > 1 && y_obj_stride < grid_elems) return RS3_E_INVALID;
  if (y_obj_stride < 0) return RS3_E_INVALID;
  const size_t y_es = (y_fp32 || ld.dtype == RS3_F32) ? 4 : 2;
  if (!aligned16(X) || !aligned16(Y) || !stride16(x_obj_stride, dtype_size(ld.dtype)) ||
      !stride16(y_obj_stride, y_es))
    return RS3_E_INVALID;
  for (int o = 0; o < n_obj; ++o) {
    if (!banks[o] || banks[o]->L != L) return RS3_E_INVALID;
    for (int p = 0; p < o; ++p)
      if (banks[p] == banks[o]) return RS3_E_INVALID;
  }
  if (Y == X) {
    if (y_fp32) return RS3_E_INVALID;
    if (n_obj > 1 && x_obj_stride != y_obj_stride) return RS3_E_INVALID;
  }
  if (ld.rope && (g->m != ld.rope_m || g->n != ld.rope_n)) return RS3_E_INVALID;
  if (ld.dtype == RS3_F32) y_fp32 = 0;
  // K^/V^ bytes of the largest bank's full ring, per head
  double kv_bytes = 0;
  for (int o = 0; o < n_obj; ++o) {
    const double kb = (double)banks[o]->host.cap * ld.dah * 4;
    if (kb > kv_bytes) kv_bytes = kb;
  }
  int S = splits_for(L, n_obj, max_sel, n_splits, kv_bytes);
  size_t q, o_b, ml;
  readout_shape(L, n_obj, max_sel, S, &q, &o_b, &ml);
  // fit_splits (automatic count into a fixed workspace): fewer key splits
  // until the partials fit
  while (fit_splits && n_splits == 0 && S > 1 && q + o_b + ml > ws_bytes) {
    --S;
    readout_shape(L, n_obj, max_sel, S, &q, &o_b, &ml);
  }
  if (ld.dtype == RS3_BF16 && (!ws || ws_bytes < q + o_b + ml)) return RS3_E_INVALID;
  memset(&a, 0, sizeof(a));
  for (int o = 0; o < n_obj; ++o) a.banks[o] = banks[o]->d_desc;
  memset(&ab, 0, sizeof(ab));
  for (int o = 0; o < n_obj; ++o) {
    const BankDev& h = banks[o]->host;
    ab.hdr[o] = h.hdr;
    ab.tiles[o] = h.tiles;
    ab.kh[o] = h.Khat;
    ab.vh[o] = h.Vhat;
    ab.ntcap[o] = h.n_tiles_cap;
  }
  a.X = X;
  a.x_stride = x_obj_stride;
  a.Y = Y;
  a.y_stride = y_obj_stride;
  a.sel_idx = sel_idx;
  a.sel_count = sel_count;
  a.sel_stride = sel_stride;
  a.WqT = ld.WqT;
  a.WoT = ld.WoT;
  a.Q = ws;
  a.Opart = ws ? (uint8_t*)ws + q : nullptr;
  a.ML = ws ? (float*)((uint8_t*)ws + q + o_b) : nullptr;
  // logits are scaled by 1/sqrt(d_h) of the layer's heads in both modes
  a.qscale = (float)(1.4426950408889634 / sqrt((double)ld.d_h));
  a.mn = mn;
  a.C = ld.C;
  a.H = ld.Ha;
  a.d_h = ld.dah;
  a.D = ld.Da;
  a.n_obj = n_obj;
  a.max_sel = max_sel;
  a.S = S;
  a.n_qt = (max_sel + 127) / 128;
  a.y_fp32 = y_fp32 ? 1 : 0;
  a.rope = ld.rope;
  a.stream_parts = 1;
  return RS3_OK;
}

rs3_status rs3_readout(const rs3_layer* L, const rs3_grid* g, int32_t n_obj, const void* X, int64_t x_obj_stride,
                       rs3_bank* const* banks, const int32_t* sel_idx, const int32_t* sel_count, int32_t sel_stride,
                       int32_t max_sel, int32_t n_splits, void* Y, int64_t y_obj_stride, int32_t y_fp32, void* ws,
                       size_t ws_bytes, void* stream) {
  Rs3ReadoutArgs a;
  Rs3AttnBanks ab;
  rs3_status st = readout_args(L, g, n_obj, X, x_obj_stride, banks, sel_idx, sel_count, sel_stride, max_sel, n_splits,
                               Y, y_obj_stride, y_fp32, ws, ws_bytes, a, ab);
  if (st != RS3_OK) return st;
  st = ensure_setup();
  if (st != RS3_OK) return st;
  return map_err(rs3_launch_readout(a, ab, L->dev.dtype, (hipStream_t)stream));
}

// ---- readout without a caller workspace ----------------------------------------
// The split partials and projected queries of rs3_readout_noalloc live in a
// fixed device array, one copy per GPU, held until the process ends.  Host
// code never passes the array's name to a kernel (in host code it stands for
// a host-side shadow): the device address comes from hipGetSymbolAddress,
// taken once per device with that device current, and is kept per device.
static __device__ __align__(256) uint8_t scratch[RS3_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int SCRATCH_MAX_DEVICES = 64;
std::mutex scratch_mu;
void* scratch_ptr[SCRATCH_MAX_DEVICES];

// The current device's copy of `scratch` (null when the device cannot be
// queried or the symbol has no address).
void* scratch_for_current_device() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= SCRATCH_MAX_DEVICES) return nullptr;
  std::lock_guard<std::mutex> lock(scratch_mu);
  if (!scratch_ptr[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return nullptr;
    scratch_ptr[dev] = ptr;
  }
  return scratch_ptr[dev];
}

}  // namespace

rs3_status rs3_readout_noalloc(const rs3_layer* L, const rs3_grid* g, int32_t n_obj, const void* X,
                               int64_t x_obj_stride, rs3_bank* const* banks, const int32_t* sel_idx,
                               const int32_t* sel_count, int32_t sel_stride, int32_t max_sel, int32_t n_splits,
                               void* Y, int64_t y_obj_stride, int32_t y_fp32, void* stream) {
  if (!L) return RS3_E_INVALID;
  void* ws = nullptr;
  size_t ws_bytes = 0;
  if (L->dev.dtype == RS3_BF16) {
    ws = scratch_for_current_device();
    if (!ws) return RS3_E_DEVICE;
    ws_bytes = RS3_NOALLOC_SCRATCH_BYTES;
  }
  Rs3ReadoutArgs a;
  Rs3AttnBanks ab;
  rs3_status st = readout_args(L, g, n_obj, X, x_obj_stride, banks, sel_idx, sel_count, sel_stride, max_sel, n_splits,
                               Y, y_obj_stride, y_fp32, ws, ws_bytes, a, ab, true);
  if (st != RS3_OK) return st;
  st = ensure_setup();
  if (st != RS3_OK) return st;
  return map_err(rs3_launch_readout(a, ab, L->dev.dtype, (hipStream_t)stream));
}

// ---- write keep-set ----------------------------------------------------------
rs3_status rs3_write_keepset(const rs3_grid* g, int32_t n_obj, const uint8_t* seed_masks, int32_t D_w,
                             int32_t fall_min, int32_t fall_max, int32_t n_copies, uint8_t* keep, int32_t* counts,
                             void* stream) {
  if (!grid_ok(g) || !seed_masks || !keep) return RS3_E_INVALID;
  if (n_obj <= 0 || n_obj > RS3_MAX_OBJ || n_copies <= 0 || n_copies > RS3_MAX_OBJ || D_w < 0)
    return RS3_E_INVALID;
  const int reach = g->m > g->n ? g->m : g->n;
  return map_err(rs3_launch_write_keepset(seed_masks, n_obj, g->m, g->n, g->s, D_w < reach ? D_w : reach, fall_min,
                                          fall_max, n_copies, keep, counts, (hipStream_t)stream));
}

// ---- closure and palette -------------------------------------------------------
static bool close_shape_ok(int32_t n_obj, int32_t H, int32_t W) {
  return n_obj >= 1 && n_obj <= RS3_MAX_OBJ && H >= 1 && H <= 16384 && W >= 1 && W <= 4096;
}

rs3_status rs3_close_workspace_size(int32_t n_obj, int32_t H, int32_t W, size_t* bytes) {
  if (!bytes || !close_shape_ok(n_obj, H, W)) return RS3_E_INVALID;
  *bytes = rs3_post_workspace_bytes(n_obj, H, W);
  return RS3_OK;
}

rs3_status rs3_close_masks(int32_t n_obj, int32_t H, int32_t W, const void* logits, rs3_dtype dt, int32_t k,
                           uint8_t* closed, uint8_t* palette, void* ws, size_t ws_bytes, void* stream) {
  if (!logits || !ws || !close_shape_ok(n_obj, H, W)) return RS3_E_INVALID;
  if (dt != RS3_BF16 && dt != RS3_F32) return RS3_E_INVALID;
  if (k < 1 || k > 15 || k % 2 == 0) return RS3_E_INVALID;
  if (ws_bytes < rs3_post_workspace_bytes(n_obj, H, W)) return RS3_E_INVALID;
  return map_err(rs3_launch_close_masks(n_obj, H, W, logits, dt, k, closed, palette, ws, (hipStream_t)stream));
}

// ---- commit ----------------------------------------------------------------
// Validates a commit call and fills its kernel arguments (no device work).
static rs3_status commit_args(rs3_bank* const* banks, int32_t n_obj, const rs3_grid* g, const void* Kmem,
                              const void* Vmem, int64_t kv_obj_stride, const uint8_t* masks, int32_t t, int32_t pin,
                              int32_t fall_min, int32_t fall_max, int32_t* kept_count, Rs3CommitArgs& a) {
  if (!banks || !grid_ok(g) || !Kmem || !Vmem || !masks) return RS3_E_INVALID;
  if (n_obj <= 0 || n_obj > RS3_MAX_OBJ) return RS3_E_INVALID;
  const int mn = g->m * g->n;
  const rs3_layer* L = banks[0] ? banks[0]->L : nullptr;
  if (!L) return RS3_E_INVALID;
  const LayerDev& ld = L->dev;
  if (n_obj > 1 && kv_obj_stride < (int64_t)mn * ld.d_kv) return RS3_E_INVALID;
  if (kv_obj_stride < 0) return RS3_E_INVALID;
  if (!aligned16(Kmem) || !aligned16(Vmem) || !stride16(kv_obj_stride, dtype_size(ld.dtype))) return RS3_E_INVALID;
  if (ld.rope && (g->m != ld.rope_m || g->n != ld.rope_n)) return RS3_E_INVALID;
  for (int o = 0; o < n_obj; ++o) {
    if (!banks[o] || banks[o]->L != L) return RS3_E_INVALID;
    for (int p = 0; p < o; ++p)
      if (banks[p] == banks[o]) return RS3_E_INVALID;
    if (pin && (banks[o]->unpinned_seen || banks[o]->pin_calls >= banks[o]->host.n_pin)) return RS3_E_INVALID;
  }
  memset(&a, 0, sizeof(a));
  for (int o = 0; o < n_obj; ++o) a.banks[o] = banks[o]->d_desc;
  a.masks = masks;
  a.Kmem = Kmem;
  a.Vmem = Vmem;
  a.kv_stride = kv_obj_stride;
  a.kept_count = kept_count;
  a.WkT = ld.WkT;
  a.WvT = ld.WvT;
  a.m = g->m;
  a.n = g->n;
  a.s = g->s;
  a.t = t;
  a.pin = pin ? 1 : 0;
  a.fall_min = fall_min;
  a.fall_max = fall_max;
  a.n_obj = n_obj;
  a.absorb = ld.absorb;
  a.rope = ld.rope;
  a.rope_mn = mn;
  for (int o = 0; o < n_obj; ++o) a.parity |= (uint64_t)(banks[o]->commits & 1u) << o;
  return RS3_OK;
}

// Host bookkeeping of a launched commit: frame-state parity and pin rules.
static void commit_done(rs3_bank* const* banks, int32_t n_obj, int32_t pin) {
  for (int o = 0; o < n_obj; ++o) {
    banks[o]->commits++;
    if (pin)
      banks[o]->pin_calls++;
    else
      banks[o]->unpinned_seen = 1;
  }
}

rs3_status rs3_commit(rs3_bank* const* banks, int32_t n_obj, const rs3_grid* g, const void* Kmem,
                      const void* Vmem, int64_t kv_obj_stride, const uint8_t* masks, int32_t t, int32_t pin,
                      int32_t fall_min, int32_t fall_max, int32_t* kept_count, void* stream) {
  Rs3CommitArgs a;
  rs3_status st = commit_args(banks, n_obj, g, Kmem, Vmem, kv_obj_stride, masks, t, pin, fall_min, fall_max,
                              kept_count, a);
  if (st != RS3_OK) return st;
  st = ensure_setup();
  if (st != RS3_OK) return st;
  const LayerDev& ld = banks[0]->L->dev;
  hipError_t e = rs3_launch_commit(a, ld.dtype, ld.d_kv, ld.Da, ld.Ha, ld.dah, (hipStream_t)stream);
  if (e != hipSuccess) return map_err(e);
  commit_done(banks, n_obj, pin);
  return RS3_OK;
}

rs3_status rs3_readout_commit(const rs3_layer* L, const rs3_grid* g, int32_t n_obj, const void* X,
                              int64_t x_obj_stride, rs3_bank* const* banks, const int32_t* sel_idx,
                              const int32_t* sel_count, int32_t sel_stride, int32_t max_sel, int32_t n_splits,
                              void* Y, int64_t y_obj_stride, int32_t y_fp32, void* ws, size_t ws_bytes,
                              const void* Kmem, const void* Vmem, int64_t kv_obj_stride, const uint8_t* masks,
                              int32_t t, int32_t pin, int32_t fall_min, int32_t fall_max, int32_t* kept_count,
                              void* stream) {
  Rs3ReadoutArgs ra;
  Rs3AttnBanks ab;
  Rs3CommitArgs ca;
  rs3_status st = readout_args(L, g, n_obj, X, x_obj_stride, banks, sel_idx, sel_count, sel_stride, max_sel,
                               n_splits, Y, y_obj_stride, y_fp32, ws, ws_bytes, ra, ab);
  if (st != RS3_OK) return st;
  st = commit_args(banks, n_obj, g, Kmem, Vmem, kv_obj_stride, masks, t, pin, fall_min, fall_max, kept_count, ca);
  if (st != RS3_OK) return st;
  st = ensure_setup();
  if (st != RS3_OK) return st;
  const LayerDev& ld = L->dev;
  const hipStream_t s = (hipStream_t)stream;
  bool pending = false;
  hipError_t e = rs3_launch_readout(ra, ab, ld.dtype, s, false, &pending);
  if (e == hipSuccess)
    e = pending ? rs3_launch_merge_commit(ra, ca, ld.d_kv, s)
                : rs3_launch_commit(ca, ld.dtype, ld.d_kv, ld.Da, ld.Ha, ld.dah, s);
  if (e != hipSuccess) return map_err(e);
  commit_done(banks, n_obj, pin);
  return RS3_OK;
}

// ---- one frame ------------------------------------------------------------
namespace {
// Layers whose attention, when it projects inside, can take the energy
// launch's projection of every cell: one head of width 64 at d_model 256.
bool frame_qproj_layer(const LayerDev& ld) {
  return ld.dtype == RS3_BF16 && ld.Ha == 1 && ld.Da == 64 && ld.C == 256 && !ld.rope;
}
struct FrameLayout {
  size_t sel, read, q, total;
};
rs3_status frame_layout(const rs3_layer* L, const rs3_grid* g, int32_t n_obj, int64_t x_obj_stride, int32_t max_sel,
                        int32_t n_splits, FrameLayout* fl) {
  size_t sel = 0, read = 0;
  rs3_status st = rs3_select_workspace_size(g, n_obj, x_obj_stride, &sel);
  if (st != RS3_OK) return st;
  st = rs3_readout_workspace_size(L, n_obj, max_sel, n_splits, &read);
  if (st != RS3_OK) return st;
  const int64_t mn = (int64_t)g->m * g->n;
  const int n_x = x_obj_stride ? n_obj : 1;
  fl->sel = align256(sel);
  fl->read = align256(read);
  fl->q = frame_qproj_layer(L->dev) ? align256((size_t)n_x * mn * 64 * 2) : 0;
  fl->total = fl->sel + fl->read + fl->q;
  return RS3_OK;
}
}  // namespace

rs3_status rs3_frame_workspace_size(const rs3_layer* L, const rs3_grid* g, int32_t n_obj, int64_t x_obj_stride,
                                    int32_t max_sel, int32_t n_splits, size_t* bytes) {
  if (!L || !bytes) return RS3_E_INVALID;
  FrameLayout fl;
  rs3_status st = frame_layout(L, g, n_obj, x_obj_stride, max_sel, n_splits, &fl);
  if (st != RS3_OK) return st;
  *bytes = fl.total;
  return RS3_OK;
}

rs3_status rs3_frame(const rs3_layer* L, const rs3_grid* g, int32_t n_obj, rs3_track* tr, rs3_bank* const* banks,
                     const rs3_frame_io* io, void* ws, size_t ws_bytes, void* stream) {
  if (!L || !io || !ws) return RS3_E_INVALID;
  FrameLayout fl;
  rs3_status st = frame_layout(L, g, n_obj, io->x_obj_stride, io->max_sel, io->n_splits, &fl);
  if (st != RS3_OK) return st;
  if (ws_bytes < fl.total) return RS3_E_INVALID;
  uint8_t* w = (uint8_t*)ws;
  const LayerDev& ld = L->dev;
  SelectLaunch sl;
  st = select_args(g, n_obj, io->read_masks, tr, io->X, io->x_obj_stride, ld.C, (rs3_dtype)ld.dtype, io->k,
                   &io->params, w, fl.sel, io->sel_idx, io->sel_count, io->prior_out, sl);
  if (st != RS3_OK) return st;
  const int mn = g->m * g->n;
  Rs3ReadoutArgs ra;
  Rs3AttnBanks ab;
  Rs3CommitArgs ca;
  st = readout_args(L, g, n_obj, io->X, io->x_obj_stride, banks, io->sel_idx, io->sel_count,
                    io->params.union_objects ? 0 : mn, io->max_sel, io->n_splits, io->Y, io->y_obj_stride, io->y_fp32,
                    w + fl.sel, fl.read, ra, ab);
  if (st != RS3_OK) return st;
  st = commit_args(banks, n_obj, g, io->Kmem, io->Vmem, io->kv_obj_stride, io->commit_masks, io->t, io->pin,
                   io->fall_min, io->fall_max, io->kept_count, ca);
  if (st != RS3_OK) return st;
  st = ensure_setup();
  if (st != RS3_OK) return st;
  const hipStream_t s = (hipStream_t)stream;
  Rs3QProjArgs qp;
  const bool pre = fl.q > 0 && io->max_sel > 0 && rs3_attn_projects(ra);
  if (pre) {
    qp.WqT = (const bf16_t*)ld.WqT;
    qp.Qall = (bf16_t*)(w + fl.sel + fl.read);
    qp.qscale = ra.qscale;
    ra.Qall = qp.Qall;
    ra.qall_stride = io->x_obj_stride ? (int64_t)mn * 64 : 0;
  }
  hipError_t e = select_launch(sl, s, pre ? &qp : nullptr);
  bool pending = false;
  if (e == hipSuccess) e = rs3_launch_readout(ra, ab, ld.dtype, s, false, &pending);
  if (e == hipSuccess)
    e = pending ? rs3_launch_merge_commit(ra, ca, ld.d_kv, s)
                : rs3_launch_commit(ca, ld.dtype, ld.d_kv, ld.Da, ld.Ha, ld.dah, s);
  if (e != hipSuccess) return map_err(e);
  commit_done(banks, n_obj, io->pin);
  return RS3_OK;
}

}  // extern "C"

// ---- the memory-attention stack ---------------------------------------------
struct rs3_stack {
  struct Layer {
    const float* ln_g[3];
    const float* ln_b[3];
    const bf16_t* Wqkv;   // packed [256][768]: W_qs | W_ks | W_vs
    const bf16_t* Wos;    // packed [256][256]
    const bf16_t* Wqc;    // packed [256][d_kv]: W_q W_k^T
    const bf16_t* Wvo;    // packed [d_kv][256]: W_v W_o
    const bf16_t* W1;     // packed [256][F]
    const bf16_t* W2;     // packed [F][256]
  };
  int32_t n_layers, C, Hs, dhs, d_kv, F;
  void* dmem;   // every layer's weights, one allocation
  std::vector<Layer> layers;
};

namespace {

// A weight W [K][N] (out = a W) in MFMA B-operand order: for each 32-column
// block nb and 16-deep step ks, 64 lanes x 8 values, lane l holding column
// 32*nb + l%32 and rows 16*ks + 8*(l/32) .. +7.  `at(k, n)` gives bf16 bits.
template <class At>
std::vector<uint8_t> pack_b(int K, int N, At at) {
  std::vector<uint8_t> out((size_t)K * N * 2);
  uint16_t* o = (uint16_t*)out.data();
  const int KS = K / 16;
  for (int nb = 0; nb < N / 32; ++nb)
    for (int ks = 0; ks < KS; ++ks)
      for (int l = 0; l < 64; ++l)
        for (int e = 0; e < 8; ++e)
          o[(((size_t)nb * KS + ks) * 64 + l) * 8 + e] = at(16 * ks + 8 * (l / 32) + e, 32 * nb + l % 32);
  return out;
}

uint16_t bits_at(const void* W, int cols, int k, int n) { return ((const uint16_t*)W)[(size_t)k * cols + n]; }

// Row-major product A [r][k] B [k][c] of bf16 matrices, accumulated in fp64
// and rounded to bf16 (nearest even); b_transposed: B is given as [c][k].
std::vector<uint16_t> product_bits(const void* A, const void* B, int r, int k, int c, bool b_transposed) {
  std::vector<uint16_t> out((size_t)r * c);
  std::vector<uint8_t> tmp(2);
  for (int i = 0; i < r; ++i)
    for (int j = 0; j < c; ++j) {
      double acc = 0.0;
      for (int kk = 0; kk < k; ++kk)
        acc += load_elem(A, (size_t)i * k + kk, RS3_BF16) *
               load_elem(B, b_transposed ? (size_t)j * k + kk : (size_t)kk * c + j, RS3_BF16);
      store_elem(tmp, 0, acc, RS3_BF16);
      memcpy(&out[(size_t)i * c + j], tmp.data(), 2);
    }
  return out;
}

// Hidden units per work-group of the MLP launch: 128 gives F/128 x ceil(M/64)
// work-groups (240 at 957 kept rows and F = 2048), each with half the
// weights of a 256-wide chunk, for twice the fp32 partials.
constexpr int STACK_HC = 128;

// Key splits of the self-attention: a launch of about 256 work-groups
// (8*n_qt*ceil(H_s*S/8)), at least two key tiles per split.
int stack_self_splits(int M, int Hs) {
  const int ntile = (M + KT - 1) / KT, n_qt = (M + 127) / 128;
  int S = n_qt > 0 ? 256 / (n_qt * Hs) : 1;
  const int most = (ntile + 1) / 2;
  if (S > most) S = most;
  if (S * Hs > RS3_MAX_SPLITS_X_HEADS) S = RS3_MAX_SPLITS_X_HEADS / Hs;
  return S < 1 ? 1 : S;
}

struct StackLayout {
  size_t z, zp, part, a1, qs, qc, kh, vh, tiles, desc, hdr, opart, ml, total;
  int S_s, ntile;
};

// Workspace of a call with M kept rows at most and S_c cross-attention splits.
void stack_layout(const rs3_stack* S, int M, int S_c, StackLayout* L) {
  const int C = S->C;
  L->S_s = stack_self_splits(M, S->Hs);
  L->ntile = (M + KT - 1) / KT;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off += align256(bytes);
    return at;
  };
  L->z = take((size_t)M * C * 4);
  L->zp = take((size_t)M * C * 4);
  L->part = take((size_t)(S->F / STACK_HC) * M * C * 4);
  L->a1 = take((size_t)M * C * 2);
  L->qs = take((size_t)M * C * 2);
  L->qc = take((size_t)M * S->d_kv * 2);
  L->kh = take((size_t)L->ntile * KT * C * 2);
  L->vh = take((size_t)L->ntile * KT * C * 2);
  L->tiles = take((size_t)L->ntile * sizeof(TileEnt));
  L->desc = take(sizeof(BankDev));
  L->hdr = take(HDR_WORDS * 4);
  const size_t op_s = (size_t)L->S_s * M * C, op_c = (size_t)S_c * M * S->d_kv;
  L->opart = take((op_s > op_c ? op_s : op_c) * 2);
  const size_t ml_s = (size_t)L->S_s * M * S->Hs, ml_c = (size_t)S_c * M;
  L->ml = take((ml_s > ml_c ? ml_s : ml_c) * 8);
  L->total = off;
}

}  // namespace

extern "C" {

rs3_status rs3_stack_create(int32_t n_layers, int32_t C, int32_t H_s, int32_t d_kv, int32_t F, rs3_dtype dt,
                            const rs3_stack_weights* layers, rs3_stack** out) {
  if (!out || !layers) return RS3_E_INVALID;
  if (n_layers < 1 || n_layers > 16 || C != 256 || d_kv != 64 || dt != RS3_BF16) return RS3_E_INVALID;
  if (H_s != 1 && H_s != 2 && H_s != 4 && H_s != 8) return RS3_E_INVALID;
  if (F < 256 || F > 8192 || F % 256 != 0) return RS3_E_INVALID;
  for (int l = 0; l < n_layers; ++l) {
    const rs3_stack_weights& w = layers[l];
    const void* ptrs[] = {w.ln1_g, w.ln1_b, w.Wqs, w.Wks, w.Wvs, w.Wos, w.ln2_g, w.ln2_b,
                          w.Wq, w.Wk, w.Wv, w.Wo, w.ln3_g, w.ln3_b, w.W1, w.W2};
    for (const void* q : ptrs)
      if (!q) return RS3_E_INVALID;
  }
  *out = nullptr;
  // per layer: QKV, W_os, W_qc, W_vo, W_1, W_2 (bf16), then six norm vectors
  const size_t mats[6] = {(size_t)3 * C * C, (size_t)C * C, (size_t)C * d_kv, (size_t)d_kv * C, (size_t)C * F,
                          (size_t)F * C};
  size_t per = 0;
  for (size_t m : mats) per += align256(m * 2);
  per += 6 * align256((size_t)C * 4);
  std::vector<uint8_t> host(per * n_layers);
  rs3_stack* S = new rs3_stack();
  S->n_layers = n_layers;
  S->C = C;
  S->Hs = H_s;
  S->dhs = C / H_s;
  S->d_kv = d_kv;
  S->F = F;
  S->dmem = nullptr;
  hipError_t e = hipMalloc(&S->dmem, host.size());
  if (e != hipSuccess) {
    delete S;
    return map_err(e);
  }
  uint8_t* dbase = (uint8_t*)S->dmem;
  for (int l = 0; l < n_layers; ++l) {
    const rs3_stack_weights& w = layers[l];
    size_t off = per * l;
    auto put = [&](const std::vector<uint8_t>& src) {
      memcpy(&host[off], src.data(), src.size());
      const uint8_t* d = dbase + off;
      off += align256(src.size());
      return (const bf16_t*)d;
    };
    rs3_stack::Layer L;
    L.Wqkv = put(pack_b(C, 3 * C, [&](int k, int n) {
      const void* W = n < C ? w.Wqs : (n < 2 * C ? w.Wks : w.Wvs);
      return bits_at(W, C, k, n % C);
    }));
    L.Wos = put(pack_b(C, C, [&](int k, int n) { return bits_at(w.Wos, C, k, n); }));
    const std::vector<uint16_t> qc = product_bits(w.Wq, w.Wk, C, C, d_kv, true);    // [C][d_kv]
    const std::vector<uint16_t> vo = product_bits(w.Wv, w.Wo, d_kv, C, C, false);   // [d_kv][C]
    L.Wqc = put(pack_b(C, d_kv, [&](int k, int n) { return qc[(size_t)k * d_kv + n]; }));
    L.Wvo = put(pack_b(d_kv, C, [&](int k, int n) { return vo[(size_t)k * C + n]; }));
    L.W1 = put(pack_b(C, F, [&](int k, int n) { return bits_at(w.W1, F, k, n); }));
    L.W2 = put(pack_b(F, C, [&](int k, int n) { return bits_at(w.W2, C, k, n); }));
    const float* nv[6] = {w.ln1_g, w.ln1_b, w.ln2_g, w.ln2_b, w.ln3_g, w.ln3_b};
    for (int j = 0; j < 6; ++j) {
      std::vector<uint8_t> v((size_t)C * 4);
      memcpy(v.data(), nv[j], v.size());
      const float* d = (const float*)put(v);
      if (j % 2 == 0)
        L.ln_g[j / 2] = d;
      else
        L.ln_b[j / 2] = d;
    }
    S->layers.push_back(L);
  }
  e = hipMemcpy(S->dmem, host.data(), host.size(), hipMemcpyHostToDevice);
  if (e != hipSuccess) {
    (void)hipFree(S->dmem);
    delete S;
    return map_err(e);
  }
  *out = S;
  return RS3_OK;
}

void rs3_stack_destroy(rs3_stack* S) {
  if (!S) return;
  if (S->dmem) (void)hipFree(S->dmem);
  delete S;
}

rs3_status rs3_stack_workspace_size(const rs3_stack* S, int32_t max_sel, int32_t n_splits, size_t* bytes) {
  if (!S || !bytes || max_sel < 0 || max_sel > RS3_MAX_MN || n_splits < 0 || n_splits > RS3_MAX_SPLITS_X_HEADS)
    return RS3_E_INVALID;
  StackLayout L;
  stack_layout(S, max_sel, n_splits > 0 ? n_splits : max_auto_splits(1), &L);
  *bytes = L.total;
  return RS3_OK;
}

rs3_status rs3_stack_readout(const rs3_stack* S, const rs3_grid* g, const void* X, rs3_bank* bank,
                             const int32_t* sel_idx, const int32_t* sel_count, int32_t max_sel, int32_t n_splits,
                             void* Y, int32_t y_fp32, void* ws, size_t ws_bytes, void* stream) {
  if (!S || !grid_ok(g) || !X || !bank || !sel_idx || !sel_count || !Y) return RS3_E_INVALID;
  const int mn = g->m * g->n;
  if (max_sel < 0 || max_sel > mn || n_splits < 0 || n_splits > RS3_MAX_SPLITS_X_HEADS) return RS3_E_INVALID;
  if (y_fp32 != 0 && y_fp32 != 1) return RS3_E_INVALID;
  if (Y == X && y_fp32) return RS3_E_INVALID;
  const LayerDev& bl = bank->L->dev;
  if (!bl.absorb || bl.dtype != RS3_BF16 || bl.C != S->C || bl.d_kv != S->d_kv || bl.rope) return RS3_E_INVALID;
  if (!aligned16(X) || !aligned16(Y) || !aligned16(ws)) return RS3_E_INVALID;
  const int n_qt = (max_sel + 127) / 128;
  const int S_c = n_splits > 0 ? n_splits
                               : auto_splits(1, 1, n_qt > 0 ? n_qt : 1, (double)bank->host.cap * bl.dah * 4);
  StackLayout L;
  stack_layout(S, max_sel, S_c, &L);
  if (max_sel > 0 && (!ws || ws_bytes < L.total)) return RS3_E_INVALID;
  rs3_status st0 = ensure_setup();
  if (st0 != RS3_OK) return st0;
  const hipStream_t st = (hipStream_t)stream;
  hipError_t e = hipSuccess;
  if (Y != X) e = rs3_launch_stack_copy(X, Y, (int64_t)mn * S->C, y_fp32, st);
  if (e != hipSuccess || max_sel == 0) return map_err(e);
  uint8_t* w = (uint8_t*)ws;
  const int C = S->C;
  const double log2e = 1.4426950408889634;

  StkArgs p;
  memset(&p, 0, sizeof(p));
  p.count = sel_count;
  p.err_hdr = bank->host.hdr;
  p.sel = sel_idx;
  p.M = max_sel;
  p.mn = mn;
  p.X = X;
  p.Y = Y;
  p.y_f32 = y_fp32;
  p.Z = (float*)(w + L.z);
  p.Zp = (float*)(w + L.zp);
  p.P = (float*)(w + L.part);
  p.NC = S->F / STACK_HC;
  p.F = S->F;
  p.A1 = (bf16_t*)(w + L.a1);
  p.Qs = (bf16_t*)(w + L.qs);
  p.Qc = (bf16_t*)(w + L.qc);
  p.qscale_s = (float)(log2e / sqrt((double)S->dhs));
  p.qscale_c = (float)(log2e / sqrt((double)C));
  p.Opart = (const bf16_t*)(w + L.opart);
  p.ML = (const float*)(w + L.ml);
  p.Kh = (bf16_t*)(w + L.kh);
  p.Vh = (bf16_t*)(w + L.vh);
  p.tiles = (TileEnt*)(w + L.tiles);
  p.desc = (BankDev*)(w + L.desc);
  p.shdr = (int32_t*)(w + L.hdr);
  p.Hs = S->Hs;
  p.dhs = S->dhs;
  p.ntile_cap = L.ntile;

  // the two attentions: self (the kept rows as a one-frame bank) and cross
  Rs3ReadoutArgs as, ac;
  Rs3AttnBanks abs_, abc;
  memset(&as, 0, sizeof(as));
  memset(&abs_, 0, sizeof(abs_));
  as.banks[0] = p.desc;
  as.sel_count = sel_count;
  as.Q = p.Qs;
  as.Opart = w + L.opart;
  as.ML = (float*)(w + L.ml);
  as.mn = mn;
  as.C = C;
  as.H = S->Hs;
  as.d_h = S->dhs;
  as.D = C;
  as.n_obj = 1;
  as.max_sel = max_sel;
  as.S = L.S_s;
  as.n_qt = n_qt;
  abs_.hdr[0] = p.shdr;
  abs_.tiles[0] = p.tiles;
  abs_.kh[0] = p.Kh;
  abs_.vh[0] = p.Vh;
  abs_.ntcap[0] = L.ntile;
  ac = as;
  ac.banks[0] = bank->d_desc;
  ac.Q = p.Qc;
  ac.H = 1;
  ac.d_h = bl.dah;
  ac.D = bl.Da;
  ac.S = S_c;
  memset(&abc, 0, sizeof(abc));
  abc.hdr[0] = bank->host.hdr;
  abc.tiles[0] = bank->host.tiles;
  abc.kh[0] = bank->host.Khat;
  abc.vh[0] = bank->host.Vhat;
  abc.ntcap[0] = bank->host.n_tiles_cap;

  // gather + the first layer's LN1
  p.ln_g = S->layers[0].ln_g[0];
  p.ln_b = S->layers[0].ln_b[0];
  e = rs3_launch_stack_rows(p, 0, st);
  for (int l = 0; l < S->n_layers && e == hipSuccess; ++l) {
    const rs3_stack::Layer& ly = S->layers[l];
    StkArgs q = p;
    q.Wqkv = ly.Wqkv;
    q.Wos = ly.Wos;
    q.Wqc = ly.Wqc;
    q.Wvo = ly.Wvo;
    q.W1 = ly.W1;
    q.W2 = ly.W2;
    q.ln2_g = ly.ln_g[1];
    q.ln2_b = ly.ln_b[1];
    q.ln3_g = ly.ln_g[2];
    q.ln3_b = ly.ln_b[2];
    q.write_bank = l == 0;
    // z += SA(LN1(z)), then LN2 and the cross-attention's queries
    e = rs3_launch_stack_qkv(q, st);
    if (e == hipSuccess) e = rs3_launch_attn(as, abs_, st, false);
    q.S = L.S_s;
    q.H_att = S->Hs;
    q.d_att = S->dhs;
    q.D_att = C;
    q.mout = p.Qs;   // the merged rows replace the queries the attention has read
    if (e == hipSuccess) e = rs3_launch_stack_merge(q, st);
    if (e == hipSuccess) e = rs3_launch_stack_post_sa(q, st);
    // z += CA(LN2(z)): one absorbed head of width C
    if (e == hipSuccess) e = rs3_launch_attn(ac, abc, st, false);
    q.S = S_c;
    q.H_att = 1;
    q.d_att = S->d_kv;
    q.D_att = S->d_kv;
    q.mout = p.Qc;
    if (e == hipSuccess) e = rs3_launch_stack_merge(q, st);
    // z += relu(LN3(z) W_1) W_2 in hidden chunks, summed with the next LN1
    // (or, after the last layer, with the scatter to Y)
    if (e == hipSuccess) e = rs3_launch_stack_mlp(q, st);
    const bool last = l == S->n_layers - 1;
    if (!last) {
      q.ln_g = S->layers[l + 1].ln_g[0];
      q.ln_b = S->layers[l + 1].ln_b[0];
    }
    if (e == hipSuccess) e = rs3_launch_stack_rows(q, last ? 2 : 1, st);
  }
  return map_err(e);
}

}  // extern "C"
