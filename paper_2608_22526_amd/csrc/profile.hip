// Optional per-kernel timing with HIP events.  When enabled, every kernel the
// library launches carries a pair of events that the runtime stamps with the
// kernel's own start and end (hipExtLaunchKernelGGL);
// rs3_profile_report() waits for them and returns per-kernel totals.
// The event pool is created at enable time, so timed calls allocate nothing.
#include <vector>

#include "rs3_internal.h"

namespace {

using rs3::u32x4;

// Read-only stream: grid-stride 16-byte loads, four in flight per thread,
// xor-reduced to one word per thread.
__global__ __launch_bounds__(256) void k_stream_read(const u32x4* __restrict__ src, size_t n16,
                                                     uint32_t* __restrict__ out) {
  const size_t tid = (size_t)blockIdx.x * 256 + threadIdx.x, nth = (size_t)gridDim.x * 256;
  uint32_t x = 0;
  size_t i = tid;
  for (; i + 3 * nth < n16; i += 4 * nth) {
    u32x4 v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) v[u] = src[i + u * nth];
#pragma unroll
    for (int u = 0; u < 4; ++u) x ^= v[u][0] ^ v[u][1] ^ v[u][2] ^ v[u][3];
  }
  for (; i < n16; i += nth) {
    const u32x4 v = src[i];
    x ^= v[0] ^ v[1] ^ v[2] ^ v[3];
  }
  out[tid] = x;
}

struct Rec {
  int id;
  int ev;  // index of the start event; ev+1 is the stop event
};

struct ProfState {
  bool on = false;
  std::vector<hipEvent_t> ev;
  std::vector<Rec> recs;
  int next = 0;
  double total_ms[RS3_K_COUNT] = {};
  int64_t count[RS3_K_COUNT] = {};
  int64_t dropped = 0;
};

ProfState P;

hipError_t fold() {
  for (const Rec& r : P.recs) {
    hipError_t e = hipEventSynchronize(P.ev[r.ev + 1]);
    if (e != hipSuccess) return e;
    float ms = 0.f;
    e = hipEventElapsedTime(&ms, P.ev[r.ev], P.ev[r.ev + 1]);
    if (e != hipSuccess) return e;
    P.total_ms[r.id] += ms;
    P.count[r.id] += 1;
  }
  P.recs.clear();
  P.next = 0;
  return hipSuccess;
}

}  // namespace

bool rs3_prof_events(int id, hipEvent_t* start, hipEvent_t* stop) {
  if (!P.on) return false;
  if (P.next + 2 > (int)P.ev.size()) {
    ++P.dropped;
    return false;
  }
  *start = P.ev[P.next];
  *stop = P.ev[P.next + 1];
  P.recs.push_back(Rec{id, P.next});
  P.next += 2;
  return true;
}

extern "C" {

rs3_status rs3_profile_enable(int32_t on, int32_t max_launches) {
  if (on) {
    if (max_launches <= 0 || max_launches > (1 << 20)) return RS3_E_INVALID;
    if ((int)P.ev.size() < 2 * max_launches) {
      for (hipEvent_t e : P.ev) (void)hipEventDestroy(e);
      P.ev.assign(2 * max_launches, nullptr);
      for (auto& e : P.ev)
        if (hipEventCreate(&e) != hipSuccess) return RS3_E_DEVICE;
    }
    P.recs.reserve(max_launches);
  }
  P.on = on != 0;
  return RS3_OK;
}

rs3_status rs3_profile_report(double* total_ms, int64_t* launches, int64_t* dropped) {
  if (!total_ms || !launches) return RS3_E_INVALID;
  if (fold() != hipSuccess) return RS3_E_DEVICE;
  for (int i = 0; i < RS3_K_COUNT; ++i) {
    total_ms[i] = P.total_ms[i];
    launches[i] = P.count[i];
  }
  if (dropped) *dropped = P.dropped;
  return RS3_OK;
}

rs3_status rs3_stream_read(const void* src, size_t bytes, uint32_t* out, void* stream) {
  if (!src || !out || ((uintptr_t)src & 15u) || (bytes & 15u)) return RS3_E_INVALID;
  const hipStream_t st = (hipStream_t)stream;
  hipLaunchKernelGGL(k_stream_read, dim3(RS3_STREAM_READ_THREADS / 256), dim3(256), 0, st, (const u32x4*)src,
                     bytes / 16, out);
  return hipGetLastError() == hipSuccess ? RS3_OK : RS3_E_DEVICE;
}

rs3_status rs3_profile_reset(void) {
  if (fold() != hipSuccess) return RS3_E_DEVICE;
  for (int i = 0; i < RS3_K_COUNT; ++i) {
    P.total_ms[i] = 0.0;
    P.count[i] = 0;
  }
  P.dropped = 0;
  return RS3_OK;
}

}  // extern "C"
