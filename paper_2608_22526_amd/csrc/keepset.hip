// The paper's fixed write keep-set (Sec. 3.2, Eq. 8): every object's seed
// mask (its mask in the frame where it is first seen) is sampled onto the
// encoder grid and grown by D_w cells (Chebyshev distance); K_w collects the
// cells of all objects.  It
// is computed once per sequence; every later write stores the tokens at K_w,
// so every stored frame has the same length.  When the undilated footprint
// count is below fall_min or above fall_max the write falls through to the
// dense path (every cell kept).
//
// k_write_keepset: one 1024-thread work-group.  The footprint is built in LDS
// as bytes; the dilation is separable: a cell is kept by the row pass when
// the nearest footprint cell of its row (scanning left and right, one thread
// per row) is within D_w, and by the column pass likewise on the row result.
// The keep-set is written n_copies times (so that it can serve as the mask of
// n_copies objects in one commit).
#include "rs3_internal.h"

namespace rs3 {

constexpr int KW_THREADS = 1024;

__global__ __launch_bounds__(KW_THREADS) void k_write_keepset(const uint8_t* seed, int n_obj, int m, int n, int s,
                                                              int D, int fall_min, int fall_max, int n_copies,
                                                              uint8_t* keep, int32_t* counts) {
  __shared__ uint8_t foot[RS3_MAX_MN];
  __shared__ uint8_t rowk[RS3_MAX_MN];
  __shared__ int tot[2];
  const int tid = threadIdx.x;
  const int mn = m * n, Wpx = n * s;
  const int64_t obj_px = (int64_t)m * s * Wpx;
  if (tid < 2) tot[tid] = 0;
  __syncthreads();
  // footprint: union of the down-sampled seed masks (cell (y, x) samples
  // pixel (y*s, x*s))
  int cnt = 0;
  for (int i = tid; i < mn; i += KW_THREADS) {
    const int y = i / n, x = i - y * n;
    const int64_t px = (int64_t)(y * s) * Wpx + (int64_t)x * s;
    uint8_t v = 0;
    for (int o = 0; o < n_obj; ++o) v |= seed[o * obj_px + px] ? 1 : 0;
    foot[i] = v;
    cnt += v;
  }
  atomicAdd(&tot[0], cnt);
  __syncthreads();
  const int footprint = tot[0];
  const bool dense = footprint < fall_min || footprint > fall_max;
  if (!dense) {
    // row pass: distance to the nearest footprint cell of the row
    for (int y = tid; y < m; y += KW_THREADS) {
      const uint8_t* f = foot + y * n;
      uint8_t* r = rowk + y * n;
      int last = -1;   // last set cell at or left of x
      for (int x = 0; x < n; ++x) {
        if (f[x]) last = x;
        r[x] = (last >= 0 && x - last <= D) ? 1 : 0;
      }
      int next = -1;   // next set cell at or right of x
      for (int x = n - 1; x >= 0; --x) {
        if (f[x]) next = x;
        if (next >= 0 && next - x <= D) r[x] = 1;
      }
    }
    __syncthreads();
    // column pass on the row result, into foot
    for (int x = tid; x < n; x += KW_THREADS) {
      int last = -1;
      for (int y = 0; y < m; ++y) {
        if (rowk[y * n + x]) last = y;
        foot[y * n + x] = (last >= 0 && y - last <= D) ? 1 : 0;
      }
      int next = -1;
      for (int y = m - 1; y >= 0; --y) {
        if (rowk[y * n + x]) next = y;
        if (next >= 0 && next - y <= D) foot[y * n + x] = 1;
      }
    }
    __syncthreads();
  }
  int kept = 0;
  for (int i = tid; i < mn; i += KW_THREADS) {
    const uint8_t v = dense ? 1 : foot[i];
    kept += v;
    for (int c = 0; c < n_copies; ++c) keep[(int64_t)c * mn + i] = v;
  }
  atomicAdd(&tot[1], kept);
  __syncthreads();
  if (tid == 0 && counts) {
    counts[0] = footprint;
    counts[1] = tot[1];
  }
}

}  // namespace rs3

using namespace rs3;

hipError_t rs3_launch_write_keepset(const uint8_t* seed, int n_obj, int m, int n, int s, int D, int fall_min,
                                    int fall_max, int n_copies, uint8_t* keep, int32_t* counts, hipStream_t st) {
  hipLaunchKernelGGL(k_write_keepset, dim3(1), dim3(KW_THREADS), 0, st, seed, n_obj, m, n, s, D, fall_min, fall_max,
                     n_copies, keep, counts);
  return hipGetLastError();
}
