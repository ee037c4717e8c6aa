// Closure of the decoded masks and the palette argmax (Sec. 3.3; the end of
// Algorithm 1).  Each object's binary mask (logit > 0) is closed with a k x k
// square, a dilation that ignores pixels outside the image followed by an
// erosion that counts them as set; the palette then takes, per pixel, the
// object with the largest logit among those whose closed mask covers it
// (lowest index on ties), 0 where none does.
//
// Three launches over bit-packed masks (bit x%64 of word x/64 of a row):
//   k_post_threshold : one wave per 64-pixel word of a row: per object a
//                      ballot of logit > 0 gives the word; the largest
//                      logit over all objects and its object are kept.  If
//                      that logit is > 0 the object covers the pixel (its
//                      mask is set there and closing only adds), so it is
//                      the palette value; such pixels need no second look.
//   k_post_close     : one work-group per (object, 8-row tile): the bit
//                      rows with a 2r-row halo (k = 2r+1) go to LDS; row
//                      dilation, column dilation, row erosion and column
//                      erosion run on whole words (shifts across the
//                      neighbouring word); writes the closed words and,
//                      when asked, the closed masks as bytes.
//   k_post_palette   : one wave per word: pixels whose largest logit was
//                      > 0 take that object; the others take the largest
//                      logit among the objects whose closed word covers
//                      them (those logits are read only there).
#include "rs3_internal.h"

namespace rs3 {

constexpr int PC_TILE = 8;    // output rows per closing work-group
constexpr int PC_RMAX = 7;    // largest radius (k <= 15)
constexpr int PC_WWMAX = 64;  // words per row (W <= 4096)
constexpr int PC_ROWS = PC_TILE + 4 * PC_RMAX;

__device__ __forceinline__ float logit_at(const bf16_t* p, int64_t i) { return bf2f(p[i]); }
__device__ __forceinline__ float logit_at(const float* p, int64_t i) { return p[i]; }

// grid: ceil(H*WW / 4) work-groups of 4 waves; wave -> (row, word).
template <typename T>
__global__ __launch_bounds__(256) void k_post_threshold(const T* logits, int n_obj, int H, int W, int WW,
                                                        uint64_t* bits, uint8_t* amax) {
  const int lane = threadIdx.x & 63;
  const int64_t word = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (word >= (int64_t)H * WW) return;
  const int y = (int)(word / WW), w = (int)(word - (int64_t)y * WW);
  const int x = 64 * w + lane;
  const bool in = x < W;
  const int64_t plane = (int64_t)H * W;
  const int64_t px = (int64_t)y * W + (in ? x : W - 1);
  float best = -INFINITY;
  int arg = 0;
  for (int o = 0; o < n_obj; ++o) {
    const float v = logit_at(logits, (int64_t)o * plane + px);
    const unsigned long long b = __ballot(in && v > 0.f);
    if (lane == 0) bits[((int64_t)o * H + y) * WW + w] = b;
    if (v > best) {
      best = v;
      arg = o;
    }
  }
  if (in) amax[px] = best > 0.f ? (uint8_t)arg : (uint8_t)0xFF;
}

// Row word w of `row` (WW words, bits past W already at `pad`) shifted so
// that bit x takes bit x - d (d > 0) or x + |d| (d < 0); words outside the
// row read as `pad_word`.
__device__ __forceinline__ uint64_t shifted(const uint64_t* row, int WW, int w, int d, uint64_t pad_word) {
  const uint64_t cur = row[w];
  if (d > 0) {
    const uint64_t lo = w > 0 ? row[w - 1] : pad_word;
    return (cur << d) | (lo >> (64 - d));
  }
  const int e = -d;
  const uint64_t hi = w + 1 < WW ? row[w + 1] : pad_word;
  return (cur >> e) | (hi << (64 - e));
}

// Sixteen mask bits -> sixteen 0/1 bytes.
__device__ __forceinline__ u32x4 bits_to_bytes16(uint32_t h) {
  auto nib = [](uint32_t n) { return (n & 1u) | ((n & 2u) << 7) | ((n & 4u) << 14) | ((n & 8u) << 21); };
  return u32x4{nib(h & 15u), nib((h >> 4) & 15u), nib((h >> 8) & 15u), nib((h >> 12) & 15u)};
}

// grid (ceil(H / PC_TILE), n_obj), block 256.
__global__ __launch_bounds__(256) void k_post_close(const uint64_t* bits, int H, int W, int WW, int r,
                                                    uint64_t* closed_bits, uint8_t* closed, int vec16) {
  __shared__ uint64_t A[PC_ROWS * PC_WWMAX];
  __shared__ uint64_t B[PC_ROWS * PC_WWMAX];
  const int o = blockIdx.y, tid = threadIdx.x;
  const int y0 = blockIdx.x * PC_TILE, y1 = min(H, y0 + PC_TILE);
  const int ya = max(0, y0 - 2 * r), yb = min(H, y1 + 2 * r);   // rows held: [ya, yb)
  const int nr = yb - ya;
  const int rem = W - 64 * (WW - 1);
  const uint64_t tail = rem == 64 ? 0ull : ~0ull << rem;   // bits past W in the last word
  const uint64_t* src = bits + (int64_t)o * H * WW;
  for (int i = tid; i < nr * WW; i += 256) A[i] = src[(int64_t)ya * WW + i];
  __syncthreads();
  // row dilation (outside unset) A -> B
  for (int i = tid; i < nr * WW; i += 256) {
    const int rr = i / WW, w = i - rr * WW;
    const uint64_t* row = A + rr * WW;
    uint64_t v = row[w];
    for (int d = 1; d <= r; ++d) v |= shifted(row, WW, w, d, 0ull) | shifted(row, WW, w, -d, 0ull);
    if (w == WW - 1) v &= ~tail;
    B[i] = v;
  }
  __syncthreads();
  // column dilation B -> A, rows [y0 - r, y1 + r) of the image; the bits
  // past W are set here, so that the erosion counts them as set
  const int ca = max(0, y0 - r), cb = min(H, y1 + r);
  for (int i = tid; i < (cb - ca) * WW; i += 256) {
    const int y = ca + i / WW, w = i - (i / WW) * WW;
    uint64_t v = 0;
    for (int yy = max(0, y - r); yy <= min(H - 1, y + r); ++yy) v |= B[(yy - ya) * WW + w];
    A[(y - ya) * WW + w] = w == WW - 1 ? (v | tail) : v;
  }
  __syncthreads();
  // row erosion (outside set: words past the row read as all set) A -> B
  for (int i = tid; i < (cb - ca) * WW; i += 256) {
    const int y = ca + i / WW, w = i - (i / WW) * WW;
    const uint64_t* row = A + (y - ya) * WW;
    uint64_t v = row[w];
    for (int d = 1; d <= r; ++d) v &= shifted(row, WW, w, d, ~0ull) & shifted(row, WW, w, -d, ~0ull);
    B[(y - ya) * WW + w] = w == WW - 1 ? (v & ~tail) : v;
  }
  __syncthreads();
  // column erosion (outside set) B -> output rows [y0, y1)
  uint64_t* dstb = closed_bits + (int64_t)o * H * WW;
  for (int i = tid; i < (y1 - y0) * WW; i += 256) {
    const int y = y0 + i / WW, w = i - (i / WW) * WW;
    uint64_t v = ~0ull;
    for (int yy = max(0, y - r); yy <= min(H - 1, y + r); ++yy) v &= B[(yy - ya) * WW + w];
    if (w == WW - 1) v &= ~tail;
    dstb[(int64_t)y * WW + w] = v;
    if (closed) {
      uint8_t* dst = closed + ((int64_t)o * H + y) * W + 64 * w;
      const int nb = min(64, W - 64 * w);
      if (vec16) {   // W % 16 == 0 and a 16-byte aligned output
        for (int c = 0; c < nb / 16; ++c) *(u32x4*)(dst + 16 * c) = bits_to_bytes16((uint32_t)(v >> (16 * c)) & 0xffffu);
      } else {
        for (int b = 0; b < nb; ++b) dst[b] = (uint8_t)((v >> b) & 1ull);
      }
    }
  }
}

// grid: ceil(H*WW / 4), block 256 (wave -> (row, word)).
template <typename T>
__global__ __launch_bounds__(256) void k_post_palette(const T* logits, int n_obj, int H, int W, int WW,
                                                      const uint64_t* closed_bits, const uint8_t* amax,
                                                      uint8_t* palette) {
  const int lane = threadIdx.x & 63;
  const int64_t word = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (word >= (int64_t)H * WW) return;
  const int y = (int)(word / WW), w = (int)(word - (int64_t)y * WW);
  const int x = 64 * w + lane;
  if (x >= W) return;
  const int64_t plane = (int64_t)H * W, px = (int64_t)y * W + x;
  const uint8_t a = amax[px];
  if (a != 0xFF) {
    palette[px] = (uint8_t)(a + 1);
    return;
  }
  float best = -INFINITY;
  int arg = -1;
  for (int o = 0; o < n_obj; ++o) {
    const uint64_t cw = closed_bits[((int64_t)o * H + y) * WW + w];
    if ((cw >> lane) & 1ull) {
      const float v = logit_at(logits, (int64_t)o * plane + px);
      if (arg < 0 || v > best) {
        best = v;
        arg = o;
      }
    }
  }
  palette[px] = (uint8_t)(arg + 1);
}

// Eight pixels per lane (rows of W % 8 == 0): one wave covers 512 pixels
// (eight words) of a row.  Each lane loads its 8 logits with 16-byte loads,
// forms 8 mask bits, and the 8 lanes of a word OR their bytes together.
template <typename T>
__device__ __forceinline__ void load8(const T* p, float* v);
template <>
__device__ __forceinline__ void load8<bf16_t>(const bf16_t* p, float* v) {
  const u32x4 w = *(const u32x4*)p;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    v[2 * j] = __uint_as_float(w[j] << 16);
    v[2 * j + 1] = __uint_as_float(w[j] & 0xffff0000u);
  }
}
template <>
__device__ __forceinline__ void load8<float>(const float* p, float* v) {
  const f32x4 a = *(const f32x4*)p, b = *(const f32x4*)(p + 4);
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    v[j] = a[j];
    v[4 + j] = b[j];
  }
}

// grid: ceil(H*G8 / 4) work-groups of 4 waves, G8 = ceil(WW / 8).
template <typename T>
__global__ __launch_bounds__(256) void k_post_threshold8(const T* logits, int n_obj, int H, int W, int WW, int G8,
                                                         uint64_t* bits, uint8_t* amax) {
  const int lane = threadIdx.x & 63;
  const int64_t wid = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (wid >= (int64_t)H * G8) return;
  const int y = (int)(wid / G8), gq = (int)(wid - (int64_t)y * G8);
  const int x0 = 512 * gq + 8 * lane;
  const bool in = x0 < W;   // W % 8 == 0: a lane's 8 pixels are all in or all out
  const int q = 8 * gq + (lane >> 3);
  const int64_t plane = (int64_t)H * W, px = (int64_t)y * W + (in ? x0 : 0);
  float best[8];
  int arg[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    best[j] = -INFINITY;
    arg[j] = 0;
  }
  for (int o = 0; o < n_obj; ++o) {
    float v[8];
    load8<T>(logits + (int64_t)o * plane + px, v);
    uint32_t b8 = 0;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      b8 |= (v[j] > 0.f ? 1u : 0u) << j;
      if (v[j] > best[j]) {
        best[j] = v[j];
        arg[j] = o;
      }
    }
    uint64_t word = in ? (uint64_t)b8 << (8 * (lane & 7)) : 0ull;
    word |= __shfl_xor(word, 1);
    word |= __shfl_xor(word, 2);
    word |= __shfl_xor(word, 4);
    if ((lane & 7) == 0 && q < WW) bits[((int64_t)o * H + y) * WW + q] = word;
  }
  if (in) {
    uint64_t a = 0;
#pragma unroll
    for (int j = 0; j < 8; ++j) a |= (uint64_t)(best[j] > 0.f ? (uint32_t)arg[j] : 0xffu) << (8 * j);
    *(uint64_t*)(amax + px) = a;
  }
}

// grid: ceil(H*G8 / 4), block 256 (8 pixels per lane, W % 8 == 0).
template <typename T>
__global__ __launch_bounds__(256) void k_post_palette8(const T* logits, int n_obj, int H, int W, int WW, int G8,
                                                       const uint64_t* closed_bits, const uint8_t* amax,
                                                       uint8_t* palette) {
  const int lane = threadIdx.x & 63;
  const int64_t wid = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (wid >= (int64_t)H * G8) return;
  const int y = (int)(wid / G8), gq = (int)(wid - (int64_t)y * G8);
  const int x0 = 512 * gq + 8 * lane;
  if (x0 >= W) return;
  const int64_t plane = (int64_t)H * W, px = (int64_t)y * W + x0;
  const uint64_t a8 = *(const uint64_t*)(amax + px);
  uint64_t out = 0;
  uint32_t need = 0;   // pixels whose largest logit is not > 0
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const uint32_t a = (uint32_t)(a8 >> (8 * j)) & 0xffu;
    if (a != 0xffu)
      out |= (uint64_t)(a + 1) << (8 * j);
    else
      need |= 1u << j;
  }
  if (need) {
    const int q = x0 >> 6, sh = x0 & 63;
    float best[8];
    int arg[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      best[j] = -INFINITY;
      arg[j] = -1;
    }
    for (int o = 0; o < n_obj; ++o) {
      const uint32_t cb = (uint32_t)(closed_bits[((int64_t)o * H + y) * WW + q] >> sh) & need;
      if (!cb) continue;
#pragma unroll
      for (int j = 0; j < 8; ++j)
        if ((cb >> j) & 1u) {
          const float v = logit_at(logits, (int64_t)o * plane + px + j);
          if (arg[j] < 0 || v > best[j]) {
            best[j] = v;
            arg[j] = o;
          }
        }
    }
#pragma unroll
    for (int j = 0; j < 8; ++j)
      if ((need >> j) & 1u) out |= (uint64_t)(arg[j] + 1) << (8 * j);
  }
  *(uint64_t*)(palette + px) = out;
}

}  // namespace rs3

using namespace rs3;

size_t rs3_post_workspace_bytes(int n_obj, int H, int W) {
  const size_t WW = (size_t)(W + 63) / 64;
  const size_t words = (size_t)n_obj * H * WW * 8;
  return 2 * ((words + 255) & ~(size_t)255) + (((size_t)H * W + 255) & ~(size_t)255);
}

hipError_t rs3_launch_close_masks(int n_obj, int H, int W, const void* logits, int dtype, int k, uint8_t* closed,
                                  uint8_t* palette, void* ws, hipStream_t st) {
  const int WW = (W + 63) / 64, G8 = (WW + 7) / 8;
  const size_t words = (size_t)n_obj * H * WW * 8;
  uint64_t* bits = (uint64_t*)ws;
  uint64_t* cbits = (uint64_t*)((uint8_t*)ws + ((words + 255) & ~(size_t)255));
  uint8_t* amax = (uint8_t*)ws + 2 * ((words + 255) & ~(size_t)255);
  const int64_t nwords = (int64_t)H * WW, ngroups = (int64_t)H * G8;
  // eight pixels per lane where rows and the logits are 16-byte aligned
  const bool wide = W % 8 == 0 && ((uintptr_t)logits & 15) == 0;
  const dim3 g1((unsigned)((nwords + 3) / 4)), g8((unsigned)((ngroups + 3) / 4));
  const bool bf = dtype == RS3_BF16;
  if (wide && bf)
    hipLaunchKernelGGL(k_post_threshold8<bf16_t>, g8, dim3(256), 0, st, (const bf16_t*)logits, n_obj, H, W, WW, G8,
                       bits, amax);
  else if (wide)
    hipLaunchKernelGGL(k_post_threshold8<float>, g8, dim3(256), 0, st, (const float*)logits, n_obj, H, W, WW, G8,
                       bits, amax);
  else if (bf)
    hipLaunchKernelGGL(k_post_threshold<bf16_t>, g1, dim3(256), 0, st, (const bf16_t*)logits, n_obj, H, W, WW, bits,
                       amax);
  else
    hipLaunchKernelGGL(k_post_threshold<float>, g1, dim3(256), 0, st, (const float*)logits, n_obj, H, W, WW, bits,
                       amax);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int vec16 = closed && W % 16 == 0 && ((uintptr_t)closed & 15) == 0;
  hipLaunchKernelGGL(k_post_close, dim3((unsigned)((H + PC_TILE - 1) / PC_TILE), (unsigned)n_obj), dim3(256), 0, st,
                     bits, H, W, WW, k / 2, cbits, closed, vec16);
  e = hipGetLastError();
  if (e != hipSuccess || !palette) return e;
  const bool wide_out = wide && ((uintptr_t)palette & 7) == 0;
  if (wide_out && bf)
    hipLaunchKernelGGL(k_post_palette8<bf16_t>, g8, dim3(256), 0, st, (const bf16_t*)logits, n_obj, H, W, WW, G8,
                       cbits, amax, palette);
  else if (wide_out)
    hipLaunchKernelGGL(k_post_palette8<float>, g8, dim3(256), 0, st, (const float*)logits, n_obj, H, W, WW, G8, cbits,
                       amax, palette);
  else if (bf)
    hipLaunchKernelGGL(k_post_palette<bf16_t>, g1, dim3(256), 0, st, (const bf16_t*)logits, n_obj, H, W, WW, cbits,
                       amax, palette);
  else
    hipLaunchKernelGGL(k_post_palette<float>, g1, dim3(256), 0, st, (const float*)logits, n_obj, H, W, WW, cbits,
                       amax, palette);
  return hipGetLastError();
}
