// Read-side keep-set: spatial prior (Sec. 3.1, Eqs. 1, 2, 5; tracker update
// of Algorithm 1) and the energy top-k inside it (Eq. 4).
//
// k_energy : e_i = sum_c x_{i,c}^2 in fp64, channels added in ascending
//            order, one lane per token row (the squares of bf16/fp32 values
//            are exact in fp64, so the sums are reproducible bit for bit).
// k_select : one 1024-thread workgroup per group.  Builds the group's prior
//            bitmap in LDS (per-object bbox, streak update, separable
//            Chebyshev dilation), then finds the k-th largest energy with an
//            MSB-first radix select over the fp64 bit patterns (energies are
//            >= 0, so unsigned order is numeric order) and emits the kept
//            cells in ascending order with two ordered block scans.
#include "rs3_internal.h"

namespace rs3 {

constexpr int SEL_THREADS = 1024;
constexpr int SEL_WAVES = SEL_THREADS / 64;

// ---------------------------------------------------------------------------
template <typename T>
__device__ __forceinline__ void load_row_chunk(const T* p, double* v);

template <>
__device__ __forceinline__ void load_row_chunk<bf16_t>(const bf16_t* p, double* v) {
  u32x4 w = *reinterpret_cast<const u32x4*>(p);
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    v[2 * j] = (double)__uint_as_float(w[j] << 16);
    v[2 * j + 1] = (double)__uint_as_float(w[j] & 0xffff0000u);
  }
}

template <>
__device__ __forceinline__ void load_row_chunk<float>(const float* p, double* v) {
  const f32x4* q = reinterpret_cast<const f32x4*>(p);
  f32x4 a = q[0], b = q[1];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    v[j] = (double)a[j];
    v[4 + j] = (double)b[j];
  }
}

// grid (ceil(mn/64), n_x), block 64.  C is a multiple of 8.
template <typename T>
__global__ __launch_bounds__(64) void k_energy(const T* __restrict__ X, int64_t x_stride, int mn,
                                                int C, double* __restrict__ e) {
  const int xi = blockIdx.y;
  const int i = blockIdx.x * 64 + threadIdx.x;
  if (i >= mn) return;
  const T* row = X + (int64_t)xi * x_stride + (int64_t)i * C;
  double acc = 0.0;
  for (int c = 0; c < C; c += 8) {
    double v[8];
    load_row_chunk<T>(row + c, v);
#pragma unroll
    for (int j = 0; j < 8; ++j) acc = acc + v[j] * v[j];
  }
  e[(int64_t)xi * mn + i] = acc;
}

// ---------------------------------------------------------------------------
// block-wide helpers for a 1024-thread workgroup
struct SelShared {
  int red[SEL_WAVES];
  unsigned long long redu[SEL_WAVES];
  int bb[4];
  int mode, r, gy0, gx0, gy1, gx1;
  int hist[256];
  int digit, remaining, full;
};

__device__ __forceinline__ int wave_incl_scan(int v, int lane) {
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    int t = __shfl_up(v, off, 64);
    if (lane >= off) v += t;
  }
  return v;
}

// Exclusive prefix over the workgroup in thread order; returns the prefix
// and writes the total to *total.
__device__ int block_excl_scan(int v, SelShared& sh, int* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int inc = wave_incl_scan(v, lane);
  if (lane == 63) sh.red[wave] = inc;
  __syncthreads();
  int wsum = 0, tot = 0;
  for (int w = 0; w < SEL_WAVES; ++w) {
    int s = sh.red[w];
    if (w < wave) wsum += s;
    tot += s;
  }
  __syncthreads();
  *total = tot;
  return wsum + inc - v;
}

__device__ int block_sum(int v, SelShared& sh) {
  int tot;
  block_excl_scan(v, sh, &tot);
  return tot;
}

__device__ unsigned long long block_minmax_u64(unsigned long long v, bool want_max, SelShared& sh) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    unsigned long long o = __shfl_xor(v, off, 64);
    v = want_max ? (o > v ? o : v) : (o < v ? o : v);
  }
  if (lane == 0) sh.redu[wave] = v;
  __syncthreads();
  unsigned long long r = sh.redu[0];
  for (int w = 1; w < SEL_WAVES; ++w) {
    unsigned long long o = sh.redu[w];
    r = want_max ? (o > r ? o : r) : (o < r ? o : r);
  }
  __syncthreads();
  return r;
}

// ---------------------------------------------------------------------------
enum { MODE_NONE = 0, MODE_MASK = 1, MODE_BOX = 2 };

// Grid rows as bitmasks of W = ceil(n/64) words (bit x%64 of word x/64).
// Used when m*W words fit a 32 KB LDS buffer.
constexpr int BIT_WORDS_MAX = 4096;

// Word w of a row shifted by b >= 1 cells toward higher (left=true: cell x
// takes cell x-b) or lower x.
__device__ __forceinline__ uint64_t row_shift(const uint64_t* row, int W, int w, int b, bool left) {
  const int q = b >> 6, rb = b & 63;
  uint64_t v = 0;
  if (left) {
    if (w - q >= 0) v = row[w - q] << rb;
    if (rb && w - q - 1 >= 0) v |= row[w - q - 1] >> (64 - rb);
  } else {
    if (w + q < W) v = row[w + q] >> rb;
    if (rb && w + q + 1 < W) v |= row[w + q + 1] << (64 - rb);
  }
  return v;
}

__device__ __forceinline__ uint64_t last_word_mask(int n, int W, int w) {
  const int rem = n - 64 * (W - 1);
  return (w == W - 1 && rem < 64) ? ((1ull << rem) - 1ull) : ~0ull;
}

// Adds one object's prior into U (LDS byte map of the group).  bufA/bufB are
// scratch areas of at least max(mn, 8*m*W) bytes.
__device__ void add_object_prior(const Rs3SelectArgs& a, int o, uint8_t* U, uint8_t* bufA, uint8_t* bufB,
                                 SelShared& sh) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int m = a.m, n = a.n, s = a.s, mn = m * n;
  const int Wpx = n * s, Hpx = m * s;
  const uint8_t* M = a.masks + (int64_t)o * Hpx * Wpx;
  if (tid == 0) {
    sh.bb[0] = 0x7fffffff;
    sh.bb[1] = 0x7fffffff;
    sh.bb[2] = -1;
    sh.bb[3] = -1;
  }
  __syncthreads();
  // bounding box of the set pixels: per-thread, then per-wave, then 4 LDS atomics per wave
  int y0 = 0x7fffffff, x0 = 0x7fffffff, y1 = -1, x1 = -1;
  const int npx = Hpx * Wpx;
  for (int p = tid; p < npx; p += SEL_THREADS) {
    if (M[p]) {
      const int y = p / Wpx, x = p - y * Wpx;
      y0 = min(y0, y);
      y1 = max(y1, y);
      x0 = min(x0, x);
      x1 = max(x1, x);
    }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    y0 = min(y0, __shfl_xor(y0, off, 64));
    x0 = min(x0, __shfl_xor(x0, off, 64));
    y1 = max(y1, __shfl_xor(y1, off, 64));
    x1 = max(x1, __shfl_xor(x1, off, 64));
  }
  if (lane == 0 && y1 >= 0) {
    atomicMin(&sh.bb[0], y0);
    atomicMin(&sh.bb[1], x0);
    atomicMax(&sh.bb[2], y1);
    atomicMax(&sh.bb[3], x1);
  }
  __syncthreads();
  if (tid == 0) {
    int32_t* tr = a.track + o * RS3_TRACK_WORDS;
    const bool nonempty = sh.bb[2] >= 0;
    int mode = MODE_NONE, r = a.r_s;
    int by0 = 0, bx0 = 0, by1 = 0, bx1 = 0;
    if (nonempty) {
      by0 = sh.bb[0];
      bx0 = sh.bb[1];
      by1 = sh.bb[2];
      bx1 = sh.bb[3];
      mode = a.seed_box ? MODE_BOX : MODE_MASK;
      tr[0] = by0;
      tr[1] = bx0;
      tr[2] = by1;
      tr[3] = bx1;
      tr[4] = 0;
      tr[5] = 1;
    } else {
      const int d = tr[4] + 1;
      tr[4] = d;
      if (tr[5]) {
        mode = MODE_BOX;
        by0 = tr[0];
        bx0 = tr[1];
        by1 = tr[2];
        bx1 = tr[3];
        r = a.r_s + min(d, a.c);
      }
    }
    sh.mode = mode;
    sh.r = r;
    sh.gy0 = by0 / s;
    sh.gx0 = bx0 / s;
    sh.gy1 = by1 / s;
    sh.gx1 = bx1 / s;
  }
  __syncthreads();
  const int mode = sh.mode, r = sh.r;
  if (mode == MODE_BOX) {
    const int ya = max(0, sh.gy0 - r), yb = min(m - 1, sh.gy1 + r);
    const int xa = max(0, sh.gx0 - r), xb = min(n - 1, sh.gx1 + r);
    for (int i = tid; i < mn; i += SEL_THREADS) {
      const int y = i / n, x = i - y * n;
      if (y >= ya && y <= yb && x >= xa && x <= xb) U[i] = 1;
    }
  } else if (mode == MODE_MASK) {
    const int W = (n + 63) >> 6;
    if (m * W <= BIT_WORDS_MAX) {
      // bitmask path: one wave per row word, ballots form the words
      uint64_t* A = reinterpret_cast<uint64_t*>(bufA);
      uint64_t* B = reinterpret_cast<uint64_t*>(bufB);
      for (int q = wave; q < m * W; q += SEL_WAVES) {
        const int y = q / W, x = 64 * (q - y * W) + lane;
        const bool set = x < n && M[(int64_t)(y * s) * Wpx + x * s] != 0;
        const uint64_t word = __ballot(set);
        if (lane == 0) A[q] = word;
      }
      __syncthreads();
      // row dilation by doubling: OR-ing the shifts by b of a set dilated by
      // a (runs clipped at the row ends included) leaves no gap when
      // b <= a+1, so the radius grows a -> a+b
      uint64_t* src = A;
      uint64_t* dst = B;
      const int rr = min(r, n);
      int done = 0;
      while (done < rr) {
        const int step = min(done + 1, rr - done);
        for (int q = tid; q < m * W; q += SEL_THREADS) {
          const int y = q / W, w = q - y * W;
          const uint64_t* row = src + y * W;
          dst[q] = (row[w] | row_shift(row, W, w, step, true) | row_shift(row, W, w, step, false)) &
                   last_word_mask(n, W, w);
        }
        __syncthreads();
        uint64_t* t = src;
        src = dst;
        dst = t;
        done += step;
      }
      // column dilation, then expand into the byte map
      for (int q = tid; q < m * W; q += SEL_THREADS) {
        const int y = q / W, w = q - y * W;
        const int ya = max(0, y - r), yb = min(m - 1, y + r);
        uint64_t v = 0;
        for (int yy = ya; yy <= yb; ++yy) v |= src[yy * W + w];
        dst[q] = v;
      }
      __syncthreads();
      for (int q = wave; q < m * W; q += SEL_WAVES) {
        const int y = q / W, x = 64 * (q - y * W) + lane;
        if (x < n && (dst[q] >> lane & 1ull)) U[y * n + x] = 1;
      }
    } else {
      // byte path (very tall grids): separable window maxima
      uint8_t* base = bufA;
      uint8_t* tmp = bufB;
      for (int i = tid; i < mn; i += SEL_THREADS) {
        const int y = i / n, x = i - y * n;
        base[i] = M[(int64_t)(y * s) * Wpx + x * s] != 0;
      }
      __syncthreads();
      for (int i = tid; i < mn; i += SEL_THREADS) {
        const int y = i / n, x = i - y * n;
        const uint8_t* row = base + y * n;
        const int xa = max(0, x - r), xb = min(n - 1, x + r);
        uint8_t v = 0;
        for (int xx = xa; xx <= xb; ++xx) v |= row[xx];
        tmp[i] = v;
      }
      __syncthreads();
      for (int i = tid; i < mn; i += SEL_THREADS) {
        const int y = i / n, x = i - y * n;
        const int ya = max(0, y - r), yb = min(m - 1, y + r);
        uint8_t v = 0;
        for (int yy = ya; yy <= yb; ++yy) v |= tmp[yy * n + x];
        if (v) U[i] = 1;
      }
    }
  }
  __syncthreads();
}

// Bytes of each scratch buffer of the select kernel (see add_object_prior).
__host__ __device__ inline int select_buf_bytes(int m, int n) {
  const int W = (n + 63) >> 6;
  const int bits = m * W <= BIT_WORDS_MAX ? 8 * m * W : 0;
  const int bytes = m * n > bits ? m * n : bits;
  return (bytes + 15) & ~15;
}

// grid n_groups, block 1024, dynamic LDS select_lds_bytes().  MAXC bounds the cells
// per thread (mn <= 1024*MAXC); with MAXC <= 16 the energy bit patterns of a
// thread's cells stay in registers, otherwise they are re-read (L2) per pass.
template <int MAXC>
__global__ __launch_bounds__(SEL_THREADS) void k_select(Rs3SelectArgs a) {
  constexpr bool REG = MAXC <= 16;
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  __shared__ SelShared sh;
  const int g = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63;
  const int mn = a.m * a.n;
  const int buf = select_buf_bytes(a.m, a.n);
  uint8_t* U = lds;
  uint8_t* base = lds + ((mn + 15) & ~15);
  uint8_t* tmp = base + buf;

  for (int i = tid; i < mn; i += SEL_THREADS) U[i] = 0;
  __syncthreads();
  if (a.union_objects) {
    for (int o = 0; o < a.n_obj; ++o) add_object_prior(a, o, U, base, tmp, sh);
  } else {
    add_object_prior(a, g, U, base, tmp, sh);
  }
  if (a.prior_out) {
    for (int i = tid; i < mn; i += SEL_THREADS) a.prior_out[(int64_t)g * mn + i] = U[i];
  }

  // Contiguous cells per thread so that block scans follow cell order.
  const int cpt = (mn + SEL_THREADS - 1) / SEL_THREADS;
  const int c0 = tid * cpt;
  const unsigned long long* ebits =
      reinterpret_cast<const unsigned long long*>(a.e + (a.x_per_obj ? (int64_t)g * mn : 0)) + c0;
  uint32_t inP = 0;
  unsigned long long kreg[REG ? MAXC : 1];
#pragma unroll
  for (int j = 0; j < MAXC; ++j) {
    const int i = c0 + j;
    const bool in = j < cpt && i < mn && U[i];
    if (in) inP |= 1u << j;
    if (REG) kreg[REG ? j : 0] = in ? ebits[j] : 0ull;
  }
  auto key_of = [&](int j) -> unsigned long long { return REG ? kreg[REG ? j : 0] : ebits[j]; };
  const int k = a.k[g];
  const int countP = block_sum(__popc(inP), sh);
  uint32_t keep = inP;
  if (countP > k) {
    unsigned long long lo = ~0ull, hi = 0;
#pragma unroll
    for (int j = 0; j < MAXC; ++j)
      if (inP >> j & 1) {
        const unsigned long long key = key_of(j);
        lo = key < lo ? key : lo;
        hi = key > hi ? key : hi;
      }
    const unsigned long long kmin = block_minmax_u64(lo, false, sh);
    const unsigned long long kmax = block_minmax_u64(hi, true, sh);
    // Result: keep keys > T, plus the first need_eq keys == T in cell order;
    // or (ge) keep every key >= T.
    unsigned long long T;
    int need_eq = 0;
    bool ge = false;
    if (k == 0) {
      T = ~0ull;
      ge = false;
    } else if (kmin == kmax) {
      T = kmin;
      need_eq = k;
    } else {
      const int h = 63 - __clzll(kmin ^ kmax);
      unsigned long long prefix = (h == 63) ? 0ull : (kmin & ~((2ull << h) - 1ull));
      int remaining = k;
      int top = h;
      while (top >= 0) {
        const int width = top + 1 < 8 ? top + 1 : 8;
        const int shift = top - width + 1;
        const unsigned dmask = (1u << width) - 1u;
        for (int bb = tid; bb < 256; bb += SEL_THREADS) sh.hist[bb] = 0;
        __syncthreads();
#pragma unroll
        for (int j = 0; j < MAXC; ++j) {
          if (inP >> j & 1) {
            const unsigned long long key = key_of(j);
            const bool match = (top >= 63) || (((key ^ prefix) >> (top + 1)) == 0ull);
            if (match) atomicAdd(&sh.hist[(unsigned)(key >> shift) & dmask], 1);
          }
        }
        __syncthreads();
        if (tid < 64) {
          // lane owns bins 4*lane .. 4*lane+3; find the digit holding the
          // remaining-th largest candidate
          const int h0 = sh.hist[4 * lane], h1 = sh.hist[4 * lane + 1];
          const int h2 = sh.hist[4 * lane + 2], h3 = sh.hist[4 * lane + 3];
          const int mine = h0 + h1 + h2 + h3;
          int suf = mine;  // inclusive suffix sum over lanes >= lane
#pragma unroll
          for (int off = 1; off < 64; off <<= 1) {
            const int t = __shfl_down(suf, off, 64);
            if (lane + off < 64) suf += t;
          }
          const int above = suf - mine;  // candidates in bins of higher lanes
          const int want = remaining;
          if (above < want && want <= suf) {
            const int hb[4] = {h0, h1, h2, h3};
            int cum = above;
            for (int bb = 3; bb >= 0; --bb) {
              if (cum + hb[bb] >= want) {
                sh.digit = 4 * lane + bb;
                sh.remaining = want - cum;
                sh.full = (cum + hb[bb] == want);
                break;
              }
              cum += hb[bb];
            }
          }
        }
        __syncthreads();
        prefix |= (unsigned long long)sh.digit << shift;
        remaining = sh.remaining;
        const bool full = sh.full;
        __syncthreads();
        if (full) {
          // every candidate with this prefix is kept: keep keys >= prefix
          ge = true;
          break;
        }
        top = shift - 1;
      }
      T = prefix;
      need_eq = remaining;
    }
    uint32_t eq = 0, gt = 0;
#pragma unroll
    for (int j = 0; j < MAXC; ++j)
      if (inP >> j & 1) {
        const unsigned long long key = key_of(j);
        if (ge ? key >= T : (key > T && T != ~0ull)) gt |= 1u << j;
        if (!ge && key == T) eq |= 1u << j;
      }
    keep = gt;
    if (!ge && k > 0) {
      int eqTot;
      int eqBefore = block_excl_scan(__popc(eq), sh, &eqTot);
#pragma unroll
      for (int j = 0; j < MAXC; ++j) {
        if (eq >> j & 1) {
          if (eqBefore < need_eq) keep |= 1u << j;
          ++eqBefore;
        }
      }
    }
  }
  int total;
  int before = block_excl_scan(__popc(keep), sh, &total);
  int32_t* out = a.sel_idx + (int64_t)g * mn;
#pragma unroll
  for (int j = 0; j < MAXC; ++j)
    if (keep >> j & 1) out[before++] = c0 + j;
  if (tid == 0) a.sel_count[g] = total;
}

}  // namespace rs3

using namespace rs3;

hipError_t rs3_launch_energy(const void* X, int64_t x_stride, int n_x, int mn, int C, int dtype,
                             double* e, hipStream_t st) {
  dim3 grid((mn + 63) / 64, n_x);
  if (dtype == RS3_BF16)
    RS3_LAUNCH(RS3_K_ENERGY, st, k_energy<bf16_t>, grid, dim3(64), 0, st, (const bf16_t*)X, x_stride, mn, C, e);
  else
    RS3_LAUNCH(RS3_K_ENERGY, st, k_energy<float>, grid, dim3(64), 0, st, (const float*)X, x_stride, mn, C, e);
  return hipGetLastError();
}

static size_t select_lds_bytes(int m, int n) {
  return (size_t)((m * n + 15) & ~15) + 2 * (size_t)select_buf_bytes(m, n);
}

hipError_t rs3_select_setup() {
  // largest layout: mn = RS3_MAX_MN with byte-sized buffers (3 * 32 KB)
  const int mx = 3 * RS3_MAX_MN + 64;
  hipError_t e = hipFuncSetAttribute((const void*)k_select<16>, hipFuncAttributeMaxDynamicSharedMemorySize, mx);
  if (e != hipSuccess) return e;
  return hipFuncSetAttribute((const void*)k_select<32>, hipFuncAttributeMaxDynamicSharedMemorySize, mx);
}

hipError_t rs3_launch_select(const Rs3SelectArgs& a, int n_groups, hipStream_t st) {
  const int mn = a.m * a.n;
  const size_t lds = select_lds_bytes(a.m, a.n);
  if (mn <= 16 * SEL_THREADS)
    RS3_LAUNCH(RS3_K_SELECT, st, k_select<16>, dim3(n_groups), dim3(SEL_THREADS), lds, st, a);
  else
    RS3_LAUNCH(RS3_K_SELECT, st, k_select<32>, dim3(n_groups), dim3(SEL_THREADS), lds, st, a);
  return hipGetLastError();
}
