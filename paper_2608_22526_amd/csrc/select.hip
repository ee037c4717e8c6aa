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
constexpr int SEL_RANK_BYTES = SEL_THREADS * (8 + 4 + 4);

// ---------------------------------------------------------------------------
// Energy of a row chunk (16 bytes: 8 bf16 or 4 fp32 channels) continued in
// ascending channel order.  Squares of bf16 and fp32 values are exact in
// fp64, so the fused multiply-add rounds exactly like the sum of the
// definition (acc + x*x).
template <typename T>
__device__ __forceinline__ double energy_chunk(u32x4 w, double acc);

template <>
__device__ __forceinline__ double energy_chunk<bf16_t>(u32x4 w, double acc) {
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const double lo = (double)__uint_as_float(w[j] << 16), hi = (double)__uint_as_float(w[j] & 0xffff0000u);
    acc = fma(lo, lo, acc);
    acc = fma(hi, hi, acc);
  }
  return acc;
}

template <>
__device__ __forceinline__ double energy_chunk<float>(u32x4 w, double acc) {
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const double v = (double)__uint_as_float(w[j]);
    acc = fma(v, v, acc);
  }
  return acc;
}

// grid (ceil(mn/64), n_x), block 256.  The block's 64 rows (contiguous in X)
// are read in column blocks of EB_CH 16-byte chunks per row with coalesced
// loads into LDS (row pitch EB_CH + 1 chunks: the per-row reads below are
// conflict-free), then lane r of wave 0 continues row r's sum.  Also writes
// the smallest and largest energy bit pattern of the block's rows to
// range[xi][block] (energies are >= 0, so bit order is numeric order).
// C*sizeof(T) is a multiple of 16.
constexpr int EB_CH = 32;
// Rows 64*bx .. of grid xi by one 256-thread block (nbx blocks per grid).
// QP (bf16 rows of 256 channels, so the block holds whole rows): waves 1 and
// 2 also project rows 0-31 and 32-63 of the block by W_q on MFMA while wave
// 0 continues the energy chains, and store them, scaled, to qp.Qall.  They
// load their W_q operands after the block's barrier, so the chains start as
// early as without the projection.
template <typename T, bool QP = false>
__device__ __forceinline__ void energy_block(const T* __restrict__ X, int64_t x_stride, int mn, int C,
                                             double* __restrict__ e, unsigned long long* __restrict__ range,
                                             int bx, int xi, int nbx, const Rs3QProjArgs* qp = nullptr) {
  __shared__ u32x4 rows[64 * (EB_CH + 1)];
  const int r0 = bx * 64, tid = threadIdx.x;
  const int nrows = min(64, mn - r0);
  const int cpr = C * (int)sizeof(T) / 16;   // chunks per row
  const u32x4* src = (const u32x4*)(X + (int64_t)xi * x_stride + (int64_t)r0 * C);
  double acc = 0.0;
  for (int cb = 0; cb < cpr; cb += EB_CH) {
    const int nch = min(EB_CH, cpr - cb);
    // chunk q = tid + 256 k of the 64 x nch block (every load issued before
    // the first LDS write; rows past the grid re-read its last row)
    u32x4 v[64 * EB_CH / 256];
#pragma unroll
    for (int k = 0; k < 64 * EB_CH / 256; ++k) {
      const int q = min(tid + 256 * k, 64 * nch - 1);
      const int r = q / nch, c = q - r * nch;
      v[k] = src[(int64_t)min(r, nrows - 1) * cpr + cb + c];
    }
#pragma unroll
    for (int k = 0; k < 64 * EB_CH / 256; ++k) {
      const int q = tid + 256 * k;
      if (q < 64 * nch) {
        const int r = q / nch, c = q - r * nch;
        rows[r * (EB_CH + 1) + c] = v[k];
      }
    }
    __syncthreads();
    if (tid < 64) {
      const u32x4* rw = rows + tid * (EB_CH + 1);
#pragma unroll 4
      for (int c = 0; c < nch; ++c) acc = energy_chunk<T>(rw[c], acc);
    } else if constexpr (QP) {
      if (tid < 192) {
        // wave 1 + w: rows 32w .. 32w+31; A = W_q^T rows (d), B = X rows; lane
        // l ends with row 32w + l%32 at d = 32 db + 8 (r/4) + 4 (l/32) + r%4
        const int w = (tid >> 6) - 1, lane = tid & 63, g = lane >> 5;
        const u32x4* xb = rows + (32 * w + (lane & 31)) * (EB_CH + 1) + g;
        // A operands: W_q^T rows 32 db + lane%32, chunk 2 ks + lane/32
        const u32x4* wg = (const u32x4*)qp->WqT + (lane & 31) * EB_CH + g;
        u32x4 wa[2][EB_CH / 2];
#pragma unroll
        for (int db = 0; db < 2; ++db)
#pragma unroll
          for (int ks = 0; ks < EB_CH / 2; ++ks) wa[db][ks] = wg[db * 32 * EB_CH + 2 * ks];
        f32x16 qa[2] = {f32x16{}, f32x16{}};
#pragma unroll
        for (int ks = 0; ks < EB_CH / 2; ++ks) {
          const u32x4 bx = xb[2 * ks];
#pragma unroll
          for (int db = 0; db < 2; ++db) qa[db] = mfma32(wa[db][ks], bx, qa[db]);
        }
        const int row = 32 * w + (lane & 31);
        if (row < nrows) {
          bf16_t* qrow = qp->Qall + ((int64_t)xi * mn + r0 + row) * 64;
          const float qs = qp->qscale;
#pragma unroll
          for (int db = 0; db < 2; ++db)
#pragma unroll
            for (int q4 = 0; q4 < 4; ++q4) {
              u32x2 pk;
              pk[0] = pack_bf16x2(qa[db][4 * q4] * qs, qa[db][4 * q4 + 1] * qs);
              pk[1] = pack_bf16x2(qa[db][4 * q4 + 2] * qs, qa[db][4 * q4 + 3] * qs);
              *(u32x2*)(qrow + 32 * db + 8 * q4 + 4 * g) = pk;
            }
        }
      }
    }
    __syncthreads();
  }
  if (tid >= 64) return;
  unsigned long long lo = ~0ull, hi = 0ull;
  if (tid < nrows) {
    e[(int64_t)xi * mn + r0 + tid] = acc;
    lo = hi = (unsigned long long)__double_as_longlong(acc);
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    const unsigned long long ol = __shfl_xor(lo, off, 64), oh = __shfl_xor(hi, off, 64);
    lo = ol < lo ? ol : lo;
    hi = oh > hi ? oh : hi;
  }
  if (tid == 0) {
    unsigned long long* r = range + 2 * ((int64_t)xi * nbx + bx);
    r[0] = lo;
    r[1] = hi;
  }
}

// Wide form for large batches (no projection): 256 rows per 256-thread
// block, one row per thread, read in column slices of EW_CH 16-byte chunks
// per row with coalesced loads through LDS (row pitch EW_CH + 1 chunks).
// The next slice's loads are issued before the current slice's sums, so the
// loads run under the four waves' sums, and every wave sums (the 64-row
// form sums in one wave while three wait).  Each wave writes the smallest
// and largest energy bits of its 64 rows to range[xi][64-row block], the
// layout of the 64-row form.
constexpr int EW_CH = 8;
constexpr int EW_ROWS = 256;
template <typename T>
__device__ __forceinline__ void energy_block_wide(const T* __restrict__ X, int64_t x_stride, int mn, int C,
                                                  double* __restrict__ e, unsigned long long* __restrict__ range,
                                                  int bx, int xi) {
  __shared__ u32x4 rows[EW_ROWS * (EW_CH + 1)];
  const int r0 = bx * EW_ROWS, tid = threadIdx.x;
  const int nrows = min(EW_ROWS, mn - r0);
  const int cpr = C * (int)sizeof(T) / 16;   // chunks per row
  const int npass = (cpr + EW_CH - 1) / EW_CH;
  const u32x4* src = (const u32x4*)(X + (int64_t)xi * x_stride + (int64_t)r0 * C);
  // slot q = tid + 256 k of the slice at chunk cb: row q / EW_CH, chunk
  // q % EW_CH (chunks past a short last slice, and rows past the grid,
  // re-read its last chunk and row)
  u32x4 v[EW_CH];
  auto load = [&](int cb) {
    const int nch = min(EW_CH, cpr - cb);
#pragma unroll
    for (int k = 0; k < EW_CH; ++k) {
      const int q = tid + EW_ROWS * k;
      const int r = q / EW_CH, c = q % EW_CH;
      v[k] = src[(int64_t)min(r, nrows - 1) * cpr + cb + min(c, nch - 1)];
    }
  };
  double acc = 0.0;
  load(0);
  for (int pass = 0; pass < npass; ++pass) {
    const int cb = pass * EW_CH, nch = min(EW_CH, cpr - cb);
    if (pass > 0) __syncthreads();   // every row of the previous slice has been summed
#pragma unroll
    for (int k = 0; k < EW_CH; ++k) {
      const int q = tid + EW_ROWS * k;
      const int r = q / EW_CH, c = q % EW_CH;
      if (c < nch) rows[r * (EW_CH + 1) + c] = v[k];
    }
    __syncthreads();
    if (pass + 1 < npass) load(cb + EW_CH);
    const u32x4* rw = rows + tid * (EW_CH + 1);
    if (nch == EW_CH) {
#pragma unroll
      for (int c = 0; c < EW_CH; ++c) acc = energy_chunk<T>(rw[c], acc);
    } else {
      for (int c = 0; c < nch; ++c) acc = energy_chunk<T>(rw[c], acc);
    }
  }
  unsigned long long lo = ~0ull, hi = 0ull;
  if (tid < nrows) {
    e[(int64_t)xi * mn + r0 + tid] = acc;
    lo = hi = (unsigned long long)__double_as_longlong(acc);
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    const unsigned long long ol = __shfl_xor(lo, off, 64), oh = __shfl_xor(hi, off, 64);
    lo = ol < lo ? ol : lo;
    hi = oh > hi ? oh : hi;
  }
  const int w = tid >> 6;
  if ((tid & 63) == 0 && 64 * w < nrows) {
    unsigned long long* r = range + 2 * ((int64_t)xi * ((mn + 63) >> 6) + (r0 >> 6) + w);
    r[0] = lo;
    r[1] = hi;
  }
}

template <typename T>
__global__ __launch_bounds__(256) void k_energy_wide(const T* __restrict__ X, int64_t x_stride, int mn, int C,
                                                     double* __restrict__ e, unsigned long long* __restrict__ range) {
  energy_block_wide<T>(X, x_stride, mn, C, e, range, blockIdx.x, blockIdx.y);
}

template <typename T, bool QP = false>
__global__ __launch_bounds__(256) void k_energy(const T* __restrict__ X, int64_t x_stride, int mn,
                                                 int C, double* __restrict__ e,
                                                 unsigned long long* __restrict__ range, Rs3QProjArgs qp) {
  energy_block<T, QP>(X, x_stride, mn, C, e, range, blockIdx.x, blockIdx.y, gridDim.x, &qp);
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
  int ncand;
  int red1[SEL_WAVES], red2[SEL_WAVES], red3[SEL_WAVES];
  unsigned long long rowbits[SEL_WAVES];   // rows with a set cell, one bit per row
  unsigned long long colbits[4];           // columns with a set cell
  unsigned long long kmin, kmax;
};

// Exclusive prefix (in thread order) of the number of set bits among the
// first cpt bits of `bits`, and the workgroup total; `red` is a private
// SEL_WAVES-entry LDS array of the call site.  Ballot-based: no LDS or
// cross-lane permutes inside a wave.
template <int MAXC>
__device__ __forceinline__ int block_scan_bits(uint32_t bits, int cpt, int* red, int* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int pre = 0, wtot = 0;
#pragma unroll
  for (int j = 0; j < MAXC; ++j)
    if (j < cpt) {
      const unsigned long long b = __ballot((bits >> j) & 1u);
      pre += __builtin_amdgcn_mbcnt_hi((uint32_t)(b >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)b, 0u));
      wtot += __popcll(b);
    }
  if (lane == 0) red[wave] = wtot;
  lds_barrier();
  int before = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < SEL_WAVES; ++w) {
    const int v = red[w];
    tot += v;
    before += w < wave ? v : 0;
  }
  *total = tot;
  return before + pre;
}

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

// One wave: the bin of sh.hist (256 bins, higher bins hold larger keys) that
// holds the want-th largest candidate -> sh.digit, the rank of that candidate
// inside its bin -> sh.remaining, and whether the bin is taken whole -> sh.full.
__device__ void find_digit(SelShared& sh, int want, int lane) {
  // lane owns bins 4*lane .. 4*lane+3
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

// Tracker update of object o (single thread) from the box of its set pixels
// (y1 < 0: empty mask), on the LDS copy of its words; writes the words back
// and publishes the prior mode, radius and grid box in sh.
__device__ void tracker_update(const Rs3SelectArgs& a, int o, int* tl, int by0, int bx0, int by1, int bx1,
                               SelShared& sh) {
  int32_t* tr = a.track + o * RS3_TRACK_WORDS;
  const bool nonempty = by1 >= 0;
  int mode = MODE_NONE, r = a.r_s;
  if (nonempty) {
    mode = a.seed_box ? MODE_BOX : MODE_MASK;
    tl[0] = by0;
    tl[1] = bx0;
    tl[2] = by1;
    tl[3] = bx1;
    tl[4] = 0;
    tl[5] = 1;
  } else {
    const int d = tl[4] + 1;
    tl[4] = d;
    if (tl[5]) {
      mode = MODE_BOX;
      by0 = tl[0];
      bx0 = tl[1];
      by1 = tl[2];
      bx1 = tl[3];
      r = a.r_s + min(d, a.c);
    }
  }
  for (int w = 0; w < RS3_TRACK_WORDS; ++w) tr[w] = tl[w];
  sh.mode = mode;
  sh.r = r;
  const int s = a.s;
  if (mode == MODE_NONE) by0 = bx0 = by1 = bx1 = 0;
  sh.gy0 = s == 1 ? by0 : by0 / s;
  sh.gx0 = s == 1 ? bx0 : bx0 / s;
  sh.gy1 = s == 1 ? by1 : by1 / s;
  sh.gx1 = s == 1 ? bx1 : bx1 / s;
}

// Register path of the prior: grids of at most SEL_THREADS rows and
// FAST_W*64 columns.  Thread y owns grid row y as FAST_W bit words; row
// dilation is shifts inside the thread, the column dilation reads the
// neighbouring rows once through LDS (rows: [m][FAST_W] words).
constexpr int FAST_W = 4;

__device__ __forceinline__ void row_dilate_regs(uint64_t* w, int W, int n, int rr) {
  int done = 0;
  while (done < rr) {
    const int step = min(min(done + 1, rr - done), 63);   // no gaps: step <= done + 1
    uint64_t o[FAST_W];
#pragma unroll
    for (int q = 0; q < FAST_W; ++q) {
      uint64_t v = w[q];
      if (q < W) {
        // cell x takes x - step (left) and x + step (right); step < 64 here
        const uint64_t lo = q > 0 ? w[q - 1] : 0ull, hi = q + 1 < W ? w[q + 1] : 0ull;
        v |= (w[q] << step) | (lo >> (64 - step));
        v |= (w[q] >> step) | (hi << (64 - step));
        v &= last_word_mask(n, W, q);
      }
      o[q] = v;
    }
#pragma unroll
    for (int q = 0; q < FAST_W; ++q) w[q] = o[q];
    done += step;
  }
}

// Adds object o's prior to the group rows g[] of this thread's grid row.
// Communication is through LDS only (lds_barrier).
__device__ void add_object_prior_fast(const Rs3SelectArgs& a, int o, uint64_t* rows, uint64_t* g,
                                      SelShared& sh) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int m = a.m, n = a.n, s = a.s, W = (n + 63) >> 6;
  const int Wpx = n * s, Hpx = m * s;
  const uint8_t* M = a.masks + (int64_t)o * Hpx * Wpx;
  int tw[RS3_TRACK_WORDS];   // tracker words (thread 0), first used after the box
  if (tid == 0)
    for (int w = 0; w < RS3_TRACK_WORDS; ++w) tw[w] = a.track[o * RS3_TRACK_WORDS + w];
  const int y = tid;
  uint64_t w[FAST_W] = {0, 0, 0, 0};
  if (y < m) {
    const uint8_t* rp = M + (int64_t)(y * s) * Wpx;
    if (s == 1 && (n & 15) == 0 && (((uintptr_t)rp) & 15) == 0) {
      for (int x0 = 0; x0 < n; x0 += 16) {
        const u32x4 v = *(const u32x4*)(rp + x0);
        uint32_t bits = 0;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          uint32_t t = v[e];
          t |= t >> 4;
          t |= t >> 2;
          t |= t >> 1;
          bits |= ((t & 1u) | ((t >> 7) & 2u) | ((t >> 14) & 4u) | ((t >> 21) & 8u)) << (4 * e);
        }
        w[x0 >> 6] |= (uint64_t)bits << (x0 & 63);
      }
    } else {
      for (int x = 0; x < n; ++x)
        if (rp[x * s]) w[x >> 6] |= 1ull << (x & 63);
    }
  }
  // bounding box in pixels.  s == 1: rows with a set cell (ballots) and the
  // OR of all rows; otherwise a scan of every pixel.
  if (s == 1) {
    const uint64_t any = w[0] | w[1] | w[2] | w[3];
    const unsigned long long rb = __ballot(any != 0ull);
    if (lane == 0) sh.rowbits[wave] = rb;
    // columns with a set cell: OR over the wave first, then one LDS atomic
    // per wave and word (atomics of every lane on one address serialise)
#pragma unroll
    for (int q = 0; q < FAST_W; ++q) {
      if (q >= W) break;
      uint64_t c = w[q];
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) c |= __shfl_xor(c, off, 64);
      if (lane == 0 && c) atomicOr(&sh.colbits[q], (unsigned long long)c);
    }
  } else {
    int y0 = 0x7fffffff, x0 = 0x7fffffff, y1 = -1, x1 = -1;
    const int npx = Hpx * Wpx;
    for (int p = tid; p < npx; p += SEL_THREADS)
      if (M[p]) {
        const int py = p / Wpx, px = p - py * Wpx;
        y0 = min(y0, py);
        y1 = max(y1, py);
        x0 = min(x0, px);
        x1 = max(x1, px);
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
  }
  lds_barrier();
  if (tid == 0) {
    int by0 = -1, bx0 = -1, by1 = -1, bx1 = -1;
    if (s == 1) {
      for (int q = 0; q < SEL_WAVES; ++q)
        if (sh.rowbits[q]) {
          const int lo = 64 * q + (int)__builtin_ctzll(sh.rowbits[q]);
          const int hi = 64 * q + 63 - (int)__builtin_clzll(sh.rowbits[q]);
          if (by0 < 0) by0 = lo;
          by1 = hi;
        }
      for (int q = 0; q < W; ++q) {
        const uint64_t c = sh.colbits[q];
        sh.colbits[q] = 0ull;   // ready for the next object
        if (c) {
          if (bx0 < 0) bx0 = 64 * q + (int)__builtin_ctzll(c);
          bx1 = 64 * q + 63 - (int)__builtin_clzll(c);
        }
      }
    } else {
      by0 = sh.bb[0];
      bx0 = sh.bb[1];
      by1 = sh.bb[2];
      bx1 = sh.bb[3];
      sh.bb[0] = 0x7fffffff;   // ready for the next object
      sh.bb[1] = 0x7fffffff;
      sh.bb[2] = -1;
      sh.bb[3] = -1;
    }
    tracker_update(a, o, tw, by0, bx0, by1, bx1, sh);
  }
  lds_barrier();
  const int mode = sh.mode, r = sh.r;
  if (mode == MODE_BOX) {
    const int ya = max(0, sh.gy0 - r), yb = min(m - 1, sh.gy1 + r);
    const int xa = max(0, sh.gx0 - r), xb = min(n - 1, sh.gx1 + r);
    if (y < m && y >= ya && y <= yb) {
#pragma unroll
      for (int q = 0; q < FAST_W; ++q) {
        const int lo = max(xa, 64 * q), hi = min(xb, 64 * q + 63);
        if (lo <= hi) {
          const int len = hi - lo + 1;
          g[q] |= (len == 64 ? ~0ull : ((1ull << len) - 1ull)) << (lo - 64 * q);
        }
      }
    }
  } else if (mode == MODE_MASK) {
    row_dilate_regs(w, W, n, min(r, n));
    if (y < m)
#pragma unroll
      for (int q = 0; q < FAST_W; ++q)
        if (q < W) rows[y * W + q] = w[q];
    lds_barrier();
    if (y < m) {
      const int ya = max(0, y - r), yb = min(m - 1, y + r);
      for (int yy = ya; yy <= yb; ++yy)
#pragma unroll
        for (int q = 0; q < FAST_W; ++q)
          if (q < W) g[q] |= rows[yy * W + q];
    }
  }
  // rows, rowbits and the mode words are rewritten by the next object
  lds_barrier();
}

// One-wave prior for grids of at most 64 rows and stride 1 (wave 0 only, no
// block barrier): lane y holds grid row y as FAST_W bit words.  The box is a
// ballot over the rows and a wave OR of the columns, the tracker update is
// wave-uniform (lane 0 writes the words back), and the column dilation
// shifts whole rows across lanes with the same doubling steps as the row
// dilation (rows past the grid hold 0).  Same prior as the block paths.
__device__ void add_object_prior_wave(const Rs3SelectArgs& a, int o, uint64_t* g) {
  const int lane = threadIdx.x & 63;
  const int m = a.m, n = a.n, W = (n + 63) >> 6;
  const uint8_t* M = a.masks + (int64_t)o * m * n;
  int32_t* tr = a.track + o * RS3_TRACK_WORDS;
  int tl[RS3_TRACK_WORDS];
#pragma unroll
  for (int w = 0; w < RS3_TRACK_WORDS; ++w) tl[w] = tr[w];
  uint64_t w[FAST_W] = {0, 0, 0, 0};
  if (lane < m) {
    const uint8_t* rp = M + (int64_t)lane * n;
    if ((n & 15) == 0 && (((uintptr_t)rp) & 15) == 0) {
      for (int x0 = 0; x0 < n; x0 += 16) {
        const u32x4 v = *(const u32x4*)(rp + x0);
        uint32_t bits = 0;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          uint32_t t = v[e];
          t |= t >> 4;
          t |= t >> 2;
          t |= t >> 1;
          bits |= ((t & 1u) | ((t >> 7) & 2u) | ((t >> 14) & 4u) | ((t >> 21) & 8u)) << (4 * e);
        }
        w[x0 >> 6] |= (uint64_t)bits << (x0 & 63);
      }
    } else {
      for (int x = 0; x < n; ++x)
        if (rp[x]) w[x >> 6] |= 1ull << (x & 63);
    }
  }
  // bounding box (grid cells = pixels at stride 1)
  const unsigned long long rb = __ballot((w[0] | w[1] | w[2] | w[3]) != 0ull);
  int by0 = -1, bx0 = -1, by1 = -1, bx1 = -1;
  if (rb) {
    by0 = (int)__builtin_ctzll(rb);
    by1 = 63 - (int)__builtin_clzll(rb);
  }
#pragma unroll
  for (int q = 0; q < FAST_W; ++q) {
    if (q >= W) break;
    uint64_t c = w[q];
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) c |= __shfl_xor(c, off, 64);
    if (c) {
      if (bx0 < 0) bx0 = 64 * q + (int)__builtin_ctzll(c);
      bx1 = 64 * q + 63 - (int)__builtin_clzll(c);
    }
  }
  // tracker update (the rule of tracker_update)
  int mode = MODE_NONE, r = a.r_s;
  if (by1 >= 0) {
    mode = a.seed_box ? MODE_BOX : MODE_MASK;
    tl[0] = by0;
    tl[1] = bx0;
    tl[2] = by1;
    tl[3] = bx1;
    tl[4] = 0;
    tl[5] = 1;
  } else {
    const int d = tl[4] + 1;
    tl[4] = d;
    if (tl[5]) {
      mode = MODE_BOX;
      by0 = tl[0];
      bx0 = tl[1];
      by1 = tl[2];
      bx1 = tl[3];
      r = a.r_s + min(d, a.c);
    }
  }
  if (lane == 0)
#pragma unroll
    for (int q = 0; q < RS3_TRACK_WORDS; ++q) tr[q] = tl[q];
  if (mode == MODE_BOX) {
    const int ya = max(0, by0 - r), yb = min(m - 1, by1 + r);
    const int xa = max(0, bx0 - r), xb = min(n - 1, bx1 + r);
    if (lane < m && lane >= ya && lane <= yb) {
#pragma unroll
      for (int q = 0; q < FAST_W; ++q) {
        const int lo = max(xa, 64 * q), hi = min(xb, 64 * q + 63);
        if (lo <= hi) {
          const int len = hi - lo + 1;
          g[q] |= (len == 64 ? ~0ull : ((1ull << len) - 1ull)) << (lo - 64 * q);
        }
      }
    }
  } else if (mode == MODE_MASK) {
    row_dilate_regs(w, W, n, min(r, n));
    const int rr = min(r, 63);   // rows are at most 64 apart
    int done = 0;
    while (done < rr) {
      const int step = min(done + 1, rr - done);   // no gaps: step <= done + 1
#pragma unroll
      for (int q = 0; q < FAST_W; ++q) {
        if (q >= W) break;
        const uint64_t up = __shfl(w[q], lane - step, 64), dn = __shfl(w[q], lane + step, 64);
        w[q] |= (lane - step >= 0 ? up : 0ull) | (lane + step < 64 ? dn : 0ull);
      }
      done += step;
    }
    if (lane < m)
#pragma unroll
      for (int q = 0; q < FAST_W; ++q) g[q] |= w[q];
  }
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
    int tw[RS3_TRACK_WORDS];
    for (int w = 0; w < RS3_TRACK_WORDS; ++w) tw[w] = a.track[o * RS3_TRACK_WORDS + w];
    tracker_update(a, o, tw, sh.bb[0], sh.bb[1], sh.bb[2], sh.bb[3], sh);
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
  uint8_t* rank_lds = tmp + buf;   // SEL_RANK_BYTES: candidate keys, cells, keep bits

  // Contiguous cells per thread so that block scans follow cell order.  The
  // energies and tracker words do not depend on the prior: load them first.
  const int cpt = (mn + SEL_THREADS - 1) / SEL_THREADS;
  const int c0 = tid * cpt;
  const unsigned long long* ebits =
      reinterpret_cast<const unsigned long long*>(a.e + (a.x_per_obj ? (int64_t)g * mn : 0)) + c0;
  unsigned long long kreg[REG ? MAXC : 1];
  if (REG) {
#pragma unroll
    for (int j = 0; j < MAXC; ++j) kreg[REG ? j : 0] = (j < cpt && c0 + j < mn) ? ebits[j] : 0ull;
  }
  // per-block energy ranges of this grid (wave 0, NR per lane), reduced later
  constexpr int NR = MAXC / 4 > 0 ? MAXC / 4 : 1;
  const int n_eblk = (mn + 63) >> 6;
  unsigned long long rlo[NR], rhi[NR];
  if (tid < 64) {
    const unsigned long long* er = a.erange + 2 * (int64_t)(a.x_per_obj ? g : 0) * n_eblk;
#pragma unroll
    for (int q = 0; q < NR; ++q) {
      const int bk = lane + 64 * q;
      rlo[q] = bk < n_eblk ? er[2 * bk] : ~0ull;
      rhi[q] = bk < n_eblk ? er[2 * bk + 1] : 0ull;
    }
  }
  if (tid == 0) {
    sh.bb[0] = 0x7fffffff;
    sh.bb[1] = 0x7fffffff;
    sh.bb[2] = -1;
    sh.bb[3] = -1;
  }
  if (tid < 4) sh.colbits[tid] = 0ull;
  if (tid < 256) sh.hist[tid] = 0;
  const int W = (a.n + 63) >> 6;
  const bool fast = a.m <= SEL_THREADS && W <= FAST_W;
  uint64_t* Gs = reinterpret_cast<uint64_t*>(base);   // fast path: group prior rows [m][W]
  if (fast && a.m <= 64 && a.s == 1 && a.prior_bits) {
    // the prior (and the tracker update) ran beside the energies
    const uint64_t* pb = a.prior_bits + (int64_t)g * 64 * FAST_W;
    if (tid < a.m * W) Gs[tid] = pb[tid];
    lds_barrier();
  } else if (fast && a.m <= 64 && a.s == 1) {
    // one wave: lane y owns grid row y
    if (tid < 64) {
      uint64_t gw[FAST_W] = {0, 0, 0, 0};
      if (a.union_objects) {
        for (int o = 0; o < a.n_obj; ++o) add_object_prior_wave(a, o, gw);
      } else {
        add_object_prior_wave(a, g, gw);
      }
      if (tid < a.m)
#pragma unroll
        for (int q = 0; q < FAST_W; ++q)
          if (q < W) Gs[tid * W + q] = gw[q];
    }
    lds_barrier();
  } else if (fast) {
    uint64_t* rows = reinterpret_cast<uint64_t*>(tmp);
    uint64_t gw[FAST_W] = {0, 0, 0, 0};
    lds_barrier();
    if (a.union_objects) {
      for (int o = 0; o < a.n_obj; ++o) add_object_prior_fast(a, o, rows, gw, sh);
    } else {
      add_object_prior_fast(a, g, rows, gw, sh);
    }
    if (tid < a.m)
#pragma unroll
      for (int q = 0; q < FAST_W; ++q)
        if (q < W) Gs[tid * W + q] = gw[q];
    lds_barrier();
  } else {
    for (int i = tid; i < mn; i += SEL_THREADS) U[i] = 0;
    __syncthreads();
    if (a.union_objects) {
      for (int o = 0; o < a.n_obj; ++o) add_object_prior(a, o, U, base, tmp, sh);
    } else {
      add_object_prior(a, g, U, base, tmp, sh);
    }
  }
  // this thread's cells c0 .. c0+cpt-1 start at grid row cy, column cx
  int cy = c0 / a.n, cx = c0 - cy * a.n;
  uint32_t inP = 0;
#pragma unroll
  for (int j = 0; j < MAXC; ++j) {
    if (j < cpt && c0 + j < mn) {
      const bool in = fast ? ((Gs[cy * W + (cx >> 6)] >> (cx & 63)) & 1ull) : U[c0 + j] != 0;
      if (in) inP |= 1u << j;
      if (++cx == a.n) {
        cx = 0;
        ++cy;
      }
    }
  }
  if (a.prior_out) {
    uint8_t* po = a.prior_out + (int64_t)g * mn + c0;
#pragma unroll
    for (int j = 0; j < MAXC; ++j)
      if (j < cpt && c0 + j < mn) po[j] = (inP >> j) & 1u;
  }
  auto key_of = [&](int j) -> unsigned long long { return REG ? kreg[REG ? j : 0] : ebits[j]; };
  const int k = a.k[g];
  int countP;
  block_scan_bits<MAXC>(inP, cpt, sh.red1, &countP);
  uint32_t keep = inP;
  if (countP > k) {
    bool done = false;
    if (tid < 64) {
      unsigned long long l = rlo[0], h = rhi[0];
#pragma unroll
      for (int q = 1; q < NR; ++q) {
        l = rlo[q] < l ? rlo[q] : l;
        h = rhi[q] > h ? rhi[q] : h;
      }
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) {
        const unsigned long long ol = __shfl_xor(l, off, 64), oh = __shfl_xor(h, off, 64);
        l = ol < l ? ol : l;
        h = oh > h ? oh : h;
      }
      if (tid == 0) {
        sh.kmin = l;
        sh.kmax = h;
      }
    }
    lds_barrier();
    // range of the grid's energies: it contains every candidate key
    const unsigned long long kmin = sh.kmin, kmax = sh.kmax;
    if (k > 0 && kmin != kmax) {
      // One histogram over 256 equal-width bins of [kmin, kmax] (bin of a key
      // is monotone in the key, so every key of a higher bin is larger), then
      // an exact rank inside the bin that holds the k-th largest key.
      const double scale = 256.0 / (double)(kmax - kmin);
      auto bin_of = [&](unsigned long long key) -> int {
        const int b = (int)((double)(key - kmin) * scale);
        return b > 255 ? 255 : b;
      };
      if (tid == 0) sh.ncand = 0;
#pragma unroll
      for (int j = 0; j < MAXC; ++j)
        if (inP >> j & 1) atomicAdd(&sh.hist[bin_of(key_of(j))], 1);
      lds_barrier();
      if (tid < 64) find_digit(sh, k, lane);
      lds_barrier();
      const int B = sh.digit, rem = sh.remaining, cntB = sh.hist[B];
      const bool full = sh.full;
      if (full || cntB <= SEL_THREADS) {
        uint32_t kp = 0, inB = 0;
#pragma unroll
        for (int j = 0; j < MAXC; ++j)
          if (inP >> j & 1) {
            const int b = bin_of(key_of(j));
            if (b > B || (full && b == B)) kp |= 1u << j;
            if (b == B) inB |= 1u << j;
          }
        if (!full) {
          unsigned long long* ck = reinterpret_cast<unsigned long long*>(rank_lds);
          int* ci = reinterpret_cast<int*>(ck + SEL_THREADS);
          uint32_t* kb = reinterpret_cast<uint32_t*>(ci + SEL_THREADS);
          kb[tid] = 0;
#pragma unroll
          for (int j = 0; j < MAXC; ++j)
            if (inB >> j & 1) {
              const int q = atomicAdd(&sh.ncand, 1);
              ck[q] = key_of(j);
              ci[q] = c0 + j;
            }
          lds_barrier();
          // exact rank of each boundary candidate among the candidates
          // (larger key first, equal keys by cell): wave w takes candidates
          // w, w + 16, ...; its lanes compare against candidates lane,
          // lane + 64, ... and a ballot counts those ranked before
          const int wave = tid >> 6;
          unsigned long long lk = 0;
          int li = 0;
          if (lane < cntB) {
            lk = ck[lane];
            li = ci[lane];
          }
          for (int i = wave; i < cntB; i += SEL_WAVES) {
            const unsigned long long key = ck[i];
            const int idx = ci[i];
            int rank = 0;
            for (int j0 = 0; j0 < cntB; j0 += 64) {
              const int j = j0 + lane;
              unsigned long long kq = lk;
              int iq = li;
              if (j0 > 0 && j < cntB) {
                kq = ck[j];
                iq = ci[j];
              }
              rank += __popcll(__ballot(j < cntB && (kq > key || (kq == key && iq < idx))));
            }
            if (lane == 0 && rank < rem) atomicOr(&kb[idx / cpt], 1u << (idx - (idx / cpt) * cpt));
          }
          lds_barrier();
          kp |= kb[tid];
        }
        keep = kp;
        done = true;
      }
    }
    if (!done) {
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
        if (tid < 64) find_digit(sh, remaining, lane);
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
  }
  int total;
  int before = block_scan_bits<MAXC>(keep, cpt, sh.red3, &total);
  int32_t* out = a.sel_idx + (int64_t)g * mn;
#pragma unroll
  for (int j = 0; j < MAXC; ++j)
    if (keep >> j & 1) out[before++] = c0 + j;
  if (tid == 0) a.sel_count[g] = total;
}

// The energies and, for grids of at most 64 rows and 256 columns at stride 1,
// the one-wave prior of every group in one launch: the prior depends only on
// the masks and the tracker state, the energies only on X, so the prior
// blocks (after the energy blocks) run beside them and leave the group's
// prior rows [m][W] in prior_bits for the selection.
template <typename T, bool QP = false, bool WIDE = false>
__global__ __launch_bounds__(256) void k_energy_prior(const T* __restrict__ X, int64_t x_stride, int mn, int C,
                                                      double* __restrict__ e, unsigned long long* __restrict__ range,
                                                      Rs3SelectArgs a, int nbx, int n_e, Rs3QProjArgs qp) {
  // the arguments of both kinds of block in one batch of loads: the argument
  // block is memory the host wrote just before the launch, and loads behind
  // the block-kind test would wait for the test's own load first
  asm volatile("" ::"s"(n_e), "s"(nbx), "s"(X), "s"(x_stride), "s"(mn), "s"(C), "s"(e), "s"(range),
               "s"(qp.WqT), "s"(qp.Qall), "s"(a.n), "s"(a.m), "s"(a.union_objects), "s"(a.n_obj), "s"(a.masks),
               "s"(a.track), "s"(a.prior_bits));
  const int b = blockIdx.x;
  if (b < n_e) {
    if constexpr (WIDE)
      energy_block_wide<T>(X, x_stride, mn, C, e, range, b % nbx, b / nbx);
    else
      energy_block<T, QP>(X, x_stride, mn, C, e, range, b % nbx, b / nbx, nbx, &qp);
    return;
  }
  const int g = b - n_e, tid = threadIdx.x;
  if (tid >= 64) return;
  const int W = (a.n + 63) >> 6;
  uint64_t gw[FAST_W] = {0, 0, 0, 0};
  if (a.union_objects) {
    for (int o = 0; o < a.n_obj; ++o) add_object_prior_wave(a, o, gw);
  } else {
    add_object_prior_wave(a, g, gw);
  }
  uint64_t* pb = a.prior_bits + (int64_t)g * 64 * FAST_W;
  if (tid < a.m)
#pragma unroll
    for (int q = 0; q < FAST_W; ++q)
      if (q < W) pb[tid * W + q] = gw[q];
}

}  // namespace rs3

using namespace rs3;

// The projection in the energy launch needs whole 256-channel bf16 rows in
// one column block.
static bool qproj_ok(int C, int dtype, const Rs3QProjArgs* qp) {
  return qp && dtype == RS3_BF16 && C == 8 * EB_CH;
}

// The wide form when it still gives a launch of at least 256 blocks.
static bool energy_wide(int n_x, int mn, const Rs3QProjArgs* qp) {
  return !qp && (int64_t)n_x * ((mn + EW_ROWS - 1) / EW_ROWS) >= 256;
}

hipError_t rs3_launch_energy(const void* X, int64_t x_stride, int n_x, int mn, int C, int dtype,
                             double* e, unsigned long long* range, hipStream_t st, const Rs3QProjArgs* qp) {
  dim3 grid((mn + 63) / 64, n_x);
  if (qp && !qproj_ok(C, dtype, qp)) return hipErrorInvalidValue;
  if (energy_wide(n_x, mn, qp)) {
    const dim3 gw((mn + EW_ROWS - 1) / EW_ROWS, n_x);
    if (dtype == RS3_BF16)
      RS3_LAUNCH(RS3_K_ENERGY, st, k_energy_wide<bf16_t>, gw, dim3(256), 0, st, (const bf16_t*)X, x_stride, mn, C, e,
                 range);
    else
      RS3_LAUNCH(RS3_K_ENERGY, st, k_energy_wide<float>, gw, dim3(256), 0, st, (const float*)X, x_stride, mn, C, e,
                 range);
    return hipGetLastError();
  }
  const Rs3QProjArgs q = qp ? *qp : Rs3QProjArgs{};
  if (qp)
    RS3_LAUNCH(RS3_K_ENERGY, st, (k_energy<bf16_t, true>), grid, dim3(256), 0, st, (const bf16_t*)X, x_stride, mn, C,
               e, range, q);
  else if (dtype == RS3_BF16)
    RS3_LAUNCH(RS3_K_ENERGY, st, k_energy<bf16_t>, grid, dim3(256), 0, st, (const bf16_t*)X, x_stride, mn, C, e,
               range, q);
  else
    RS3_LAUNCH(RS3_K_ENERGY, st, k_energy<float>, grid, dim3(256), 0, st, (const float*)X, x_stride, mn, C, e,
               range, q);
  return hipGetLastError();
}

bool rs3_select_prior_beside(int m, int n, int s) { return m <= 64 && s == 1 && n <= 64 * FAST_W; }

hipError_t rs3_launch_energy_prior(const void* X, int64_t x_stride, int n_x, int mn, int C, int dtype, double* e,
                                   unsigned long long* range, const Rs3SelectArgs& a, int n_groups, hipStream_t st,
                                   const Rs3QProjArgs* qp) {
  if (qp && !qproj_ok(C, dtype, qp)) return hipErrorInvalidValue;
  const Rs3QProjArgs q = qp ? *qp : Rs3QProjArgs{};
  if (energy_wide(n_x, mn, qp)) {
    const int nbw = (mn + EW_ROWS - 1) / EW_ROWS, n_w = nbw * n_x;
    const dim3 gw(n_w + n_groups);
    if (dtype == RS3_BF16)
      RS3_LAUNCH(RS3_K_ENERGY, st, (k_energy_prior<bf16_t, false, true>), gw, dim3(256), 0, st, (const bf16_t*)X,
                 x_stride, mn, C, e, range, a, nbw, n_w, q);
    else
      RS3_LAUNCH(RS3_K_ENERGY, st, (k_energy_prior<float, false, true>), gw, dim3(256), 0, st, (const float*)X,
                 x_stride, mn, C, e, range, a, nbw, n_w, q);
    return hipGetLastError();
  }
  const int nbx = (mn + 63) / 64, n_e = nbx * n_x;
  const dim3 grid(n_e + n_groups);
  if (qp)
    RS3_LAUNCH(RS3_K_ENERGY, st, (k_energy_prior<bf16_t, true>), grid, dim3(256), 0, st, (const bf16_t*)X, x_stride,
               mn, C, e, range, a, nbx, n_e, q);
  else if (dtype == RS3_BF16)
    RS3_LAUNCH(RS3_K_ENERGY, st, k_energy_prior<bf16_t>, grid, dim3(256), 0, st, (const bf16_t*)X, x_stride, mn, C, e,
               range, a, nbx, n_e, q);
  else
    RS3_LAUNCH(RS3_K_ENERGY, st, k_energy_prior<float>, grid, dim3(256), 0, st, (const float*)X, x_stride, mn, C, e,
               range, a, nbx, n_e, q);
  return hipGetLastError();
}

static size_t select_lds_bytes(int m, int n) {
  return (size_t)((m * n + 15) & ~15) + 2 * (size_t)select_buf_bytes(m, n) + SEL_RANK_BYTES;
}

hipError_t rs3_select_setup() {
  // largest layout: mn = RS3_MAX_MN with byte-sized buffers (3 * 32 KB)
  const int mx = 3 * RS3_MAX_MN + 64 + SEL_RANK_BYTES;
  hipError_t e = hipFuncSetAttribute((const void*)k_select<4>, hipFuncAttributeMaxDynamicSharedMemorySize, mx);
  if (e != hipSuccess) return e;
  e = hipFuncSetAttribute((const void*)k_select<16>, hipFuncAttributeMaxDynamicSharedMemorySize, mx);
  if (e != hipSuccess) return e;
  return hipFuncSetAttribute((const void*)k_select<32>, hipFuncAttributeMaxDynamicSharedMemorySize, mx);
}

hipError_t rs3_launch_select(const Rs3SelectArgs& a, int n_groups, hipStream_t st) {
  const int mn = a.m * a.n;
  const size_t lds = select_lds_bytes(a.m, a.n);
  if (mn <= 4 * SEL_THREADS)
    RS3_LAUNCH(RS3_K_SELECT, st, k_select<4>, dim3(n_groups), dim3(SEL_THREADS), lds, st, a);
  else if (mn <= 16 * SEL_THREADS)
    RS3_LAUNCH(RS3_K_SELECT, st, k_select<16>, dim3(n_groups), dim3(SEL_THREADS), lds, st, a);
  else
    RS3_LAUNCH(RS3_K_SELECT, st, k_select<32>, dim3(n_groups), dim3(SEL_THREADS), lds, st, a);
  return hipGetLastError();
}
