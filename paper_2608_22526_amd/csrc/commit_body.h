// Device code of the store-sparse commit (Sec. 3.2, Eq. 8): mask compaction,
// ring placement, tile list and the append with the K/V projections, shared
// by the commit kernels and the fused merge + commit launch.
#pragma once

#include "device_util.h"

namespace rs3 {

constexpr int CP_THREADS = 1024;
constexpr int CP_WAVES = CP_THREADS / 64;
constexpr int CP_MAX_CPT = RS3_MAX_MN / CP_THREADS;

struct CpShared {
  int red[CP_WAVES];
  int red2[CP_WAVES];
  int ok, start, len;
};

__device__ __forceinline__ int cp_wave_incl_scan(int v, int lane) {
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    int t = __shfl_up(v, off, 64);
    if (lane >= off) v += t;
  }
  return v;
}

__device__ int cp_block_excl_scan(int v, CpShared& sh, int* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int inc = cp_wave_incl_scan(v, lane);
  if (lane == 63) sh.red[wave] = inc;
  __syncthreads();
  int wsum = 0, tot = 0;
  for (int w = 0; w < CP_WAVES; ++w) {
    int s = sh.red[w];
    if (w < wave) wsum += s;
    tot += s;
  }
  __syncthreads();
  *total = tot;
  return wsum + inc - v;
}

__device__ __forceinline__ uint64_t tile_mask(const int32_t* fr, int nf, int tile) {
  const int64_t t0 = (int64_t)tile * KT, t1 = t0 + KT;
  uint64_t msk = 0;
  for (int f = 0; f < nf; ++f) {
    int64_t fs = fr[4 * f], fe = fs + fr[4 * f + 1];
    int64_t a = fs > t0 ? fs : t0, e = fe < t1 ? fe : t1;
    if (a < e) {
      int lo = (int)(a - t0), hi = (int)(e - t0);
      uint64_t bits = (hi - lo == 64) ? ~0ull : (((1ull << (hi - lo)) - 1ull) << lo);
      msk |= bits;
    }
  }
  return msk;
}


// Exclusive prefix (thread order) of the set bits among the first n bits of
// `bits`, and the workgroup total, from ballots; `red` is an LDS array of
// CP_WAVES entries private to the call site.
__device__ __forceinline__ int cp_scan_bits(uint32_t bits, int n, int* red, int* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int pre = 0, wtot = 0;
  for (int j = 0; j < n; ++j) {
    const unsigned long long b = __ballot((bits >> j) & 1u);
    pre += __builtin_amdgcn_mbcnt_hi((uint32_t)(b >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)b, 0u));
    wtot += __popcll(b);
  }
  if (lane == 0) red[wave] = wtot;
  lds_barrier();
  int before = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < CP_WAVES; ++w) {
    const int v = red[w];
    tot += v;
    before += w < wave ? v : 0;
  }
  *total = tot;
  return before + pre;
}

// Ring placement by one wave (lane l holds frames 4l .. 4l+3 of the
// key-ordered table, f_max <= 256): the count and overlap evictions of the
// placement rule both remove a prefix of the unpinned frames, found with
// ballots; survivors move to their new slots in one scatter.  Returns the
// start row or -1 (capacity; table unchanged), the new frame count, pin end
// and resident key count.
__device__ __forceinline__ int place_frame_wave(const BankDev& b, int32_t* fr, int nf, int pin_end, int L, int t, int pin,
                                int* nf_out, int* pin_end_out, int* keys_out) {
  const int lane = threadIdx.x & 63;
  int fs[4], fl[4], fw[4], fp[4];
  bool fv[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int f = 4 * lane + k;
    fv[k] = f < nf;
    fs[k] = fv[k] ? fr[4 * f] : 0;
    fl[k] = fv[k] ? fr[4 * f + 1] : 0;
    fw[k] = fv[k] ? fr[4 * f + 2] : 0;
    fp[k] = fv[k] ? fr[4 * f + 3] : 0;
  }
  int n_pf = 0;
#pragma unroll
  for (int k = 0; k < 4; ++k) n_pf += __popcll(__ballot(fv[k] && fp[k]));
  int start, E = 0;
  if (pin) {
    if ((int64_t)pin_end + L > b.cap || nf >= b.f_max) return -1;
    start = pin_end;
  } else {
    if (L > b.cap - pin_end) return -1;
    const int e1 = nf >= b.f_max ? nf - (b.f_max - 1) : 0;   // make room for one frame
    if (e1 > nf - n_pf) return -1;   // unreachable while n_pin < f_max
    start = (nf - 1 >= n_pf + e1) ? fr[4 * (nf - 1)] + fr[4 * (nf - 1) + 1] : pin_end;
    if ((int64_t)start + L > b.cap) start = pin_end;
    // newest remaining unpinned frame that overlaps [start, start+L)
    int imax = -1;
    if (L > 0) {
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int f = 4 * lane + k;
        const bool hit = fv[k] && !fp[k] && f >= n_pf + e1 && fl[k] > 0 && fs[k] < start + L &&
                         start < fs[k] + fl[k];
        const unsigned long long bm = __ballot(hit);
        if (bm) imax = max(imax, 4 * (63 - (int)__builtin_clzll(bm)) + k);
      }
    }
    E = max(e1, imax >= 0 ? imax - n_pf + 1 : 0);
  }
  // survivors: pinned frames stay, unpinned frames past the evicted prefix
  // move down by E; the new frame goes last
  int keys = 0;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int f = 4 * lane + k;
    if (!fv[k] || (!fp[k] && f < n_pf + E)) continue;
    keys += fl[k];
    const int d = fp[k] ? f : f - E;
    if (d != f) {
      fr[4 * d] = fs[k];
      fr[4 * d + 1] = fl[k];
      fr[4 * d + 2] = fw[k];
      fr[4 * d + 3] = fp[k];
    }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) keys += __shfl_xor(keys, off, 64);
  const int slot = nf - E;
  if (lane == 0) {
    fr[4 * slot] = start;
    fr[4 * slot + 1] = L;
    fr[4 * slot + 2] = t;
    fr[4 * slot + 3] = pin ? 1 : 0;
  }
  *nf_out = slot + 1;
  *pin_end_out = pin ? pin_end + L : pin_end;
  *keys_out = keys + L;
  return start;
}

// Tiles per thread whose masks the rebuild keeps in registers (bank rings of
// up to 8*1024 tiles, 512K rows).
constexpr int TILES_REG = 8;

// Rebuilds the resident tile list (ascending tiles with their row masks)
// and hdr NTILES from the LDS frame table; every thread of the workgroup.
__device__ __forceinline__ void rebuild_tiles(const BankDev& b, const int32_t* sfr, int nf, CpShared& sh) {
  const int tid = threadIdx.x;
  const int nt = b.n_tiles_cap;
  const int tpt = (nt + CP_THREADS - 1) / CP_THREADS;
  const int t0 = tid * tpt;
  int ntot = 0, pos = 0;
  if (tpt <= TILES_REG) {
    // one pass over the frames: OR each frame's rows into the masks of this
    // thread's tiles (frame entries are read by every thread at once)
    uint64_t msk[TILES_REG];
#pragma unroll
    for (int j = 0; j < TILES_REG; ++j) msk[j] = 0ull;
    // rows stay below 2^26, so 32-bit row arithmetic cannot overflow
    const int r_lo = t0 * KT, r_hi = (t0 + tpt) * KT;
    for (int f0 = 0; f0 < nf; f0 += 4) {
      int4 fe4[4];   // four frame entries per LDS read burst
#pragma unroll
      for (int u = 0; u < 4; ++u) fe4[u] = *(const int4*)&sfr[4 * (f0 + u < nf ? f0 + u : f0)];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int fs = fe4[u].x, fe = fs + fe4[u].y;
        const int a = fs > r_lo ? fs : r_lo, e = fe < r_hi ? fe : r_hi;
        if (f0 + u >= nf || a >= e) continue;
#pragma unroll
        for (int j = 0; j < TILES_REG; ++j) {
          const int ta = (t0 + j) * KT, te = ta + KT;
          const int x = a > ta ? a : ta, y = e < te ? e : te;
          if (j < tpt && x < y) {
            const int lo = x - ta, n = y - x;
            msk[j] |= (n == 64 ? ~0ull : ((1ull << n) - 1ull)) << lo;
          }
        }
      }
    }
    uint32_t live = 0;
#pragma unroll
    for (int j = 0; j < TILES_REG; ++j)
      if (j < tpt && t0 + j < nt && msk[j]) live |= 1u << j;
    pos = cp_scan_bits(live, tpt, sh.red2, &ntot);
#pragma unroll
    for (int j = 0; j < TILES_REG; ++j)
      if (live >> j & 1) {
        TileEnt te;
        te.tile = t0 + j;
        te.pad = 0;
        te.mask = msk[j];
        b.tiles[pos++] = te;
      }
    if (tid == 0) b.hdr[HDR_NTILES] = ntot;
    return;
  }
  if (tpt <= 32) {
    uint32_t live = 0;
    for (int j = 0; j < tpt; ++j)
      if (t0 + j < nt && tile_mask(sfr, nf, t0 + j)) live |= 1u << j;
    pos = cp_scan_bits(live, tpt, sh.red2, &ntot);
  } else {
    int cnt = 0;
    for (int j = 0; j < tpt; ++j)
      if (t0 + j < nt && tile_mask(sfr, nf, t0 + j)) ++cnt;
    pos = cp_block_excl_scan(cnt, sh, &ntot);
  }
  for (int j = 0; j < tpt; ++j) {
    if (t0 + j >= nt) break;
    const uint64_t msk = tile_mask(sfr, nf, t0 + j);
    if (msk) {
      TileEnt te;
      te.tile = t0 + j;
      te.pad = 0;
      te.mask = msk;
      b.tiles[pos++] = te;
    }
  }
  if (tid == 0) b.hdr[HDR_NTILES] = ntot;
}

// ---------------------------------------------------------------------------
// Append of rows r0 .. r0+rows-1 of the new frame (ring rows start + r0 + r)
// by the NT threads of a work-group.  src[r] (LDS) is the kept cell of row
// r; with a.from_ring the rows are already in the raw ring.
// bf16: the kept rows are read once (16-byte loads) into LDS and written to
// the raw ring from the same registers; the projections then read their row
// operands from LDS:
//   K^ rows: C = A B, A = kept K rows (64 x d_kv), B = W_k (d_kv x D):
//     lane holds column d, rows = keys  -> Khat[tile][h][key][d%d_h]
//   V^ as its transpose: C = W_v^T (D x d_kv) V^T (d_kv x 64):
//     lane holds column = key, rows = d -> Vhat[tile][h][d%d_h][vslot(key)]
// rows_lds: 2 * 64 * (d_kv + 8) bf16.
template <int NT>
__device__ __forceinline__ void append_bf16(const Rs3CommitArgs& a, const BankDev& b, int o, int start, int r0,
                                            int rows, const int* src, bf16_t* rows_lds) {
  constexpr int NW = NT / 64;
  const int d_kv = b.d_kv, d_h = b.d_h, H = b.H, D = H * d_h;
  const int lg_dh = 31 - __clz(d_h);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, g = lane >> 5;
  const int RS = d_kv + 8;  // padded LDS row
  bf16_t* sK = rows_lds;
  bf16_t* sV = rows_lds + 64 * RS;
  const bf16_t* Km = (const bf16_t*)a.Kmem + (int64_t)o * a.kv_stride;
  const bf16_t* Vm = (const bf16_t*)a.Vmem + (int64_t)o * a.kv_stride;
  bf16_t* Kr = (bf16_t*)b.Kraw;
  bf16_t* Vr = (bf16_t*)b.Vraw;
  const int cpr = d_kv / 8;
  for (int q = tid; q < 64 * cpr; q += NT) {
    const int r = q / cpr, c = q - r * cpr;
    u32x4 kv = {0, 0, 0, 0}, vv = {0, 0, 0, 0};
    if (r < rows) {
      const int64_t j = start + r0 + r;
      if (a.from_ring) {
        kv = gload((const u32x4*)(Kr + j * d_kv + 8 * c));
        vv = gload((const u32x4*)(Vr + j * d_kv + 8 * c));
      } else {
        const int cell = src[r];
        kv = gload((const u32x4*)(Km + (int64_t)cell * d_kv + 8 * c));
        vv = gload((const u32x4*)(Vm + (int64_t)cell * d_kv + 8 * c));
        gstore((u32x4*)(Kr + j * d_kv + 8 * c), kv);
        gstore((u32x4*)(Vr + j * d_kv + 8 * c), vv);
      }
    }
    *(u32x4*)(sK + r * RS + 8 * c) = kv;
    *(u32x4*)(sV + r * RS + 8 * c) = vv;
  }
  lds_barrier();
  bf16_t* Kh = (bf16_t*)b.Khat;
  bf16_t* Vh = (bf16_t*)b.Vhat;
  if (a.absorb) {
    // attention on the raw rows (one head of width d_kv): K rows as they
    // are, V rows transposed into slot order
    for (int q = tid; q < rows * cpr; q += NT) {
      const int r = q / cpr, c = q - r * cpr;
      const int j = start + r0 + r;
      gstore((u32x4*)(Kh + ((int64_t)(j >> 6) * KT + (j & 63)) * d_kv + 8 * c), *(const u32x4*)(sK + r * RS + 8 * c));
    }
    // consecutive lanes take consecutive keys of one V^ row, so that a
    // wave's stores fall in one or two 128-byte lines of the tile
    for (int q = tid; q < rows * d_kv; q += NT) {
      const int d = q / rows, r = q - d * rows;
      const int j = start + r0 + r;
      gstore(Vh + ((int64_t)(j >> 6) * d_kv + d) * KT + vslot(j & 63), sV[r * RS + d]);
    }
    return;
  }
  const bf16_t* WkT = (const bf16_t*)a.WkT;
  const bf16_t* WvT = (const bf16_t*)a.WvT;
  const int nblk = 2 * (D / 32);
  for (int blk = wave; blk < nblk; blk += NW) {
    const int mb = blk & 1, nb = blk >> 1;
    const int rr = 32 * mb + (lane & 31);   // key row fed by this lane
    const int dcol = 32 * nb + (lane & 31);
    const bf16_t* krow = sK + rr * RS + 8 * g;
    const bf16_t* vrow = sV + rr * RS + 8 * g;
    const bf16_t* wk = WkT + (int64_t)dcol * d_kv + 8 * g;
    const bf16_t* wv = WvT + (int64_t)dcol * d_kv + 8 * g;
    f32x16 ck = {}, cv = {};
    for (int ks = 0; ks < d_kv; ks += 16) {
      ck = mfma32(*(const u32x4*)(krow + ks), gload((const u32x4*)(wk + ks)), ck);   // rows = keys, cols = d
      cv = mfma32(gload((const u32x4*)(wv + ks)), *(const u32x4*)(vrow + ks), cv);   // rows = d, cols = keys
    }
    // V^ first (its accumulators are then free while K^ is turned):
    // row = d (32nb + c_row), column = key (rr)
    if (rr < rows) {
      const int j = start + r0 + rr;
      const int64_t tb = (int64_t)(j >> 6) * H;
      const int slot = vslot(j & 63);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int d = 32 * nb + c_row(r, lane);
        const int h = d >> lg_dh, dd = d & (d_h - 1);
        gstore(Vh + ((tb + h) * d_h + dd) * KT + slot, __builtin_bit_cast(bf16_t, (__bf16)cv[r]));
      }
    }
    // K^: row = key (32mb + c_row), column = d (dcol)
    {
      const int h = dcol >> lg_dh, dd = dcol & (d_h - 1);
      if (a.rope) {
        // Eq. 7 on the key side: the key kept from cell src[row] turns by
        // that cell's factors (lanes l and l^1 hold columns 2p and 2p+1)
        const float2* rope = (const float2*)a.rope;
        const int hp = d_h >> 1, p = dd >> 1;
        const float sgn = (dd & 1) ? 1.f : -1.f;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int kr = 32 * mb + c_row(r, lane);
          const int cell = kr < rows ? min(max(src[kr], 0), a.rope_mn - 1) : 0;
          typedef float f32x2 __attribute__((ext_vector_type(2)));
          const f32x2 cs = gload((const f32x2*)(rope + (int64_t)cell * hp + p));
          const float v = ck[r], w = __shfl_xor(v, 1);
          ck[r] = v * cs[0] + sgn * w * cs[1];
        }
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int kr = 32 * mb + c_row(r, lane);
        if (kr < rows) {
          const int j = start + r0 + kr;
          gstore(Kh + (((int64_t)(j >> 6) * H + h) * KT + (j & 63)) * d_h + dd, __builtin_bit_cast(bf16_t, (__bf16)ck[r]));
        }
      }
    }
  }
}

// fp32: for d_kv <= 64 the kept rows are staged in LDS (sK, sV: 64 rows of
// F32_STAGE_KV + 4 floats each), and so is each block of 64 rows of W_k^T or
// W_v^T (sW: 64 x (d_kv + 1) floats, the odd pitch keeps the 64 lanes of a
// wave, one output column each, on distinct banks); a thread computes the
// output columns d0 + lane of the rows wave, wave + NT/64, ...  Otherwise
// plain FMA loops over the rows just written to the ring.
constexpr int F32_STAGE_KV = 64;
constexpr int F32_SP = F32_STAGE_KV + 4;   // row pitch: 16-byte aligned rows
constexpr int F32_WP = F32_STAGE_KV + 1;   // W block pitch

template <int NT>
__device__ __forceinline__ void append_f32(const Rs3CommitArgs& a, const BankDev& b, int o, int start, int r0,
                                           int rows, const int* src, float* sK, float* sV, float* sW) {
  const int tid = threadIdx.x;
  const int d_kv = b.d_kv, d_h = b.d_h, H = b.H, D = H * d_h;
  const bool stage = d_kv <= F32_STAGE_KV;
  const float* Km = (const float*)a.Kmem + (int64_t)o * a.kv_stride;
  const float* Vm = (const float*)a.Vmem + (int64_t)o * a.kv_stride;
  float* Kr = (float*)b.Kraw;
  float* Vr = (float*)b.Vraw;
  for (int q = tid; q < rows * d_kv; q += NT) {
    const int r = q / d_kv, c = q - r * d_kv;
    const int64_t j = start + r0 + r;
    float kv, vv;
    if (a.from_ring) {
      kv = gload(Kr + j * d_kv + c);
      vv = gload(Vr + j * d_kv + c);
    } else {
      const int cell = src[r];
      kv = gload(Km + (int64_t)cell * d_kv + c);
      vv = gload(Vm + (int64_t)cell * d_kv + c);
      gstore(Kr + j * d_kv + c, kv);
      gstore(Vr + j * d_kv + c, vv);
    }
    if (stage) {
      sK[r * F32_SP + c] = kv;
      sV[r * F32_SP + c] = vv;
    }
  }
  __syncthreads();   // also publishes the ring rows read back below
  const float* WkT = (const float*)a.WkT;
  const float* WvT = (const float*)a.WvT;
  float* Kh = (float*)b.Khat;
  float* Vh = (float*)b.Vhat;
  if (stage) {
    const int lane = tid & 63, wave = tid >> 6;
    for (int pass = 0; pass < 2; ++pass) {
      const float* WT = pass == 0 ? WkT : WvT;
      const float* sX = pass == 0 ? sK : sV;
      for (int d0 = 0; d0 < D; d0 += 64) {
        const int nd = min(64, D - d0);
        if (!a.absorb) {
          for (int q = tid; q < nd * d_kv; q += NT) {
            const int dd = q / d_kv, c = q - dd * d_kv;
            sW[dd * F32_WP + c] = gload(WT + (int64_t)(d0 + dd) * d_kv + c);
          }
          __syncthreads();
        }
        const int d = d0 + lane;
        if (lane < nd) {
          const int h = d / d_h, dd = d - h * d_h;
          for (int r = wave; r < rows; r += NT / 64) {
            float acc;
            if (a.absorb) {   // attention on the raw rows
              acc = sX[r * F32_SP + d];
            } else {
              float a0 = 0.f, a1 = 0.f;
              for (int c = 0; c < d_kv; c += 2) {   // d_kv is a multiple of 16
                a0 = fmaf(sX[r * F32_SP + c], sW[lane * F32_WP + c], a0);
                a1 = fmaf(sX[r * F32_SP + c + 1], sW[lane * F32_WP + c + 1], a1);
              }
              acc = a0 + a1;
            }
            const int j = start + r0 + r, tile = j >> 6, kk = j & 63;
            if (pass == 0)
              gstore(Kh + (((int64_t)tile * H + h) * KT + kk) * d_h + dd, acc);
            else
              gstore(Vh + (((int64_t)tile * H + h) * d_h + dd) * KT + vslot(kk), acc);
          }
        }
        if (!a.absorb) __syncthreads();   // the next block rewrites sW
      }
    }
  } else {
    for (int q = tid; q < rows * D; q += NT) {
      const int r = q / D, d = q - r * D;
      const int j = start + r0 + r;
      const float* kr = Kr + (int64_t)j * d_kv;
      const float* vr = Vr + (int64_t)j * d_kv;
      float sk, sv;
      if (a.absorb) {  // attention on the raw rows
        sk = gload(kr + d);
        sv = gload(vr + d);
      } else {
        const float* wk = WkT + (int64_t)d * d_kv;
        const float* wv = WvT + (int64_t)d * d_kv;
        sk = 0.f;
        sv = 0.f;
        for (int c = 0; c < d_kv; ++c) {
          sk = fmaf(gload(kr + c), gload(wk + c), sk);
          sv = fmaf(gload(vr + c), gload(wv + c), sv);
        }
      }
      const int tile = j >> 6, kk = j & 63, h = d / d_h, dd = d - h * d_h;
      gstore(Kh + (((int64_t)tile * H + h) * KT + kk) * d_h + dd, sk);
      gstore(Vh + (((int64_t)tile * H + h) * d_h + dd) * KT + vslot(kk), sv);
    }
  }
  if (a.rope) {
    // Eq. 7 on the key side: each K^ row written above turns by the factors
    // of the cell it was kept from
    __syncthreads();
    const int hp = d_h / 2;
    for (int q = tid; q < rows * (D / 2); q += NT) {
      const int r = q / (D / 2), d = 2 * (q - r * (D / 2));
      const int h = d / d_h, dd = d - h * d_h;
      const int j = start + r0 + r, tile = j >> 6, kk = j & 63;
      const int cell = min(max(src[r], 0), a.rope_mn - 1);
      const float* f = a.rope + ((int64_t)cell * hp + (dd >> 1)) * 2;
      float* kp = Kh + (((int64_t)tile * H + h) * KT + kk) * d_h + dd;
      const float xe = kp[0], xo = kp[1];
      kp[0] = xe * f[0] - xo * f[1];
      kp[1] = xe * f[1] + xo * f[0];
    }
  }
}

// ---------------------------------------------------------------------------
// Frame tables of up to CP_FMAX frames are staged in LDS (f_max <= 256 is
// checked on the host).
constexpr int CP_FMAX = 256;

// The commit of object o by one work-group of CP_THREADS threads: y = 0
// writes the new frame state, y >= 1 appends kept rows.  dyn: the dynamic
// LDS, frame table [CP_FMAX][4] int32, then the append's row stage.
template <bool BF16>
__device__ __forceinline__ void commit_block(const Rs3CommitArgs& a, int o, int y, int32_t* dyn) {
  int32_t* sfr = dyn;
  uint8_t* stage = (uint8_t*)(dyn + 4 * CP_FMAX);
  __shared__ CpShared sh;
  __shared__ int spos[64];
  const int tid = threadIdx.x;
  const BankDev& b = *a.banks[o];
  // the descriptor words the placement needs, in one batch of loads (each
  // read behind a branch would otherwise wait for the one before)
  asm volatile("" ::"s"(b.f_max), "s"(b.frames), "s"(b.hdr), "s"(b.cap), "s"(b.n_pin), "s"(b.pos));
  const int p = (int)((a.parity >> o) & 1);   // current copy of the frame state
  const int m = a.m, n = a.n, s = a.s, mn = m * n, W = n * s;
  const uint8_t* M = a.masks + (int64_t)o * (m * s) * W;
  const int cpt = (mn + CP_THREADS - 1) / CP_THREADS;   // thread t owns cells c0 = t*cpt ...
  const int c0 = tid * cpt;
  // frame table, header words and mask cells are independent: load together
  const int f_max = b.f_max;
  const int32_t fr_w = tid < 4 * f_max ? b.frames[4 * f_max * p + tid] : 0;
  int nf0 = 0, pin_end0 = 0;
  if (tid < 64) {
    nf0 = b.hdr[HDR_NFRAMES + HDR_COPY * p];
    pin_end0 = b.hdr[HDR_PINEND + HDR_COPY * p];
  }
  uint32_t bits = 0;
  if (s == 1 && cpt == 4 && c0 + 4 <= mn && ((((uintptr_t)M) + c0) & 3) == 0) {
    uint32_t t = *(const uint32_t*)(M + c0);
    t |= t >> 4;
    t |= t >> 2;
    t |= t >> 1;
    bits = (t & 1u) | ((t >> 7) & 2u) | ((t >> 14) & 4u) | ((t >> 21) & 8u);
  } else if (c0 < mn) {
    int yy = c0 / n, x = c0 - yy * n;
    for (int j = 0; j < cpt && c0 + j < mn; ++j) {
      if (M[(int64_t)(yy * s) * W + x * s]) bits |= 1u << j;
      if (++x == n) {
        x = 0;
        ++yy;
      }
    }
  }
  const int nc = c0 < mn ? min(cpt, mn - c0) : 0;   // cells of this thread
  int total;
  int before = cp_scan_bits(bits, cpt, sh.red, &total);
  if (total < a.fall_min || total > a.fall_max) {   // dense fall-through: every cell
    bits = nc == 32 ? ~0u : ((1u << nc) - 1u);
    before = c0 < mn ? c0 : mn;
    total = mn;
  }
  if (tid < 4 * f_max) sfr[tid] = fr_w;
  lds_barrier();
  if (tid < 64) {
    int nf = nf0, pin_end = pin_end0, keys = 0;
    const int start = place_frame_wave(b, sfr, nf0, pin_end0, total, a.t, a.pin, &nf, &pin_end, &keys);
    if (tid == 0) {
      sh.ok = start >= 0;
      sh.start = start;
      sh.len = nf;
      if (y == 0) {   // the new state goes to the other copy
        const int q = 1 - p;
        if (a.kept_count) a.kept_count[o] = total;
        if (start >= 0) {
          b.hdr[HDR_NFRAMES + HDR_COPY * q] = nf;
          b.hdr[HDR_PINEND + HDR_COPY * q] = pin_end;
          b.hdr[HDR_PSTART] = start;
          b.hdr[HDR_PLEN] = total;
          b.hdr[HDR_NKEYS] = keys;
        } else {
          b.hdr[HDR_NFRAMES + HDR_COPY * q] = nf0;
          b.hdr[HDR_PINEND + HDR_COPY * q] = pin_end0;
          b.hdr[HDR_PLEN] = -1;
          set_err(b.hdr, RS3_E_CAPACITY);
        }
      }
    }
  }
  lds_barrier();
  if (y == 0) {
    // frame table copy 1-p: the new table, or the unchanged one (the rule
    // returns before touching it when the frame does not fit)
    const int nfw = sh.ok ? sh.len : nf0;
    if (tid < 4 * nfw) b.frames[4 * f_max * (1 - p) + tid] = sfr[tid];
    if (sh.ok) rebuild_tiles(b, sfr, sh.len, sh);
    return;
  }
  if (!sh.ok) return;
  // kept rows [(y-1)*rows_per_wg, y*rows_per_wg) of the new frame, 64 per round
  const int start = sh.start;
  const int r_end = min(total, y * a.rows_per_wg);
  for (int r0 = (y - 1) * a.rows_per_wg; r0 < r_end; r0 += 64) {
    {   // kept cells of rows r0 .. r0+63
      int k = before;
      for (int j = 0; j < cpt; ++j)
        if (bits >> j & 1) {
          if (k >= r0 && k < r0 + 64) spos[k - r0] = c0 + j;
          ++k;
        }
    }
    lds_barrier();
    const int rows = min(64, total - r0);
    if (tid < rows) b.pos[start + r0 + tid] = spos[tid];
    if constexpr (BF16)
      append_bf16<CP_THREADS>(a, b, o, start, r0, rows, spos, (bf16_t*)stage);
    else
      append_f32<CP_THREADS>(a, b, o, start, r0, rows, spos, (float*)stage, (float*)stage + 64 * F32_SP,
                             (float*)stage + 2 * 64 * F32_SP);
    __syncthreads();   // the next round rewrites spos and the row stage
  }
}

// Kept rows appended per work-group: 64, or a multiple of 64 (appended in
// rounds) so that a call launches about 1024 work-groups -- every work-group
// scans the whole mask, which many-object calls would otherwise repeat
// thousands of times.
inline int commit_rows_per_wg(int n_obj, int mn) {
  constexpr int CP_MAX_WGS = 1024;
  const int64_t blocks64 = (int64_t)n_obj * ((mn + 63) / 64);
  return 64 * (int)((blocks64 + CP_MAX_WGS - 1) / CP_MAX_WGS);
}

inline size_t commit_stage_bytes(int dtype, int d_kv) {
  return dtype == RS3_BF16 ? (size_t)2 * 64 * (d_kv + 8) * 2 : (size_t)(2 * 64 * F32_SP + 64 * F32_WP) * 4;
}

}  // namespace rs3
