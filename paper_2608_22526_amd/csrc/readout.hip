// Read-sparse memory readout (Sec. 3.1, Eq. 6, with the residual reading:
// y = x + S(A), unselected rows returned unchanged).
//
// bf16 path (three kernels, plus a grid copy when Y is not X):
//   k_qproj    gather the selected rows of X and project them,
//              Q~ = X[sel] W_q * log2(e)/sqrt(d_h)  (32x32x16 bf16 MFMA);
//   k_attn     split-KV flash attention over the resident 64-key tiles of
//              the object's bank.  Each wave owns 32 queries and computes
//              the transposed logits S^T = K^ Q~^T, so the 32 logits of a
//              query sit in one lane (plus its partner lane l^32): the
//              online-softmax max and sum need one cross-lane exchange.  The
//              probabilities go straight from the accumulator registers into
//              the B operand of O^T += V^T P^T (the V^ tile is stored with
//              keys in MFMA slot order), K^/V^ tiles are staged in LDS;
//   k_combine  merges the key splits (log-sum-exp weights), multiplies by
//              W_o (MFMA), adds the residual and scatters y into Y[sel].
// fp32 path: one workgroup per selected row (FMA loops), for the small
// fp32 workloads that need 1e-4 agreement.
#include "rs3_internal.h"

namespace rs3 {

__device__ __forceinline__ int sel_count_of(const Rs3ReadoutArgs& a, int o, BankDev& b,
                                            bool report) {
  int cnt = a.sel_count[a.sel_stride ? o : 0];
  if (cnt > a.max_sel || cnt < 0) {
    if (report) set_err(b.hdr, RS3_E_INVALID);
    cnt = cnt < 0 ? 0 : a.max_sel;
  }
  return cnt;
}

// True iff sel[r] is in range and larger than its predecessor.
__device__ __forceinline__ bool sel_ok(const int32_t* sel, int r, int mn) {
  int i = sel[r];
  return i >= 0 && i < mn && (r == 0 || sel[r - 1] < i);
}

// ---------------------------------------------------------------------------
// grid (n_obj, ceil(max_sel/64), D/64), block 256: 64 rows x 64 columns.
__global__ __launch_bounds__(256) void k_qproj(Rs3ReadoutArgs a) {
  const int o = blockIdx.x, r0 = blockIdx.y * 64, c0 = blockIdx.z * 64;
  BankDev& b = *a.banks[o];
  const bool report = blockIdx.z == 0 && threadIdx.x == 0;
  const int cnt = sel_count_of(a, o, b, report && blockIdx.y == 0);
  if (r0 >= cnt) return;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, g = lane >> 5;
  const int32_t* sel = a.sel_idx + (int64_t)o * a.sel_stride;
  const int C = a.C, D = a.D;
  const bf16_t* X = (const bf16_t*)a.X + (int64_t)o * a.x_stride;
  const int row = r0 + 32 * (wave & 1) + (lane & 31);
  const bool rv = row < cnt;
  if (blockIdx.z == 0 && threadIdx.x < 64 && r0 + threadIdx.x < cnt &&
      !sel_ok(sel, r0 + threadIdx.x, a.mn))
    set_err(b.hdr, RS3_E_INVALID);
  int src = rv ? sel[row] : 0;
  if (src < 0 || src >= a.mn) src = 0;
  const bf16_t* xr = X + (int64_t)src * C;
  const int col = c0 + 32 * (wave >> 1) + (lane & 31);
  const bf16_t* wr = (const bf16_t*)a.WqT + (int64_t)col * C;
  f32x16 acc = {};
  for (int k = 0; k < C; k += 16) {
    u32x4 av = *(const u32x4*)(xr + k + 8 * g);
    u32x4 bv = *(const u32x4*)(wr + k + 8 * g);
    acc = mfma32(av, bv, acc);
  }
  bf16_t* Q = (bf16_t*)a.Q + (int64_t)o * a.max_sel * D;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    int rr = r0 + 32 * (wave & 1) + c_row(r, lane);
    if (rr < cnt) Q[(int64_t)rr * D + col] = f2bf(acc[r] * a.qscale);
  }
}

// ---------------------------------------------------------------------------
// LDS tiles are stored without padding; the 16-byte chunks of each row are
// permuted by an XOR with a few row bits so that the 32 (or 8) rows read by
// one MFMA operand load land in distinct LDS banks.
template <int CPR>
__device__ __forceinline__ int chunk_swz(int r) {
  return CPR >= 8 ? (r & 7) : ((r >> 1) & (CPR - 1));
}

// Direct-to-LDS loads of resident tile t (K^ then V^ of head h) into a stage.
template <int DH>
__device__ __forceinline__ void attn_issue(const bf16_t* Kh, const bf16_t* Vh, const TileEnt* tiles, int t,
                                           int h, int H, uint8_t* lds, int stage, int wave, const int* koff,
                                           const int* voff) {
  constexpr int KB = KT * DH * 2;
  constexpr int NI = DH / 32;
  const int tile = tiles[t].tile;
  const bf16_t* kg = Kh + ((int64_t)tile * H + h) * (KT * DH);
  const bf16_t* vg = Vh + ((int64_t)tile * H + h) * (DH * KT);
  uint8_t* kd = lds + stage * 2 * KB;
  uint8_t* vd = kd + KB;
#pragma unroll
  for (int j = 0; j < NI; ++j) {
    const int i = wave + 4 * j;
    __builtin_amdgcn_global_load_lds(kg + koff[j], kd + i * 1024, 16, 0, 0);
    __builtin_amdgcn_global_load_lds(vg + voff[j], vd + i * 1024, 16, 0, 0);
  }
}

// grid 8*n_qt*ceil(G/8) with G = n_obj*H*S key groups, block 256 (4 waves x
// 32 queries).  Block b -> key group 8*((b>>3)/n_qt) + (b&7), query tile
// (b>>3) % n_qt, so all query tiles of one key group share an XCD (and its L2).
// K^/V^ tiles are streamed into two LDS stages with direct-to-LDS loads
// (global_load_lds_dwordx4): the next tile is in flight while the current one
// is multiplied.
template <int DH>
__global__ __launch_bounds__(256) void k_attn(Rs3ReadoutArgs a, int G) {
  constexpr int CPRK = DH / 8;            // 16-byte chunks per K row
  constexpr int KB = KT * DH * 2;         // bytes of one K (or V) tile
  constexpr int STAGE = 2 * KB;
  constexpr int NI = DH / 32;             // DMA instructions per wave per tensor
  __shared__ __attribute__((aligned(1024))) uint8_t lds[2 * STAGE];
  const int bid = blockIdx.x;
  const int rest = bid >> 3;
  const int qt = rest % a.n_qt;
  const int kvg = (rest / a.n_qt) * 8 + (bid & 7);
  if (kvg >= G) return;
  const int s = kvg % a.S, oh = kvg / a.S, h = oh % a.H, o = oh / a.H;
  BankDev& b = *a.banks[o];
  const int cnt = sel_count_of(a, o, b, false);
  const int row0 = qt * 128;
  if (row0 >= cnt) return;
  const int ntiles = b.hdr[HDR_NTILES];
  const int tps = split_tiles(ntiles, a.S);
  const int tb = min(s * tps, ntiles), te = min(tb + tps, ntiles);
  if (tb >= te) return;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, g = lane >> 5;
  const bf16_t* Kh = (const bf16_t*)b.Khat;
  const bf16_t* Vh = (const bf16_t*)b.Vhat;
  const TileEnt* tiles = b.tiles;
  const int H = a.H;

  // per-lane DMA source offsets inside a tile (elements), fixed for all tiles
  int koff[NI], voff[NI];
#pragma unroll
  for (int j = 0; j < NI; ++j) {
    const int p = (wave + 4 * j) * 64 + lane;          // LDS chunk written by this lane
    const int r = p / CPRK, pc = p % CPRK;
    koff[j] = (r * CPRK + (pc ^ chunk_swz<CPRK>(r))) * 8;
    const int rv = p >> 3, pcv = p & 7;
    voff[j] = (rv * 8 + (pcv ^ (rv & 7))) * 8;
  }
  attn_issue<DH>(Kh, Vh, tiles, tb, h, H, lds, 0, wave, koff, voff);

  const int qrow = row0 + 32 * wave + (lane & 31);
  const bool qv = qrow < cnt;
  const bf16_t* Qp = (const bf16_t*)a.Q + ((int64_t)o * a.max_sel + (qv ? qrow : 0)) * a.D + h * DH;
  u32x4 qreg[DH / 16];
#pragma unroll
  for (int ks = 0; ks < DH / 16; ++ks)
    qreg[ks] = qv ? *(const u32x4*)(Qp + 16 * ks + 8 * g) : u32x4{0, 0, 0, 0};

  f32x16 acc[DH / 32];
#pragma unroll
  for (int dt = 0; dt < DH / 32; ++dt) acc[dt] = f32x16{};
  float m_run = -INFINITY, l_run = 0.f;
  // LDS read offsets of this lane's operand rows
  int kro[2], ksw[2];
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) {
    const int r = 32 * kb + (lane & 31);
    kro[kb] = r * CPRK * 16;
    ksw[kb] = chunk_swz<CPRK>(r);
  }
  const int vsw = lane & 7;
  uint64_t msk = tiles[tb].mask;

  for (int t = tb; t < te; ++t) {
    const int st = (t - tb) & 1;
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    uint64_t msk_next = 0;
    if (t + 1 < te) {
      attn_issue<DH>(Kh, Vh, tiles, t + 1, h, H, lds, st ^ 1, wave, koff, voff);
      msk_next = tiles[t + 1].mask;
    }
    const uint8_t* Kl = lds + st * STAGE;
    const uint8_t* Vl = Kl + KB;

    f32x16 sc[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      sc[kb] = f32x16{};
#pragma unroll
      for (int ks = 0; ks < DH / 16; ++ks) {
        const int c = (2 * ks + g) ^ ksw[kb];
        sc[kb] = mfma32(*(const u32x4*)(Kl + kro[kb] + c * 16), qreg[ks], sc[kb]);
      }
    }
    float mx = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = 32 * kb + c_row(r, lane);
        const float v = (msk >> key & 1ull) ? sc[kb][r] : -INFINITY;
        sc[kb][r] = v;
        mx = fmaxf(mx, v);
      }
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    const float m_new = fmaxf(m_run, mx);
    const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
    const float alpha = __builtin_amdgcn_exp2f(m_run - m_use);
    float psum = 0.f;
    u32x4 pk[2][2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int hf = 0; hf < 2; ++hf)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const float p0 = __builtin_amdgcn_exp2f(sc[kb][8 * hf + 2 * j] - m_use);
          const float p1 = __builtin_amdgcn_exp2f(sc[kb][8 * hf + 2 * j + 1] - m_use);
          psum += p0 + p1;
          pk[kb][hf][j] = pack_bf16x2(p0, p1);
        }
    l_run = l_run * alpha + psum;
    m_run = m_new;
#pragma unroll
    for (int dt = 0; dt < DH / 32; ++dt) {
      acc[dt] *= alpha;
      const uint8_t* vrow = Vl + (32 * dt + (lane & 31)) * 128;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {
          const int c = (4 * kb + 2 * hf + g) ^ vsw;
          acc[dt] = mfma32(*(const u32x4*)(vrow + c * 16), pk[kb][hf], acc[dt]);
        }
    }
    msk = msk_next;
  }
  const float l_tot = l_run + __shfl_xor(l_run, 32, 64);
  if (!qv) return;
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  const int64_t prow = ((int64_t)o * a.S + s) * a.max_sel + qrow;
  bf16_t* op = (bf16_t*)a.Opart + prow * a.D + h * DH;
#pragma unroll
  for (int dt = 0; dt < DH / 32; ++dt)
#pragma unroll
    for (int q4 = 0; q4 < 4; ++q4) {
      const int d = 32 * dt + 8 * q4 + 4 * g;
      u32x2 w;
      w[0] = pack_bf16x2(acc[dt][4 * q4] * inv, acc[dt][4 * q4 + 1] * inv);
      w[1] = pack_bf16x2(acc[dt][4 * q4 + 2] * inv, acc[dt][4 * q4 + 3] * inv);
      *(u32x2*)(op + d) = w;
    }
  if (g == 0) {
    float* ml = a.ML + (prow * a.H + h) * 2;
    ml[0] = m_run;
    ml[1] = l_tot;
  }
}

// ---------------------------------------------------------------------------
template <typename OutT>
__device__ __forceinline__ void store_out(OutT* p, float v);
template <>
__device__ __forceinline__ void store_out<bf16_t>(bf16_t* p, float v) { *p = f2bf(v); }
template <>
__device__ __forceinline__ void store_out<float>(float* p, float v) { *p = v; }

template <typename OutT>
__device__ __forceinline__ void copy_out(OutT* p, bf16_t x);
template <>
__device__ __forceinline__ void copy_out<bf16_t>(bf16_t* p, bf16_t x) { *p = x; }
template <>
__device__ __forceinline__ void copy_out<float>(float* p, bf16_t x) { *p = bf2f(x); }

// grid (n_obj, ceil(max_sel/16)), block 512.  Dynamic LDS: merged O rows
// (16 x (D+8) bf16) then the per-(row, head, split) weights (16*H*S floats).
// 1. every (row, head, split) triple loads its (m, l) pair; per (row, head)
//    the merge weights w_s = 2^(m_s - M) l_s / sum are formed in LDS;
// 2. each thread merges one 8-column chunk over all active splits;
// 3. y = x + O W_o on a 32x32x16 MFMA whose rows 16..31 are zero.
constexpr int CB_ROWS = 16;
constexpr int CB_THREADS = 512;
template <typename OutT>
__global__ __launch_bounds__(CB_THREADS) void k_combine(Rs3ReadoutArgs a) {
  extern __shared__ __attribute__((aligned(16))) uint8_t cl[];
  const int o = blockIdx.x, r0 = blockIdx.y * CB_ROWS;
  BankDev& b = *a.banks[o];
  const int cnt = sel_count_of(a, o, b, false);
  if (r0 >= cnt) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, g = lane >> 5;
  const int D = a.D, C = a.C, H = a.H, d_h = a.d_h, S = a.S, OS = D + 8;
  bf16_t* Os = (bf16_t*)cl;
  float* wts = (float*)(cl + ((CB_ROWS * OS * 2 + 15) & ~15));
  const int ntiles = b.hdr[HDR_NTILES];
  const int SA = ntiles > 0 ? active_splits(ntiles, S) : 0;
  const int32_t* sel = a.sel_idx + (int64_t)o * a.sel_stride;
  const int64_t base = (int64_t)o * S * a.max_sel;

  // 1a. (m, l) of every active split: wts[(rr*H + h)*SA + s] = m, then l after
  for (int q = tid; q < CB_ROWS * H * SA; q += CB_THREADS) {
    const int s = q % SA, rh = q / SA, h = rh % H, rr = rh / H, row = r0 + rr;
    float m = -INFINITY, l = 0.f;
    if (row < cnt) {
      const float* ml = a.ML + ((base + (int64_t)s * a.max_sel + row) * H + h) * 2;
      m = ml[0];
      l = ml[1];
    }
    wts[q] = m;
    wts[CB_ROWS * H * SA + q] = l;
  }
  __syncthreads();
  // 1b. weights per (row, head)
  for (int rh = tid; rh < CB_ROWS * H; rh += CB_THREADS) {
    float* mv = wts + rh * SA;
    const float* lv = wts + CB_ROWS * H * SA + rh * SA;
    float M = -INFINITY;
    for (int s = 0; s < SA; ++s) M = fmaxf(M, mv[s]);
    float W = 0.f;
    if (M != -INFINITY)
      for (int s = 0; s < SA; ++s) W += __builtin_amdgcn_exp2f(mv[s] - M) * lv[s];
    const float iw = W > 0.f ? 1.f / W : 0.f;
    for (int s = 0; s < SA; ++s) mv[s] = (M != -INFINITY) ? __builtin_amdgcn_exp2f(mv[s] - M) * lv[s] * iw : 0.f;
  }
  __syncthreads();
  // 2. merged O rows into LDS
  const bf16_t* Op = (const bf16_t*)a.Opart;
  const int cpr = D / 8;
  for (int q = tid; q < CB_ROWS * cpr; q += CB_THREADS) {
    const int rr = q / cpr, d0 = 8 * (q - rr * cpr), h = d0 / d_h, row = r0 + rr;
    float acc8[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    if (row < cnt) {
      const float* w = wts + (rr * H + h) * SA;
      const bf16_t* src = Op + (base + row) * D + d0;
      const int64_t sstride = (int64_t)a.max_sel * D;
#pragma unroll 8
      for (int s = 0; s < SA; ++s) {
        const float ws = w[s];
        const u32x4 v = *(const u32x4*)(src + s * sstride);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          acc8[2 * j] += ws * __uint_as_float(v[j] << 16);
          acc8[2 * j + 1] += ws * __uint_as_float(v[j] & 0xffff0000u);
        }
      }
    }
    u32x4 pk;
#pragma unroll
    for (int j = 0; j < 4; ++j) pk[j] = pack_bf16x2(acc8[2 * j], acc8[2 * j + 1]);
    *(u32x4*)&Os[rr * OS + d0] = pk;
  }
  __syncthreads();
  // 3. y = x + O W_o for the block's rows, columns split over the waves
  const bf16_t* X = (const bf16_t*)a.X + (int64_t)o * a.x_stride;
  OutT* Y = (OutT*)a.Y + (int64_t)o * a.y_stride;
  const bf16_t* WoT = (const bf16_t*)a.WoT;
  const bool arow = (lane & 31) < CB_ROWS;
  const bf16_t* orow = &Os[(arow ? (lane & 31) : 0) * OS + 8 * g];
  for (int nb = wave; nb < C / 32; nb += CB_THREADS / 64) {
    const int col = 32 * nb + (lane & 31);
    const bf16_t* wr = WoT + (int64_t)col * D;
    f32x16 acc = {};
    for (int k = 0; k < D; k += 16) {
      const u32x4 av = arow ? *(const u32x4*)(orow + k) : u32x4{0, 0, 0, 0};
      acc = mfma32(av, *(const u32x4*)(wr + k + 8 * g), acc);
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int rr = c_row(r, lane);
      const int row = r0 + rr;
      if (rr >= CB_ROWS || row >= cnt || !sel_ok(sel, row, a.mn)) continue;
      const int64_t off = (int64_t)sel[row] * C + col;
      const bf16_t xv = X[off];
      if (ntiles == 0)
        copy_out<OutT>(&Y[off], xv);
      else
        store_out<OutT>(&Y[off], bf2f(xv) + acc[r]);
    }
  }
}

// Y[o] = X[o] (or the shared X) for every cell, converting to OutT.
template <typename InT, typename OutT>
__global__ __launch_bounds__(256) void k_copy_grid(const InT* X, int64_t x_stride, OutT* Y,
                                                   int64_t y_stride, int64_t count) {
  const int o = blockIdx.y;
  const InT* x = X + (int64_t)o * x_stride;
  OutT* y = Y + (int64_t)o * y_stride;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < count; i += (int64_t)gridDim.x * 256) {
    if constexpr (sizeof(InT) == sizeof(OutT)) {
      y[i] = x[i];
    } else {
      copy_out<OutT>(&y[i], x[i]);
    }
  }
}

// 16-byte vector copy for same-type grids (count16 = bytes / 16 per object).
__global__ __launch_bounds__(256) void k_copy_grid16(const u32x4* X, int64_t x_stride16, u32x4* Y,
                                                     int64_t y_stride16, int64_t count16) {
  const int o = blockIdx.y;
  const u32x4* x = X + (int64_t)o * x_stride16;
  u32x4* y = Y + (int64_t)o * y_stride16;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < count16; i += (int64_t)gridDim.x * 256)
    y[i] = x[i];
}

// ---------------------------------------------------------------------------
// fp32 path: grid (n_obj, max_sel), block 256, one selected row per block.
__global__ __launch_bounds__(256) void k_readout_f32(Rs3ReadoutArgs a) {
  extern __shared__ float sm[];
  __shared__ float pr[KT];
  __shared__ float st[4];  // m_run, l_run, alpha
  const int o = blockIdx.x, r = blockIdx.y, tid = threadIdx.x;
  BankDev& b = *a.banks[o];
  const int cnt = sel_count_of(a, o, b, r == 0 && tid == 0);
  if (r >= cnt) return;
  const int32_t* sel = a.sel_idx + (int64_t)o * a.sel_stride;
  if (!sel_ok(sel, r, a.mn)) {
    if (tid == 0) set_err(b.hdr, RS3_E_INVALID);
    return;
  }
  const int C = a.C, D = a.D, H = a.H, d_h = a.d_h;
  float* xs = sm;        // [C]
  float* q = sm + C;     // [D]
  float* oacc = q + D;   // [D]
  const int i = sel[r];
  const float* x = (const float*)a.X + (int64_t)o * a.x_stride + (int64_t)i * C;
  float* y = (float*)a.Y + (int64_t)o * a.y_stride + (int64_t)i * C;
  for (int c = tid; c < C; c += 256) xs[c] = x[c];
  const int ntiles = b.hdr[HDR_NTILES];
  __syncthreads();
  if (ntiles == 0) {
    for (int c = tid; c < C; c += 256) y[c] = xs[c];
    return;
  }
  const float* WqT = (const float*)a.WqT;
  for (int d = tid; d < D; d += 256) {
    float s = 0.f;
    for (int c = 0; c < C; ++c) s = fmaf(xs[c], WqT[(int64_t)d * C + c], s);
    q[d] = s * a.qscale;
    oacc[d] = 0.f;
  }
  __syncthreads();
  const float* Kh = (const float*)b.Khat;
  const float* Vh = (const float*)b.Vhat;
  for (int h = 0; h < H; ++h) {
    if (tid == 0) {
      st[0] = -INFINITY;
      st[1] = 0.f;
    }
    __syncthreads();
    for (int t = 0; t < ntiles; ++t) {
      const TileEnt ent = b.tiles[t];
      const float* kg = Kh + ((int64_t)ent.tile * H + h) * (KT * d_h);
      const float* vg = Vh + ((int64_t)ent.tile * H + h) * (d_h * KT);
      if (tid < KT) {
        float s = -INFINITY;
        if (ent.mask >> tid & 1ull) {
          s = 0.f;
          for (int u = 0; u < d_h; ++u) s = fmaf(q[h * d_h + u], kg[tid * d_h + u], s);
        }
        pr[tid] = s;
      }
      __syncthreads();
      if (tid == 0) {
        float mx = -INFINITY;
        for (int j = 0; j < KT; ++j) mx = fmaxf(mx, pr[j]);
        const float m_new = fmaxf(st[0], mx);
        const float alpha = exp2f(st[0] - m_new);
        float ps = 0.f;
        for (int j = 0; j < KT; ++j) {
          const float p = exp2f(pr[j] - m_new);
          pr[j] = p;
          ps += p;
        }
        st[1] = st[1] * alpha + ps;
        st[0] = m_new;
        st[2] = alpha;
      }
      __syncthreads();
      const float alpha = st[2];
      for (int u = tid; u < d_h; u += 256) {
        float acc = oacc[h * d_h + u] * alpha;
        for (int j = 0; j < KT; ++j) acc = fmaf(pr[j], vg[u * KT + vslot(j)], acc);
        oacc[h * d_h + u] = acc;
      }
      __syncthreads();
    }
    const float inv = 1.f / st[1];
    for (int u = tid; u < d_h; u += 256) oacc[h * d_h + u] *= inv;
    __syncthreads();
  }
  const float* WoT = (const float*)a.WoT;
  for (int c = tid; c < C; c += 256) {
    float s = 0.f;
    for (int d = 0; d < D; ++d) s = fmaf(oacc[d], WoT[(int64_t)c * D + d], s);
    y[c] = xs[c] + s;
  }
}

}  // namespace rs3

using namespace rs3;

static size_t combine_lds_bytes(int D, int H, int S) {
  return (((size_t)CB_ROWS * (D + 8) * 2 + 15) & ~(size_t)15) + (size_t)2 * CB_ROWS * H * S * 4;
}

hipError_t rs3_launch_readout(const Rs3ReadoutArgs& a, int dtype, hipStream_t st) {
  const int64_t cells = (int64_t)a.mn * a.C;
  const bool in_place = a.Y == a.X && !a.y_fp32;
  if (!in_place) {
    dim3 grid((unsigned)((cells + 255) / 256 < 2048 ? (cells + 255) / 256 : 2048), a.n_obj);
    if (dtype == RS3_BF16 && !a.y_fp32) {
      int64_t c16 = cells * 2 / 16;
      dim3 g16((unsigned)((c16 + 255) / 256 < 2048 ? (c16 + 255) / 256 : 2048), a.n_obj);
      RS3_LAUNCH(RS3_K_COPY, st, k_copy_grid16, g16, dim3(256), 0, st, (const u32x4*)a.X, a.x_stride * 2 / 16,
                         (u32x4*)a.Y, a.y_stride * 2 / 16, c16);
    } else if (dtype == RS3_BF16) {
      RS3_LAUNCH(RS3_K_COPY, st, (k_copy_grid<bf16_t, float>), grid, dim3(256), 0, st, (const bf16_t*)a.X,
                         a.x_stride, (float*)a.Y, a.y_stride, cells);
    } else {
      int64_t c16 = cells * 4 / 16;
      dim3 g16((unsigned)((c16 + 255) / 256 < 2048 ? (c16 + 255) / 256 : 2048), a.n_obj);
      RS3_LAUNCH(RS3_K_COPY, st, k_copy_grid16, g16, dim3(256), 0, st, (const u32x4*)a.X, a.x_stride * 4 / 16,
                         (u32x4*)a.Y, a.y_stride * 4 / 16, c16);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (a.max_sel == 0) return hipSuccess;
  if (dtype == RS3_F32) {
    size_t lds = (size_t)(a.C + 2 * a.D) * 4;
    RS3_LAUNCH(RS3_K_READOUT_F32, st, k_readout_f32, dim3(a.n_obj, a.max_sel), dim3(256), lds, st, a);
    return hipGetLastError();
  }
  RS3_LAUNCH(RS3_K_QPROJ, st, k_qproj, dim3(a.n_obj, (a.max_sel + 63) / 64, a.D / 64), dim3(256), 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int G = a.n_obj * a.H * a.S;
  const int nblk = 8 * a.n_qt * ((G + 7) / 8);
  switch (a.d_h) {
    case 32: RS3_LAUNCH(RS3_K_ATTN, st, k_attn<32>, dim3(nblk), dim3(256), 0, st, a, G); break;
    case 64: RS3_LAUNCH(RS3_K_ATTN, st, k_attn<64>, dim3(nblk), dim3(256), 0, st, a, G); break;
    case 128: RS3_LAUNCH(RS3_K_ATTN, st, k_attn<128>, dim3(nblk), dim3(256), 0, st, a, G); break;
    case 256: RS3_LAUNCH(RS3_K_ATTN, st, k_attn<256>, dim3(nblk), dim3(256), 0, st, a, G); break;
    default: return hipErrorInvalidValue;
  }
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  const size_t lds = combine_lds_bytes(a.D, a.H, a.S);
  const dim3 cgrid(a.n_obj, (a.max_sel + CB_ROWS - 1) / CB_ROWS);
  if (a.y_fp32)
    RS3_LAUNCH(RS3_K_COMBINE, st, k_combine<float>, cgrid, dim3(CB_THREADS), lds, st, a);
  else
    RS3_LAUNCH(RS3_K_COMBINE, st, k_combine<bf16_t>, cgrid, dim3(CB_THREADS), lds, st, a);
  return hipGetLastError();
}

hipError_t rs3_readout_setup() {
  // H * S <= RS3_MAX_SPLITS_X_HEADS and D <= 1024 (checked on the host)
  const int max_lds = (int)combine_lds_bytes(1024, 1, RS3_MAX_SPLITS_X_HEADS);
  hipError_t e = hipFuncSetAttribute((const void*)k_combine<bf16_t>, hipFuncAttributeMaxDynamicSharedMemorySize,
                                     max_lds);
  if (e != hipSuccess) return e;
  return hipFuncSetAttribute((const void*)k_combine<float>, hipFuncAttributeMaxDynamicSharedMemorySize, max_lds);
}
