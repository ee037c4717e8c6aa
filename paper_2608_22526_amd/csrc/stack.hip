// The L-layer memory-attention stack on the kept queries (Sec. 3.1, "Sparse
// memory attention": the sparse readout applies at the input of each layer
// of the memory-attention stack, not only the first).  The rows
// are gathered once before the first layer and scattered once after the
// last; in between, every layer is
//     z += SA(LN1(z))  among the kept rows      (one-frame bank of the kept rows)
//     z += CA(LN2(z))  against the memory bank  (the readout of Eq. 6, absorbed)
//     z += W2 relu(W1 LN3(z))
// with the residual stream z in fp32 and every matrix product on bf16 MFMA
// (32x32x16, fp32 accumulation).
//
// The attentions run on the readout's split-KV attention kernel unchanged.
// The self-attention's keys and values are laid out by the QKV product's
// epilogue as a bank of one frame whose tiles are the 64-row blocks of the
// kept set; the cross-attention reads the real ring bank, whose rows a layer
// of one absorbed head uses as they are (W_q W_k^T on the query side,
// W_v W_o on the output side), so one bank serves every layer.
//
// Launches of one layer (n kept rows; the first layer's LN1 comes from the
// gather launch, every later one from the previous layer's last launch):
//   k_stk_qkv      64x64 tiles: LN1 rows x [W_qs | W_ks | W_vs] -> queries,
//                  key and value tiles of the self-attention's bank
//   k_attn         self-attention; k_stk_merge merges its key splits
//   k_stk_post_sa  32 whole rows per work-group: z += O W_os, LN2, queries of
//                  the cross-attention (x W_q W_k^T)
//   k_attn         cross-attention; k_stk_merge merges its key splits
//   k_stk_mlp      32 rows x 128 hidden units per work-group: z' = z + O W_vo
//                  (kept by the first hidden chunk), LN3, relu(. W_1[:, chunk])
//                  W_2[chunk, :] -> an fp32 partial per chunk
//   k_stk_rows     z = z' + the partials in chunk order, then the next
//                  layer's LN1, or after the last layer the scatter to Y
// Weights are stored in MFMA operand order (pack_b on the host): the B
// operand of one 32-column block and one 16-deep step is 64 lanes x 16
// bytes, contiguous, so every weight load of a wave is one 1 KB run.
#include "device_util.h"

namespace rs3 {

constexpr int SG_C = 256;    // d_model of the stack
constexpr int SG_PITCH = SG_C + 8;   // bf16 elements per LDS row of a 256-wide A operand
constexpr float SG_LN_EPS = 1e-5f;

// B operand of the packed weight Wp (KS 16-deep steps) for 32-column block
// nb and step ks: lane l holds column 32*nb + l%32, rows 16*ks + 8*(l/32) .. +7.
__device__ __forceinline__ u32x4 ldb(const bf16_t* Wp, int KS, int nb, int ks, int lane) {
  return gload((const u32x4*)(Wp + (((int64_t)nb * KS + ks) * 64 + lane) * 8));
}

// A operand from a row-major LDS tile: rows r0 + l%32, columns 16*ks + 8*(l/32) .. +7.
__device__ __forceinline__ u32x4 lda(const bf16_t* As, int pitch, int r0, int ks, int lane) {
  return *(const u32x4*)(As + (r0 + (lane & 31)) * pitch + 16 * ks + 8 * (lane >> 5));
}

// LayerNorm of one 256-wide row held 4 channels per lane (every lane of the
// wave holds a quarter-row slice), with gain g and shift b: bf16 pairs.
__device__ __forceinline__ u32x2 ln_row(f32x4 z, const f32x4& g, const f32x4& b) {
  const float mean = wave_sum(z[0] + z[1] + z[2] + z[3]) * (1.f / SG_C);
  z -= mean;
  const float var = wave_sum(z[0] * z[0] + z[1] * z[1] + z[2] * z[2] + z[3] * z[3]) * (1.f / SG_C);
  const f32x4 y = z * (1.f / sqrtf(var + SG_LN_EPS)) * g + b;
  return u32x2{pack_bf16x2(y[0], y[1]), pack_bf16x2(y[2], y[3])};
}

// Kept-row count of the call, clamped into [0, M]; a count outside that
// range is reported in the bank's error word by work-group (0, 0).
__device__ __forceinline__ int stk_count(const StkArgs& p) {
  int cnt = gload(p.count);
  if (cnt < 0 || cnt > p.M) {
    if (blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x == 0) set_err(p.err_hdr, RS3_E_INVALID);
    cnt = cnt < 0 ? 0 : p.M;
  }
  return cnt;
}

// Cell of kept row r, or -1 for an entry out of range or not above its
// predecessor (such rows are reported and never written to Y).
__device__ __forceinline__ int stk_cell(const StkArgs& p, int r) {
  const int i = gload(p.sel + r);
  const int prev = r > 0 ? gload(p.sel + r - 1) : -1;
  return (i >= 0 && i < p.mn && prev < i) ? i : -1;
}

// ---- prologues: the A chunk [64][kn] of rows row0.. in LDS (bf16) ----------
// grid ceil(M*D_att/8 / 256), block 256: one thread per (kept row, 8 columns)
// merges the attention's key splits (partials O/l and (m, l) per split, row
// and head: Opart [S][M][D_att], ML [S][M][H_att][2]) by log-sum-exp into the
// normalised bf16 rows mout [M][D_att].  The splits are loaded eight at a time
// without branches (split indices past S re-read the last split and are
// masked); a split without keys holds l = 0 and adds nothing, its O words
// (never written) replaced by zero; a row with no key at all gets O = 0.
__global__ __launch_bounds__(256) void k_stk_merge(StkArgs p) {
  const int D = p.D_att, cpr = D / 8;
  const int64_t it = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (it >= (int64_t)p.M * cpr) return;
  const int row = (int)(it / cpr), d0 = 8 * (int)(it - (int64_t)row * cpr), h = d0 / p.d_att;
  const int cnt = stk_count(p);
  if (row >= cnt) return;
  float M = -INFINITY, W = 0.f;
  float acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  typedef float f32x2 __attribute__((ext_vector_type(2)));
  for (int s0 = 0; s0 < p.S; s0 += 8) {
    f32x2 ml[8];
    u32x4 v[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int64_t prow = (int64_t)min(s0 + i, p.S - 1) * p.M + row;
      ml[i] = gload((const f32x2*)(p.ML + (prow * p.H_att + h) * 2));
      v[i] = gload((const u32x4*)(p.Opart + prow * D + d0));
    }
    bool on[8];
    float mb = -INFINITY;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      on[i] = s0 + i < p.S && ml[i][1] > 0.f;
      mb = __builtin_elementwise_maximum(mb, on[i] ? ml[i][0] : -INFINITY);
    }
    if (mb == -INFINITY) continue;
    const float Mn = __builtin_elementwise_maximum(M, mb);
    const float sc = __builtin_amdgcn_exp2f(M - Mn);   // 0 while M = -inf
    W *= sc;
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] *= sc;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float w = on[i] ? __builtin_amdgcn_exp2f(ml[i][0] - Mn) * ml[i][1] : 0.f;
      W += w;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const uint32_t x = on[i] ? v[i][e] : 0u;
        acc[2 * e] += w * __uint_as_float(x << 16);
        acc[2 * e + 1] += w * __uint_as_float(x & 0xffff0000u);
      }
    }
    M = Mn;
  }
  const float inv = W > 0.f ? 1.f / W : 0.f;
  u32x4 out;
#pragma unroll
  for (int e = 0; e < 4; ++e) out[e] = pack_bf16x2(acc[2 * e] * inv, acc[2 * e + 1] * inv);
  *(u32x4*)(p.mout + (int64_t)row * D + d0) = out;
}

// The self-attention's one-frame bank: descriptor, header (tile and key
// counts from the device count) and tile list, by work-group (0, 0) of the
// first layer's QKV product.
__device__ __forceinline__ void write_self_bank(const StkArgs& p, int cnt) {
  const int tid = threadIdx.x;
  const int ntiles = (cnt + KT - 1) / KT;
  if (tid == 0) {
    BankDev d = {};
    d.cap = p.ntile_cap * KT;
    d.f_max = 1;
    d.d_kv = p.dhs;
    d.H = p.Hs;
    d.d_h = p.dhs;
    d.dtype = RS3_BF16;
    d.n_tiles_cap = p.ntile_cap;
    d.Khat = p.Kh;
    d.Vhat = p.Vh;
    d.hdr = p.shdr;
    d.tiles = p.tiles;
    *p.desc = d;
  }
  if (tid < HDR_WORDS) {
    int v = 0;
    if (tid == HDR_NFRAMES) v = ntiles > 0;
    if (tid == HDR_PLEN) v = -1;
    if (tid == HDR_NTILES) v = ntiles;
    if (tid == HDR_NKEYS) v = cnt;
    p.shdr[tid] = v;
  }
  for (int t = tid; t < p.ntile_cap; t += 256) {
    const int left = cnt - t * KT;
    TileEnt e;
    e.tile = t;
    e.pad = 0;
    e.mask = left >= KT ? ~0ull : (left > 0 ? (1ull << left) - 1ull : 0ull);
    p.tiles[t] = e;
  }
}

// grid ceil(n/4), block 256: one row per wave, 4 channels per lane.
//  ROWS_GATHER: z = X[sel[r]] (the gather; invalid entries are reported)
//  ROWS_REDUCE: z = z' + P[0] + P[1] + ... (the MLP's chunk partials, in order)
//  both       : Z[r] = z and A1[r] = LN(z) (the next QKV product's rows)
//  ROWS_FINAL : z as in REDUCE, scattered to Y[sel[r]] (bf16 or fp32)
enum { ROWS_GATHER = 0, ROWS_REDUCE = 1, ROWS_FINAL = 2 };
template <int MODE>
__global__ __launch_bounds__(256) void k_stk_rows(StkArgs p) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int cnt = stk_count(p);
  const int r = blockIdx.x * 4 + wave;
  if (r >= cnt) return;
  const int64_t off = (int64_t)r * SG_C + 4 * lane;
  f32x4 z;
  int cell = 0;
  if constexpr (MODE != ROWS_REDUCE) cell = stk_cell(p, r);
  if constexpr (MODE == ROWS_GATHER) {
    if (cell < 0 && lane == 0) set_err(p.err_hdr, RS3_E_INVALID);
    const u32x2 v = gload((const u32x2*)((const bf16_t*)p.X + (int64_t)max(cell, 0) * SG_C + 4 * lane));
    z = f32x4{__uint_as_float(v[0] << 16), __uint_as_float(v[0] & 0xffff0000u), __uint_as_float(v[1] << 16),
              __uint_as_float(v[1] & 0xffff0000u)};
  } else {
    constexpr int B = 8;   // partials loaded per batch
    z = gload((const f32x4*)(p.Zp + off));
    for (int c0 = 0; c0 < p.NC; c0 += B) {
      f32x4 pc[B];
#pragma unroll
      for (int c = 0; c < B; ++c)
        if (c0 + c < p.NC) pc[c] = gload((const f32x4*)(p.P + (int64_t)(c0 + c) * p.M * SG_C + off));
#pragma unroll
      for (int c = 0; c < B; ++c)
        if (c0 + c < p.NC) z += pc[c];
    }
  }
  if constexpr (MODE == ROWS_FINAL) {
    if (cell < 0) return;
    const int64_t yo = (int64_t)cell * SG_C + 4 * lane;
    if (p.y_f32)
      *(f32x4*)((float*)p.Y + yo) = z;
    else
      *(u32x2*)((bf16_t*)p.Y + yo) = u32x2{pack_bf16x2(z[0], z[1]), pack_bf16x2(z[2], z[3])};
  } else {
    const f32x4 g = gload((const f32x4*)(p.ln_g + 4 * lane));
    const f32x4 b = gload((const f32x4*)(p.ln_b + 4 * lane));
    *(f32x4*)(p.Z + off) = z;
    *(u32x2*)(p.A1 + off) = ln_row(z, g, b);
  }
}

// grid (ceil(n/64), 12), block 256: the 64x64 output tile (blockIdx.x,
// blockIdx.y) of A1 [n][256] x [W_qs | W_ks | W_vs]; each wave one 32x32
// MFMA tile.  Columns [0, 256) -> Qs (times qscale_s), [256, 512) -> the
// key tile blockIdx.x of the self-attention's bank ([H][64][d_h], rows past
// the count zero), [512, 768) -> its value tile ([H][d_h][64] in slot order).
// With write_bank, work-group (0, 0) also writes that bank's descriptor,
// header and tile list from the device count.
__global__ __launch_bounds__(256) void k_stk_qkv(StkArgs p) {
  __shared__ __attribute__((aligned(16))) bf16_t As[64 * SG_PITCH];
  const int row0 = blockIdx.x * 64, col0 = blockIdx.y * 64;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, g = lane >> 5;
  const int cnt = stk_count(p);
  if (p.write_bank && blockIdx.x == 0 && blockIdx.y == 0) write_self_bank(p, cnt);
  if (row0 >= cnt) return;
  const int wr = wave & 1, wc = wave >> 1;
  const int nb = (col0 >> 5) + wc;
  u32x4 bw[16];
#pragma unroll
  for (int ks = 0; ks < 16; ++ks) bw[ks] = ldb(p.Wqkv, 16, nb, ks, lane);
  u32x4 av[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int u = tid + 256 * j, r = u >> 5, c8 = u & 31;
    av[j] = gload((const u32x4*)(p.A1 + (int64_t)min(row0 + r, cnt - 1) * SG_C + 8 * c8));
  }
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int u = tid + 256 * j, r = u >> 5, c8 = u & 31;
    *(u32x4*)(As + r * SG_PITCH + 8 * c8) = row0 + r < cnt ? av[j] : u32x4{0, 0, 0, 0};
  }
  __syncthreads();
  f32x16 acc = {};
#pragma unroll
  for (int ks = 0; ks < 16; ++ks) acc = mfma32(lda(As, SG_PITCH, 32 * wr, ks, lane), bw[ks], acc);
  const int col = col0 + 32 * wc + (lane & 31);
  const int rbase = row0 + 32 * wr;
  const int region = col0 / SG_C, c = col - region * SG_C;
  const int h = c / p.dhs, d = c - h * p.dhs;
  if (region == 0) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int row = rbase + c_row(r, lane);
      if (row < cnt) p.Qs[(int64_t)row * SG_C + c] = f2bf(acc[r] * p.qscale_s);
    }
  } else if (region == 1) {
    bf16_t* kt = p.Kh + ((int64_t)blockIdx.x * p.Hs + h) * KT * p.dhs + d;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int j = 32 * wr + c_row(r, lane);
      kt[j * p.dhs] = row0 + j < cnt ? f2bf(acc[r]) : (bf16_t)0;
    }
  } else {
    // the eight results r = 0..7 (and 8..15) of a lane are keys whose V^
    // slots are 32*wr + 8*g + r (+16): one 16-byte store each
    bf16_t* vt = p.Vh + (((int64_t)blockIdx.x * p.Hs + h) * p.dhs + d) * KT + 32 * wr + 8 * g;
#pragma unroll
    for (int hf = 0; hf < 2; ++hf) {
      u32x4 pk;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int q0 = 8 * hf + 2 * e;
        const float v0 = rbase + c_row(q0, lane) < cnt ? acc[q0] : 0.f;
        const float v1 = rbase + c_row(q0 + 1, lane) < cnt ? acc[q0 + 1] : 0.f;
        pk[e] = pack_bf16x2(v0, v1);
      }
      *(u32x4*)(vt + 16 * hf) = pk;
    }
  }
}

// grid ceil(n/32), block 256, LDS PS_LDS: 32 whole rows per work-group.
//   z += O W_os  (O: the self-attention's merged output, in Qs)
//   Qc = qscale_c * LN2(z) (W_q W_k^T)
// Wave w holds output columns [64w, 64w+64) of the first product (two
// 32x32 tiles); waves 0 and 1 take the two 32-column blocks of the second.
constexpr size_t PS_O = 0, PS_Z = 32 * SG_PITCH * 2, PS_A = PS_Z + 32 * SG_C * 4;
constexpr size_t PS_LDS = PS_A + 32 * SG_PITCH * 2;
__global__ __launch_bounds__(256) void k_stk_post_sa(StkArgs p) {
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  bf16_t* Os = (bf16_t*)(lds + PS_O);
  float* Zs = (float*)(lds + PS_Z);
  bf16_t* As = (bf16_t*)(lds + PS_A);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int row0 = blockIdx.x * 32;
  const int cnt = stk_count(p);
  if (row0 >= cnt) return;
  u32x4 bo[2][16];
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int ks = 0; ks < 16; ++ks) bo[t][ks] = ldb(p.Wos, 16, 2 * wave + t, ks, lane);
  u32x4 ov[4];
  f32x4 zv[8];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int u = tid + 256 * j, r = u >> 5, c8 = u & 31;
    ov[j] = gload((const u32x4*)(p.Qs + (int64_t)min(row0 + r, cnt - 1) * SG_C + 8 * c8));
  }
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int u = tid + 256 * j, r = u >> 6, c4 = u & 63;
    zv[j] = gload((const f32x4*)(p.Z + (int64_t)min(row0 + r, cnt - 1) * SG_C + 4 * c4));
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int u = tid + 256 * j, r = u >> 5, c8 = u & 31;
    *(u32x4*)(Os + r * SG_PITCH + 8 * c8) = row0 + r < cnt ? ov[j] : u32x4{0, 0, 0, 0};
  }
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int u = tid + 256 * j, r = u >> 6, c4 = u & 63;
    *(f32x4*)(Zs + r * SG_C + 4 * c4) = zv[j];
  }
  __syncthreads();
  f32x16 acc[2] = {};
#pragma unroll
  for (int ks = 0; ks < 16; ++ks) {
    const u32x4 a = lda(Os, SG_PITCH, 0, ks, lane);
    acc[0] = mfma32(a, bo[0][ks], acc[0]);
    acc[1] = mfma32(a, bo[1][ks], acc[1]);
  }
  // the cross-attention's W_q W_k^T operands (waves 0 and 1), in flight over the norm
  u32x4 bq[16];
  if (wave < 2) {
#pragma unroll
    for (int ks = 0; ks < 16; ++ks) bq[ks] = ldb(p.Wqc, 16, wave, ks, lane);
  }
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) Zs[c_row(r, lane) * SG_C + 64 * wave + 32 * t + (lane & 31)] += acc[t][r];
  __syncthreads();
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int u = tid + 256 * j, r = u >> 6, c4 = u & 63;
    if (row0 + r < cnt) *(f32x4*)(p.Z + (int64_t)(row0 + r) * SG_C + 4 * c4) = *(const f32x4*)(Zs + r * SG_C + 4 * c4);
  }
  {
    const f32x4 g = gload((const f32x4*)(p.ln2_g + 4 * lane));
    const f32x4 b = gload((const f32x4*)(p.ln2_b + 4 * lane));
    f32x4 zz[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) zz[i] = *(const f32x4*)(Zs + (8 * wave + i) * SG_C + 4 * lane);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      u32x2 y = ln_row(zz[i], g, b);
      if (row0 + 8 * wave + i >= cnt) y = u32x2{0, 0};
      *(u32x2*)(As + (8 * wave + i) * SG_PITCH + 4 * lane) = y;
    }
  }
  __syncthreads();
  if (wave < 2) {
    f32x16 q = {};
#pragma unroll
    for (int ks = 0; ks < 16; ++ks) q = mfma32(lda(As, SG_PITCH, 0, ks, lane), bq[ks], q);
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int row = row0 + c_row(r, lane);
      if (row < cnt) p.Qc[(int64_t)row * 64 + 32 * wave + (lane & 31)] = f2bf(q[r] * p.qscale_c);
    }
  }
}

// grid (ceil(n/RM), F/HC), block 256, LDS MlLds<RM>::BYTES: rows [RM bx, +RM)
// and hidden units [HC by, +HC).
//   z' = z + O W_vo            (O: the cross-attention's merged output, in Qc;
//                               the chunk-0 work-group stores z' to Zp)
//   P[by] = relu(LN3(z') W_1[:, chunk]) W_2[chunk, :]    (fp32)
// Wave w holds output columns [64w, 64w+64) of the W_vo and W_2 products and
// HC/4 hidden units of the W_1 product, for every 32-row half.  The hidden
// units reuse the LDS of z'.  At 32 rows a work-group takes 54 KB of LDS, so
// two share a CU and one's memory waits run under the other's work.
constexpr int ML_OP = 64 + 8;   // LDS pitch of the 64-wide O rows
template <int RM>
struct MlLds {
  static constexpr size_t O = 0, A = RM * ML_OP * 2, Z = A + RM * SG_PITCH * 2, BYTES = Z + RM * SG_C * 4;
};
constexpr int STACK_MLP_RM = 32;   // rows per work-group of the launch
template <int HC, int RM>
__global__ __launch_bounds__(256) void k_stk_mlp(StkArgs p) {
  static_assert(HC == 256 || HC == 128, "hidden units per work-group");
  static_assert(RM == 64 || RM == 32, "rows per work-group");
  constexpr int TW = HC / 128;   // 32-column blocks of the hidden chunk per wave
  constexpr int NI = RM / 32;    // 32-row halves
  using LL = MlLds<RM>;
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  bf16_t* Ob = (bf16_t*)(lds + LL::O);
  bf16_t* As = (bf16_t*)(lds + LL::A);
  float* Zs = (float*)(lds + LL::Z);
  bf16_t* Hs = (bf16_t*)(lds + LL::Z);   // after LN3
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int row0 = blockIdx.x * RM, chunk = blockIdx.y;
  const int cnt = stk_count(p);
  if (row0 >= cnt) return;
  u32x4 bv[2][4];
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) bv[t][ks] = ldb(p.Wvo, 4, 2 * wave + t, ks, lane);
  u32x4 ov[NI];
#pragma unroll
  for (int j = 0; j < NI; ++j) {
    const int u = tid + 256 * j, r = u >> 3, c8 = u & 7;
    ov[j] = gload((const u32x4*)(p.Qc + (int64_t)min(row0 + r, cnt - 1) * 64 + 8 * c8));
  }
  f32x4 zv[RM / 4];
#pragma unroll
  for (int j = 0; j < RM / 4; ++j) {
    const int u = tid + 256 * j, r = u >> 6, c4 = u & 63;
    zv[j] = gload((const f32x4*)(p.Z + (int64_t)min(row0 + r, cnt - 1) * SG_C + 4 * c4));
  }
#pragma unroll
  for (int j = 0; j < NI; ++j) {
    const int u = tid + 256 * j, r = u >> 3, c8 = u & 7;
    *(u32x4*)(Ob + r * ML_OP + 8 * c8) = row0 + r < cnt ? ov[j] : u32x4{0, 0, 0, 0};
  }
#pragma unroll
  for (int j = 0; j < RM / 4; ++j) {
    const int u = tid + 256 * j, r = u >> 6, c4 = u & 63;
    *(f32x4*)(Zs + r * SG_C + 4 * c4) = zv[j];
  }
  __syncthreads();
  f32x16 acc[NI][2];
#pragma unroll
  for (int i = 0; i < NI; ++i)
#pragma unroll
    for (int t = 0; t < 2; ++t) acc[i][t] = f32x16{};
#pragma unroll
  for (int ks = 0; ks < 4; ++ks)
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const u32x4 a = lda(Ob, ML_OP, 32 * i, ks, lane);
#pragma unroll
      for (int t = 0; t < 2; ++t) acc[i][t] = mfma32(a, bv[t][ks], acc[i][t]);
    }
  // W_1 operands of this hidden chunk, in flight over the residual and the norm
  u32x4 bw[2][16];
#pragma unroll
  for (int t = 0; t < TW; ++t)
#pragma unroll
    for (int ks = 0; ks < 16; ++ks) bw[t][ks] = ldb(p.W1, 16, (HC / 32) * chunk + TW * wave + t, ks, lane);
#pragma unroll
  for (int i = 0; i < NI; ++i)
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        Zs[(32 * i + c_row(r, lane)) * SG_C + 64 * wave + 32 * t + (lane & 31)] += acc[i][t][r];
  __syncthreads();
  if (chunk == 0) {
#pragma unroll
    for (int j = 0; j < RM / 4; ++j) {
      const int u = tid + 256 * j, r = u >> 6, c4 = u & 63;
      if (row0 + r < cnt)
        *(f32x4*)(p.Zp + (int64_t)(row0 + r) * SG_C + 4 * c4) = *(const f32x4*)(Zs + r * SG_C + 4 * c4);
    }
  }
  {
    const f32x4 g = gload((const f32x4*)(p.ln3_g + 4 * lane));
    const f32x4 b = gload((const f32x4*)(p.ln3_b + 4 * lane));
    constexpr int RW = RM / 4;   // rows per wave
    f32x4 zz[RW];
#pragma unroll
    for (int i = 0; i < RW; ++i) zz[i] = *(const f32x4*)(Zs + (RW * wave + i) * SG_C + 4 * lane);
#pragma unroll
    for (int i = 0; i < RW; ++i) {
      u32x2 y = ln_row(zz[i], g, b);
      if (row0 + RW * wave + i >= cnt) y = u32x2{0, 0};
      *(u32x2*)(As + (RW * wave + i) * SG_PITCH + 4 * lane) = y;
    }
  }
  __syncthreads();   // LN3 rows complete; z' no longer read (its LDS takes the hidden units)
#pragma unroll
  for (int i = 0; i < NI; ++i)
#pragma unroll
    for (int t = 0; t < 2; ++t) acc[i][t] = f32x16{};
#pragma unroll
  for (int ks = 0; ks < 16; ++ks)
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const u32x4 a = lda(As, SG_PITCH, 32 * i, ks, lane);
#pragma unroll
      for (int t = 0; t < TW; ++t) acc[i][t] = mfma32(a, bw[t][ks], acc[i][t]);
    }
  // W_2 operands: rows [HC chunk, +HC) of W_2 are its steps [HC/16 chunk, +HC/16)
  constexpr int KS2 = HC / 16;
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int ks = 0; ks < KS2; ++ks) bw[t][ks] = ldb(p.W2, p.F / 16, 2 * wave + t, KS2 * chunk + ks, lane);
#pragma unroll
  for (int i = 0; i < NI; ++i)
#pragma unroll
    for (int t = 0; t < TW; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        Hs[(32 * i + c_row(r, lane)) * SG_PITCH + 32 * TW * wave + 32 * t + (lane & 31)] =
            f2bf(fmaxf(acc[i][t][r], 0.f));
  __syncthreads();
#pragma unroll
  for (int i = 0; i < NI; ++i)
#pragma unroll
    for (int t = 0; t < 2; ++t) acc[i][t] = f32x16{};
#pragma unroll
  for (int ks = 0; ks < KS2; ++ks)
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const u32x4 a = lda(Hs, SG_PITCH, 32 * i, ks, lane);
#pragma unroll
      for (int t = 0; t < 2; ++t) acc[i][t] = mfma32(a, bw[t][ks], acc[i][t]);
    }
  float* P = p.P + (int64_t)chunk * p.M * SG_C;
#pragma unroll
  for (int i = 0; i < NI; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int row = row0 + 32 * i + c_row(r, lane);
      if (row >= cnt) continue;
#pragma unroll
      for (int t = 0; t < 2; ++t) P[(int64_t)row * SG_C + 64 * wave + 32 * t + (lane & 31)] = acc[i][t][r];
    }
}

// Y <- X for every cell (bf16 -> bf16 or fp32), 8 channels per thread.
template <bool F32OUT>
__global__ __launch_bounds__(256) void k_stk_copy(const bf16_t* X, void* Y, int64_t chunks) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < chunks; i += (int64_t)gridDim.x * 256) {
    const u32x4 v = gload((const u32x4*)(X + 8 * i));
    if constexpr (F32OUT) {
      float* y = (float*)Y + 8 * i;
      *(f32x4*)y = f32x4{__uint_as_float(v[0] << 16), __uint_as_float(v[0] & 0xffff0000u),
                         __uint_as_float(v[1] << 16), __uint_as_float(v[1] & 0xffff0000u)};
      *(f32x4*)(y + 4) = f32x4{__uint_as_float(v[2] << 16), __uint_as_float(v[2] & 0xffff0000u),
                               __uint_as_float(v[3] << 16), __uint_as_float(v[3] & 0xffff0000u)};
    } else {
      *((u32x4*)Y + i) = v;
    }
  }
}

}  // namespace rs3

using namespace rs3;

hipError_t rs3_launch_stack_rows(const StkArgs& p, int mode, hipStream_t st) {
  if (p.M <= 0) return hipSuccess;
  const dim3 grid((unsigned)((p.M + 3) / 4));
  if (mode == ROWS_GATHER)
    RS3_LAUNCH(RS3_K_STACK_ROWS, st, k_stk_rows<ROWS_GATHER>, grid, dim3(256), 0, st, p);
  else if (mode == ROWS_REDUCE)
    RS3_LAUNCH(RS3_K_STACK_ROWS, st, k_stk_rows<ROWS_REDUCE>, grid, dim3(256), 0, st, p);
  else
    RS3_LAUNCH(RS3_K_STACK_ROWS, st, k_stk_rows<ROWS_FINAL>, grid, dim3(256), 0, st, p);
  return hipGetLastError();
}

hipError_t rs3_launch_stack_qkv(const StkArgs& p, hipStream_t st) {
  if (p.M <= 0) return hipSuccess;
  RS3_LAUNCH(RS3_K_STACK_GEMM, st, k_stk_qkv, dim3((unsigned)((p.M + 63) / 64), 3 * SG_C / 64), dim3(256), 0, st, p);
  return hipGetLastError();
}

hipError_t rs3_launch_stack_post_sa(const StkArgs& p, hipStream_t st) {
  if (p.M <= 0) return hipSuccess;
  RS3_LAUNCH(RS3_K_STACK_GEMM, st, k_stk_post_sa, dim3((unsigned)((p.M + 31) / 32)), dim3(256), PS_LDS, st, p);
  return hipGetLastError();
}

hipError_t rs3_launch_stack_mlp(const StkArgs& p, hipStream_t st) {
  if (p.M <= 0) return hipSuccess;
  if (p.F % 256 != 0 || (p.NC != p.F / 256 && p.NC != p.F / 128)) return hipErrorInvalidValue;
  constexpr int RM = STACK_MLP_RM;
  const dim3 grid((unsigned)((p.M + RM - 1) / RM), p.NC);
  if (p.NC == p.F / 128)
    RS3_LAUNCH(RS3_K_STACK_MLP, st, (k_stk_mlp<128, RM>), grid, dim3(256), MlLds<RM>::BYTES, st, p);
  else
    RS3_LAUNCH(RS3_K_STACK_MLP, st, (k_stk_mlp<256, RM>), grid, dim3(256), MlLds<RM>::BYTES, st, p);
  return hipGetLastError();
}

hipError_t rs3_launch_stack_merge(const StkArgs& p, hipStream_t st) {
  const int64_t items = (int64_t)p.M * (p.D_att / 8);
  if (items == 0) return hipSuccess;
  if (p.D_att % 8 != 0 || p.d_att % 8 != 0) return hipErrorInvalidValue;
  RS3_LAUNCH(RS3_K_STACK_MERGE, st, k_stk_merge, dim3((unsigned)((items + 255) / 256)), dim3(256), 0, st, p);
  return hipGetLastError();
}

hipError_t rs3_launch_stack_copy(const void* X, void* Y, int64_t elems, int y_f32, hipStream_t st) {
  const int64_t chunks = elems / 8;
  if (chunks == 0) return hipSuccess;
  const unsigned nb = (unsigned)((chunks + 255) / 256 < 2048 ? (chunks + 255) / 256 : 2048);
  if (y_f32)
    RS3_LAUNCH(RS3_K_COPY, st, k_stk_copy<true>, dim3(nb), dim3(256), 0, st, (const bf16_t*)X, Y, chunks);
  else
    RS3_LAUNCH(RS3_K_COPY, st, k_stk_copy<false>, dim3(nb), dim3(256), 0, st, (const bf16_t*)X, Y, chunks);
  return hipGetLastError();
}

hipError_t rs3_stack_setup() {
  constexpr int RM = STACK_MLP_RM;
  hipError_t e = hipFuncSetAttribute((const void*)k_stk_mlp<256, RM>, hipFuncAttributeMaxDynamicSharedMemorySize,
                                     (int)MlLds<RM>::BYTES);
  if (e == hipSuccess)
    e = hipFuncSetAttribute((const void*)k_stk_mlp<128, RM>, hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)MlLds<RM>::BYTES);
  if (e == hipSuccess)
    e = hipFuncSetAttribute((const void*)k_stk_post_sa, hipFuncAttributeMaxDynamicSharedMemorySize, (int)PS_LDS);
  return e;
}
