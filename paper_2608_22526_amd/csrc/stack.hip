// The L-layer memory-attention stack on the kept queries (Sec. 3.1, "Sparse
// memory attention": the stack is patched at every layer's entry).  The rows
// are gathered once before the first layer and scattered once after the
// last; in between, every layer is
//     z += SA(LN1(z))  among the kept rows      (one-frame bank of the kept rows)
//     z += CA(LN2(z))  against the memory bank  (the readout of Eq. 6, absorbed)
//     z += W2 relu(W1 LN3(z))
// with the residual stream z in fp32 and every matrix product on bf16 MFMA.
//
// The attentions run on the readout's split-KV attention kernel unchanged.
// The self-attention's keys and values are laid out by the QKV product's
// epilogue as a bank of one frame whose tiles are the 64-row blocks of the
// kept set; the cross-attention reads the real ring bank, whose rows a layer
// of one absorbed head uses as they are (W_q W_k^T on the query side,
// W_v W_o on the output side), so one bank serves every layer.
//
// Every product is one launch of k_stk_gemm: a 64x64 output tile per
// work-group of four waves (one 32x32 MFMA tile each), the A operand staged
// in LDS by one of the prologues, B read from the transposed weights W^T
// [N][K] (16-byte runs along K).
#include "device_util.h"

namespace rs3 {

constexpr int SG_BM = 64;    // rows per work-group (= keys per bank tile)
constexpr int SG_BN = 64;    // columns per work-group
constexpr int SG_KC = 256;   // contraction chunk staged in LDS
constexpr int SG_PITCH = SG_KC + 8;   // bf16 elements per LDS row
constexpr size_t SG_LDS = (size_t)SG_BM * SG_PITCH * 2;
constexpr int SG_C = 256;    // d_model of the stack
constexpr float SG_LN_EPS = 1e-5f;

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// Kept-row count of the call, clamped into [0, M]; a count outside that
// range is reported in the bank's error word by work-group (0, 0).
__device__ __forceinline__ int stk_count(const StkGemmArgs& p) {
  int cnt = gload(p.count);
  if (cnt < 0 || cnt > p.M) {
    if (blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x == 0) set_err(p.err_hdr, RS3_E_INVALID);
    cnt = cnt < 0 ? 0 : p.M;
  }
  return cnt;
}

// Cell of kept row r, or -1 for an entry out of range or not above its
// predecessor (such rows are reported and never written to Y).
__device__ __forceinline__ int stk_cell(const StkGemmArgs& p, int r) {
  const int i = gload(p.sel + r);
  const int prev = r > 0 ? gload(p.sel + r - 1) : -1;
  return (i >= 0 && i < p.mn && prev < i) ? i : -1;
}

// ---- prologues: the A chunk [64][kn] of rows row0.. in LDS (bf16) ----------
// plain bf16 rows of A [M][K]
__device__ __forceinline__ void pro_bf16(const StkGemmArgs& p, int row0, int cnt, int kc, int kn, bf16_t* As) {
  const int cpr = kn / 8;
  for (int u = threadIdx.x; u < SG_BM * cpr; u += 256) {
    const int r = u / cpr, c8 = u - r * cpr;
    u32x4 v = {0, 0, 0, 0};
    if (row0 + r < cnt) v = gload((const u32x4*)((const bf16_t*)p.A + (int64_t)(row0 + r) * p.K + kc + 8 * c8));
    *(u32x4*)(As + r * SG_PITCH + 8 * c8) = v;
  }
}

// LayerNorm of the fp32 rows of Z (GATHER: of the kept cells of the bf16
// grid X, and the column-block-0 work-group stores them to Z): each wave
// normalises 16 rows, a lane holding 4 channels.
template <bool GATHER>
__device__ __forceinline__ void pro_ln(const StkGemmArgs& p, int row0, int cnt, bf16_t* As) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  f32x4 z[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int r = min(row0 + 16 * wave + i, cnt - 1);
    if constexpr (GATHER) {
      const int cell = stk_cell(p, r);
      if (cell < 0 && blockIdx.y == 0 && lane == 0) set_err(p.err_hdr, RS3_E_INVALID);
      const u32x2 v = gload((const u32x2*)((const bf16_t*)p.X + (int64_t)max(cell, 0) * SG_C + 4 * lane));
      z[i] = f32x4{__uint_as_float(v[0] << 16), __uint_as_float(v[0] & 0xffff0000u), __uint_as_float(v[1] << 16),
                   __uint_as_float(v[1] & 0xffff0000u)};
    } else {
      z[i] = gload((const f32x4*)(p.Z + (int64_t)r * SG_C + 4 * lane));
    }
  }
  const f32x4 g = gload((const f32x4*)(p.ln_g + 4 * lane));
  const f32x4 b = gload((const f32x4*)(p.ln_b + 4 * lane));
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int lr = 16 * wave + i;
    u32x2 o = {0, 0};
    if (row0 + lr < cnt) {
      if constexpr (GATHER) {
        if (blockIdx.y == 0) *(f32x4*)(p.Zw + (int64_t)(row0 + lr) * SG_C + 4 * lane) = z[i];
      }
      const float mean = wave_sum(z[i][0] + z[i][1] + z[i][2] + z[i][3]) * (1.f / SG_C);
      const f32x4 d = z[i] - mean;
      const float var = wave_sum(d[0] * d[0] + d[1] * d[1] + d[2] * d[2] + d[3] * d[3]) * (1.f / SG_C);
      const float rs = 1.f / sqrtf(var + SG_LN_EPS);
      const f32x4 y = d * rs * g + b;
      o = u32x2{pack_bf16x2(y[0], y[1]), pack_bf16x2(y[2], y[3])};
    }
    *(u32x2*)(As + lr * SG_PITCH + 4 * lane) = o;
  }
}

// Log-sum-exp merge of the attention's key splits (partials O/l, (m, l) per
// split, row and head) into the normalised rows O [64][K] (K = the attention
// width).  A split without keys holds l = 0 and adds nothing; a row with no
// key at all (empty bank) gets O = 0.
__device__ __forceinline__ void pro_merge(const StkGemmArgs& p, int row0, int cnt, bf16_t* As) {
  const int D = p.K, cpr = D / 8;
  for (int it = threadIdx.x; it < SG_BM * cpr; it += 256) {
    const int r = it / cpr, d0 = 8 * (it - r * cpr), h = d0 / p.d_att;
    u32x4 out = {0, 0, 0, 0};
    const int row = row0 + r;
    if (row < cnt) {
      float M = -INFINITY, W = 0.f;
      float acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
      for (int s = 0; s < p.S; ++s) {
        const int64_t prow = (int64_t)s * p.M + row;
        const float m = gload(p.ML + (prow * p.H_att + h) * 2), l = gload(p.ML + (prow * p.H_att + h) * 2 + 1);
        if (!(l > 0.f)) continue;
        const u32x4 v = gload((const u32x4*)(p.Opart + prow * D + d0));
        if (m > M) {
          const float sc = __builtin_amdgcn_exp2f(M - m);
          W *= sc;
#pragma unroll
          for (int e = 0; e < 8; ++e) acc[e] *= sc;
          M = m;
        }
        const float w = __builtin_amdgcn_exp2f(m - M) * l;
        W += w;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          acc[2 * e] += w * __uint_as_float(v[e] << 16);
          acc[2 * e + 1] += w * __uint_as_float(v[e] & 0xffff0000u);
        }
      }
      const float inv = W > 0.f ? 1.f / W : 0.f;
#pragma unroll
      for (int e = 0; e < 4; ++e) out[e] = pack_bf16x2(acc[2 * e] * inv, acc[2 * e + 1] * inv);
    }
    *(u32x4*)(As + r * SG_PITCH + d0) = out;
  }
}

// The self-attention's one-frame bank: descriptor, header (tile and key
// counts from the device count) and tile list, by work-group (0, 0) of the
// first layer's QKV product.
__device__ __forceinline__ void write_self_bank(const StkGemmArgs& p, int cnt) {
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

// grid (ceil(M/64), N/64), block 256, LDS SG_LDS.
template <int AM, int EM>
__global__ __launch_bounds__(256) void k_stk_gemm(StkGemmArgs p) {
  extern __shared__ __attribute__((aligned(16))) uint8_t lds_raw[];
  bf16_t* As = (bf16_t*)lds_raw;
  const int row0 = blockIdx.x * SG_BM, col0 = blockIdx.y * SG_BN;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, g = lane >> 5;
  const int cnt = stk_count(p);
  if constexpr (EM == STK_E_QKV) {
    if (p.write_bank && blockIdx.x == 0 && blockIdx.y == 0) write_self_bank(p, cnt);
  }
  if (row0 >= cnt) return;
  const int wr = wave & 1, wc = wave >> 1;
  const int col = col0 + 32 * wc + (lane & 31);
  const bf16_t* wrow = p.WT + (int64_t)col * p.K;
  f32x16 acc = {};
  for (int kc = 0; kc < p.K; kc += SG_KC) {
    const int kn = min(SG_KC, p.K - kc);
    u32x4 bw[SG_KC / 16];
#pragma unroll
    for (int ks = 0; ks < SG_KC / 16; ++ks)
      if (16 * ks < kn) bw[ks] = gload((const u32x4*)(wrow + kc + 16 * ks + 8 * g));
    if (kc > 0) __syncthreads();   // the previous chunk's operands are read
    if constexpr (AM == STK_A_BF16) pro_bf16(p, row0, cnt, kc, kn, As);
    if constexpr (AM == STK_A_LN) pro_ln<false>(p, row0, cnt, As);
    if constexpr (AM == STK_A_GLN) pro_ln<true>(p, row0, cnt, As);
    if constexpr (AM == STK_A_MERGE) pro_merge(p, row0, cnt, As);
    __syncthreads();
    const bf16_t* arow = As + (32 * wr + (lane & 31)) * SG_PITCH + 8 * g;
#pragma unroll
    for (int ks = 0; ks < SG_KC / 16; ++ks)
      if (16 * ks < kn) acc = mfma32(*(const u32x4*)(arow + 16 * ks), bw[ks], acc);
  }
  const int rbase = row0 + 32 * wr;
  if constexpr (EM == STK_E_STORE) {
    bf16_t* out = (bf16_t*)p.out;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int row = rbase + c_row(r, lane);
      if (row >= cnt) continue;
      float v = acc[r] * p.scale;
      if (p.relu) v = fmaxf(v, 0.f);
      out[(int64_t)row * p.N + col] = f2bf(v);
    }
  } else if constexpr (EM == STK_E_RESID) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int row = rbase + c_row(r, lane);
      if (row >= cnt) continue;
      float* zp = p.Zw + (int64_t)row * SG_C + col;
      *zp = *zp + acc[r];
    }
  } else if constexpr (EM == STK_E_SCATTER) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int row = rbase + c_row(r, lane);
      if (row >= cnt) continue;
      const int cell = stk_cell(p, row);
      if (cell < 0) continue;
      const float y = p.Z[(int64_t)row * SG_C + col] + acc[r];
      if (p.y_f32)
        ((float*)p.Y)[(int64_t)cell * SG_C + col] = y;
      else
        ((bf16_t*)p.Y)[(int64_t)cell * SG_C + col] = f2bf(y);
    }
  } else {   // STK_E_QKV: columns [0, C) queries, [C, 2C) keys, [2C, 3C) values
    const int region = col0 / SG_C, c = col - region * SG_C;
    const int h = c / p.dhs, d = c - h * p.dhs;
    if (region == 0) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = rbase + c_row(r, lane);
        if (row < cnt) p.Qs[(int64_t)row * SG_C + c] = f2bf(acc[r] * p.scale);
      }
    } else if (region == 1) {
      // K^ tile rb: [H][64][d_h], rows past the count zero
      bf16_t* kt = p.Kh + ((int64_t)blockIdx.x * p.Hs + h) * KT * p.dhs + d;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int j = 32 * wr + c_row(r, lane);
        kt[j * p.dhs] = row0 + j < cnt ? f2bf(acc[r]) : (bf16_t)0;
      }
    } else {
      // V^ tile rb: [H][d_h][64] in slot order; the eight results r = 0..7
      // (and 8..15) of a lane are keys whose slots are 32*wr + 8*g + r (+16)
      bf16_t* vt = p.Vh + (((int64_t)blockIdx.x * p.Hs + h) * p.dhs + d) * KT + 32 * wr + 8 * g;
#pragma unroll
      for (int hf = 0; hf < 2; ++hf) {
        u32x4 pk;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int r0 = 8 * hf + 2 * e;
          const float v0 = rbase + c_row(r0, lane) < cnt ? acc[r0] : 0.f;
          const float v1 = rbase + c_row(r0 + 1, lane) < cnt ? acc[r0 + 1] : 0.f;
          pk[e] = pack_bf16x2(v0, v1);
        }
        *(u32x4*)(vt + 16 * hf) = pk;
      }
    }
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

template <int AM, int EM>
static hipError_t launch_gemm(const StkGemmArgs& p, hipStream_t st) {
  const dim3 grid((unsigned)((p.M + SG_BM - 1) / SG_BM), (unsigned)(p.N / SG_BN));
  RS3_LAUNCH(RS3_K_STACK_GEMM, st, (k_stk_gemm<AM, EM>), grid, dim3(256), SG_LDS, st, p);
  return hipGetLastError();
}

hipError_t rs3_launch_stack_gemm(const StkGemmArgs& p, int am, int em, hipStream_t st) {
  if (p.M <= 0) return hipSuccess;
  if (p.N % SG_BN != 0 || p.K % 16 != 0) return hipErrorInvalidValue;
  if ((am == STK_A_LN || am == STK_A_GLN) && p.K != SG_C) return hipErrorInvalidValue;
  if (am == STK_A_MERGE && p.K > SG_KC) return hipErrorInvalidValue;
#define RS3_SG(A, E) \
  if (am == A && em == E) return launch_gemm<A, E>(p, st);
  RS3_SG(STK_A_GLN, STK_E_QKV)
  RS3_SG(STK_A_LN, STK_E_QKV)
  RS3_SG(STK_A_MERGE, STK_E_RESID)
  RS3_SG(STK_A_LN, STK_E_STORE)
  RS3_SG(STK_A_BF16, STK_E_RESID)
  RS3_SG(STK_A_BF16, STK_E_SCATTER)
#undef RS3_SG
  return hipErrorInvalidValue;
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
