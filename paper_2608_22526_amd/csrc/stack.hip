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

template <int CTRL>
__device__ __forceinline__ float dppf(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}

// Sum over the 64 lanes, the same value in every lane: within rows of 16
// lanes by DPP (quad swaps, half-row and row mirrors), then across rows by
// v_permlane16_swap and v_permlane32_swap.  Each step adds a lane to a
// partner that adds it back, so every lane holds the same bits.
__device__ __forceinline__ float wave_sum(float v) {
  v += dppf<0xB1>(v);    // quad_perm(1, 0, 3, 2)
  v += dppf<0x4E>(v);    // quad_perm(2, 3, 0, 1)
  v += dppf<0x141>(v);   // row_half_mirror
  v += dppf<0x140>(v);   // row_mirror
  auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = __uint_as_float(r[0]) + __uint_as_float(r[1]);
  r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
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
// LayerNorm of the fp32 rows of Z (GATHER: of the kept cells of the bf16
// grid X, and the column-block-0 work-group stores them to Z): each wave
// normalises 16 rows, a lane holding 4 channels.  Rows past the count are
// computed on a clamped row and stored as zero, so the 16 reductions carry
// no branch and interleave.
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
  if constexpr (GATHER) {
    if (blockIdx.y == 0) {
#pragma unroll
      for (int i = 0; i < 16; ++i)
        if (row0 + 16 * wave + i < cnt) *(f32x4*)(p.Zw + (int64_t)(row0 + 16 * wave + i) * SG_C + 4 * lane) = z[i];
    }
  }
  float sm[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) sm[i] = wave_sum(z[i][0] + z[i][1] + z[i][2] + z[i][3]);
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    z[i] -= sm[i] * (1.f / SG_C);
    sm[i] = wave_sum(z[i][0] * z[i][0] + z[i][1] * z[i][1] + z[i][2] * z[i][2] + z[i][3] * z[i][3]);
  }
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int lr = 16 * wave + i;
    const float rs = 1.f / sqrtf(sm[i] * (1.f / SG_C) + SG_LN_EPS);
    const f32x4 y = z[i] * rs * g + b;
    u32x2 o = {pack_bf16x2(y[0], y[1]), pack_bf16x2(y[2], y[3])};
    if (row0 + lr >= cnt) o = u32x2{0, 0};
    *(u32x2*)(As + lr * SG_PITCH + 4 * lane) = o;
  }
}

// grid ceil(M*K/8 / 256), block 256: one thread per (kept row, 8 columns)
// merges the attention's key splits (partials O/l and (m, l) per split, row
// and head: Opart [S][M][K], ML [S][M][H_att][2]) by log-sum-exp into the
// normalised bf16 rows out [M][K].  The splits are loaded eight at a time
// without branches (split indices past S re-read the last split and are
// masked); a split without keys holds l = 0 and adds nothing, its O words
// (never written) replaced by zero; a row with no key at all gets O = 0.
__global__ __launch_bounds__(256) void k_stk_merge(StkGemmArgs p) {
  const int D = p.K, cpr = D / 8;
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
  *(u32x4*)((bf16_t*)p.out + (int64_t)row * D + d0) = out;
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
  if constexpr (AM == STK_A_BF16) {
    // register double buffer: chunk kc+1's A rows and B operands are in
    // flight while chunk kc is multiplied
    constexpr int AU = SG_BM * SG_KC / 8 / 256;   // 16-byte A units per thread and chunk
    u32x4 av[AU], bw[SG_KC / 16];
    auto load = [&](int kc) {
      const int kn = min(SG_KC, p.K - kc), cpr = kn / 8;
#pragma unroll
      for (int j = 0; j < AU; ++j) {
        const int u = threadIdx.x + 256 * j, r = u / cpr, c8 = u - r * cpr;
        const int rr = min(row0 + r, cnt - 1);
        if (u < SG_BM * cpr) av[j] = gload((const u32x4*)((const bf16_t*)p.A + (int64_t)rr * p.K + kc + 8 * c8));
      }
#pragma unroll
      for (int ks = 0; ks < SG_KC / 16; ++ks)
        if (16 * ks < kn) bw[ks] = gload((const u32x4*)(wrow + kc + 16 * ks + 8 * g));
    };
    load(0);
    for (int kc = 0; kc < p.K; kc += SG_KC) {
      const int kn = min(SG_KC, p.K - kc), cpr = kn / 8;
      if (kc > 0) __syncthreads();   // the previous chunk's operands are read
#pragma unroll
      for (int j = 0; j < AU; ++j) {
        const int u = threadIdx.x + 256 * j, r = u / cpr, c8 = u - r * cpr;
        if (u < SG_BM * cpr) *(u32x4*)(As + r * SG_PITCH + 8 * c8) = row0 + r < cnt ? av[j] : u32x4{0, 0, 0, 0};
      }
      u32x4 bc[SG_KC / 16];
#pragma unroll
      for (int ks = 0; ks < SG_KC / 16; ++ks) bc[ks] = bw[ks];
      __syncthreads();
      if (kc + SG_KC < p.K) load(kc + SG_KC);
      const bf16_t* arow = As + (32 * wr + (lane & 31)) * SG_PITCH + 8 * g;
#pragma unroll
      for (int ks = 0; ks < SG_KC / 16; ++ks)
        if (16 * ks < kn) acc = mfma32(*(const u32x4*)(arow + 16 * ks), bc[ks], acc);
    }
  } else {
    // LayerNorm prologues: K = d_model = one chunk
    u32x4 bw[SG_KC / 16];
#pragma unroll
    for (int ks = 0; ks < SG_KC / 16; ++ks) bw[ks] = gload((const u32x4*)(wrow + 16 * ks + 8 * g));
    if constexpr (AM == STK_A_LN) pro_ln<false>(p, row0, cnt, As);
    if constexpr (AM == STK_A_GLN) pro_ln<true>(p, row0, cnt, As);
    __syncthreads();
    const bf16_t* arow = As + (32 * wr + (lane & 31)) * SG_PITCH + 8 * g;
#pragma unroll
    for (int ks = 0; ks < SG_KC / 16; ++ks) acc = mfma32(*(const u32x4*)(arow + 16 * ks), bw[ks], acc);
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
  if (am == STK_A_BF16 && p.K % 64 != 0) return hipErrorInvalidValue;
#define RS3_SG(A, E) \
  if (am == A && em == E) return launch_gemm<A, E>(p, st);
  RS3_SG(STK_A_GLN, STK_E_QKV)
  RS3_SG(STK_A_LN, STK_E_QKV)
  RS3_SG(STK_A_LN, STK_E_STORE)
  RS3_SG(STK_A_BF16, STK_E_RESID)
  RS3_SG(STK_A_BF16, STK_E_SCATTER)
#undef RS3_SG
  return hipErrorInvalidValue;
}

hipError_t rs3_launch_stack_merge(const StkGemmArgs& p, hipStream_t st) {
  const int64_t items = (int64_t)p.M * (p.K / 8);
  if (items == 0) return hipSuccess;
  if (p.K % 8 != 0 || p.d_att % 8 != 0) return hipErrorInvalidValue;
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
