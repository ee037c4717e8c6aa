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
#include <algorithm>

#include "combine.h"

namespace rs3 {

// ---------------------------------------------------------------------------
// grid (n_obj, ceil(max_sel/64), D/64), block 256: 64 rows x 64 columns.
__global__ __launch_bounds__(256) void k_qproj(Rs3ReadoutArgs a) {
  const int o = blockIdx.x, r0 = blockIdx.y * 64, c0 = blockIdx.z * 64;
  BankDev& b = *a.banks[o];
  const int cnt = sel_count_of(a, o, b, false);   // reported by the merge kernel
  if (r0 >= cnt) return;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, g = lane >> 5;
  const int32_t* sel = a.sel_idx + (int64_t)o * a.sel_stride;
  const int C = a.C, D = a.D;
  const bf16_t* X = (const bf16_t*)a.X + (int64_t)o * a.x_stride;
  const int row = r0 + 32 * (wave & 1) + (lane & 31);
  const bool rv = row < cnt;
  int src = rv ? sel[row] : 0;
  if (src < 0 || src >= a.mn) src = 0;
  const bf16_t* xr = X + (int64_t)src * C;
  const int col = c0 + 32 * (wave >> 1) + (lane & 31);
  const bf16_t* wr = (const bf16_t*)a.WqT + (int64_t)col * C;
  f32x16 acc = {};
  // 16 k steps per batch, all loads of a batch issued before its MFMAs
  constexpr int KB = 16;
  for (int k0 = 0; k0 < C; k0 += 16 * KB) {
    u32x4 av[KB], bv[KB];
#pragma unroll
    for (int j = 0; j < KB; ++j)
      if (k0 + 16 * j < C) {
        av[j] = *(const u32x4*)(xr + k0 + 16 * j + 8 * g);
        bv[j] = *(const u32x4*)(wr + k0 + 16 * j + 8 * g);
      }
#pragma unroll
    for (int j = 0; j < KB; ++j)
      if (k0 + 16 * j < C) acc = mfma32(av[j], bv[j], acc);
  }
  if (a.rope) {
    // Eq. 7: the row gathered from cell sel[row] turns by that cell's
    // factors.  Lanes l and l^1 hold columns 2p and 2p+1 of the same rows;
    // lane j < 32 holds the cell of row j of this wave's 32.
    const float2* rope = (const float2*)a.rope;
    const int hp = a.d_h >> 1, p = (col & (a.d_h - 1)) >> 1;
    const float sgn = (col & 1) ? 1.f : -1.f;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int cell = __shfl(src, c_row(r, lane));
      const float2 cs = rope[(int64_t)cell * hp + p];
      const float v = acc[r], w = __shfl_xor(v, 1);
      acc[r] = v * cs.x + sgn * w * cs.y;
    }
  }
  bf16_t* Q = (bf16_t*)a.Q + (int64_t)o * a.max_sel * D;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    int rr = r0 + 32 * (wave & 1) + c_row(r, lane);
    if (rr < cnt) Q[(int64_t)rr * D + col] = f2bf(acc[r] * a.qscale);
  }
}

// ---------------------------------------------------------------------------
// The attention streams the object's resident keys in 32-key half tiles
// through nst LDS stages (nst-1 half tiles in flight; nst = 4 or 8, chosen
// at launch with the dynamic LDS size).  One stage holds
//   K : 32 rows (keys) x DH bf16, row pitch DH*2 + 16 bytes
//   V : DH rows x 32 keys (slot order), row pitch 64 + 16 bytes
// The pitch is an odd number of 16-byte chunks, so the 16 rows read by one
// LDS cycle (64 banks x 4 bytes) fall on 16 distinct bank groups, and every
// operand offset is a compile-time immediate.  Direct-to-LDS loads write
// 64 x 16 contiguous bytes per wave instruction; lanes that land on a pad
// chunk (or past the rows) load a harmless duplicate chunk.  Every wave
// issues the same number of loads per stage, so the waits are immediates.
template <int DH>
struct AttnLds {
  static constexpr int CPR = DH / 8;                          // data chunks per K row
  static constexpr int KP = (CPR + 1) * 16;                   // K row pitch, bytes
  static constexpr int VP = 5 * 16;                           // V row pitch, bytes
  static constexpr int NK = ((32 * (CPR + 1) + 63) / 64 + 3) / 4 * 4;   // K loads (wave instructions)
  static constexpr int NV = ((DH * 5 + 63) / 64 + 3) / 4 * 4;           // V loads
  static constexpr int KREG = NK * 1024;
  static constexpr int STAGE = KREG + NV * 1024;
  static constexpr int PER_WAVE = (NK + NV) / 4;              // loads per wave per stage
};

// Per-lane source offsets (elements) of the direct-to-LDS loads of one half
// tile; identical for every tile, so they are computed once per kernel.
template <int DH>
struct AttnDmaOffsets {
  int k[AttnLds<DH>::NK / 4];
  int v[AttnLds<DH>::NV / 4];
};

template <int DH>
__device__ __forceinline__ AttnDmaOffsets<DH> attn_dma_offsets(int wave, int lane) {
  using L = AttnLds<DH>;
  AttnDmaOffsets<DH> d;
#pragma unroll
  for (int j = 0; j < L::NK / 4; ++j) {
    const int p = (4 * j + wave) * 64 + lane;
    const int r = p / (L::CPR + 1), c = p % (L::CPR + 1);
    d.k[j] = (r < 32 && c < L::CPR) ? (r * L::CPR + c) * 8 : 0;
  }
#pragma unroll
  for (int j = 0; j < L::NV / 4; ++j) {
    const int p = (4 * j + wave) * 64 + lane;
    const int r = p / 5, c = p % 5;
    d.v[j] = (r < DH && c < 4) ? r * KT + c * 8 : 0;
  }
  return d;
}

// One direct-to-LDS load: 16 bytes per lane from g into the wave's 1 KB at
// lds_wave (lane l lands at lds_wave + 16 l).
__device__ __forceinline__ void dma16(const void* g, void* lds_wave) {
  __builtin_amdgcn_global_load_lds(g, lds_wave, 16, 0, 0);
}

// Direct-to-LDS loads of half tile `half` of bank tile `tile`, head h, into
// a stage.  `tile`, `half` and `wave` are wave-uniform (scalar registers).
template <int DH>
__device__ __forceinline__ void attn_issue(const bf16_t* Kh, const bf16_t* Vh, int tile, int half, int h, int H,
                                           uint8_t* stage, int wave, const AttnDmaOffsets<DH>& off) {
  using L = AttnLds<DH>;
  const bf16_t* kg = Kh + ((int64_t)tile * H + h) * (KT * DH) + half * 32 * DH;
  const bf16_t* vg = Vh + ((int64_t)tile * H + h) * (DH * KT) + half * 32;
#pragma unroll
  for (int j = 0; j < L::NK / 4; ++j) dma16(kg + off.k[j], stage + (4 * j + wave) * 1024);
#pragma unroll
  for (int j = 0; j < L::NV / 4; ++j) dma16(vg + off.v[j], stage + L::KREG + (4 * j + wave) * 1024);
}

// Value of lane l^32 for every lane (v_permlane32_swap: both halves come back
// in registers; op(r[0], r[1]) combines a lane with its partner).
__device__ __forceinline__ float max_with_partner(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __builtin_elementwise_maximum(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float sum_with_partner(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Workgroup barrier without a memory fence: the fence of __syncthreads()
// would wait for every outstanding load, including the K/V prefetches.
// LDS stages are published by the explicit vmcnt waits before it.
__device__ __forceinline__ void stage_barrier() { asm volatile("s_barrier" ::: "memory"); }

// s_waitcnt encoding: wait until at most n vector-memory ops are outstanding.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// Waits until at most `later` stages of PW loads each are still in flight
// (`later` is wave-uniform and at most MAXL).
template <int PW, int MAXL>
__device__ __forceinline__ void wait_stages(int later) {
  if constexpr (MAXL >= 6) if (later >= 6) { wait_vmcnt<6 * PW>(); return; }
  if constexpr (MAXL >= 5) if (later == 5) { wait_vmcnt<5 * PW>(); return; }
  if constexpr (MAXL >= 4) if (later == 4) { wait_vmcnt<4 * PW>(); return; }
  if constexpr (MAXL >= 3) if (later == 3) { wait_vmcnt<3 * PW>(); return; }
  if constexpr (MAXL >= 2) if (later == 2) { wait_vmcnt<2 * PW>(); return; }
  if (later == 1) {
    wait_vmcnt<PW>();
    return;
  }
  wait_vmcnt<0>();
}

// Query projection inside the attention (heads of width DH <= 64, d_model
// C = 8*PC with PC = 32): Q~^T block dt (32 d x 32 queries) = rows
// h*DH + 32*dt .. of W_q^T (A operand) times the wave's 32 gathered rows of
// X (B operand), fp32 accumulation over C in 16-deep steps, as the separate
// projection kernel does.  Both operands are staged in LDS with coalesced
// 16-byte loads (the W_q rows of a head are one contiguous block; each X row
// is 32 consecutive chunks), in the stage buffers, which are free until the
// first key/value DMA.  Row pitch PC*16 + 16 bytes: conflict-free reads of
// 32 rows x 16 bytes.
constexpr int PJ_PC = 32;                          // 16-byte chunks per row (C = 256)
constexpr int PJ_PITCH = PJ_PC * 16 + 16;          // bytes
constexpr int PJ_XCH = 128 * PJ_PC / 256;          // X chunks per thread (16)
template <int DH>
struct AttnProj {
  static constexpr int WCH = DH * PJ_PC / 256;     // W chunks per thread
  static constexpr int XS = 0;                     // X rows [128][PITCH]
  static constexpr int WS = 128 * PJ_PITCH;        // W rows [DH][PITCH]
  static constexpr int BYTES = WS + DH * PJ_PITCH;
};

// Loads of the projection's operands: W chunks need only the arguments,
// X chunks the gathered row indices (rows past the selected count read any
// valid row; their results are discarded).
// NT threads share the loads (256 or 512): thread t loads W chunks
// t + NT*j and X chunk t%32 of rows t/32 + (NT/32)*i.
template <int DH, int NT>
__device__ __forceinline__ void attn_proj_load_w(const bf16_t* WqT, int h, int tid,
                                                 u32x4 (&wv)[AttnProj<DH>::WCH * 256 / NT]) {
  const u32x4* wb = (const u32x4*)(WqT + (int64_t)h * DH * PJ_PC * 8);
#pragma unroll
  for (int j = 0; j < AttnProj<DH>::WCH * 256 / NT; ++j) wv[j] = gload(wb + tid + NT * j);
}

template <int NT>
__device__ __forceinline__ void attn_proj_rows(const int32_t* sel, int row0, int max_sel, int tid,
                                               int (&src)[PJ_XCH * 256 / NT]) {
#pragma unroll
  for (int i = 0; i < PJ_XCH * 256 / NT; ++i)
    src[i] = gload(sel + min(row0 + (tid >> 5) + (NT / 32) * i, max_sel - 1));
}

template <int NT>
__device__ __forceinline__ void attn_proj_load_x(const bf16_t* X, int mn, int tid, const int (&src)[PJ_XCH * 256 / NT],
                                                 u32x4 (&xv)[PJ_XCH * 256 / NT]) {
#pragma unroll
  for (int i = 0; i < PJ_XCH * 256 / NT; ++i) {
    const int r = (src[i] < 0 || src[i] >= mn) ? 0 : src[i];
    xv[i] = gload((const u32x4*)(X + (int64_t)r * PJ_PC * 8) + (tid & 31));
  }
}

template <int DH, int NT>
__device__ __forceinline__ void attn_project(uint8_t* lds, int tid, int wave, int lane, float qs,
                                             const u32x4 (&wv)[AttnProj<DH>::WCH * 256 / NT],
                                             const u32x4 (&xv)[PJ_XCH * 256 / NT], u32x4* qreg) {
  using P = AttnProj<DH>;
  const int g = lane >> 5;
#pragma unroll
  for (int j = 0; j < P::WCH * 256 / NT; ++j) {
    const int q = tid + NT * j;
    *(u32x4*)(lds + P::WS + (q / PJ_PC) * PJ_PITCH + (q % PJ_PC) * 16) = wv[j];
  }
#pragma unroll
  for (int i = 0; i < PJ_XCH * 256 / NT; ++i)
    *(u32x4*)(lds + P::XS + ((tid >> 5) + (NT / 32) * i) * PJ_PITCH + (tid & 31) * 16) = xv[i];
  lds_barrier();
  f32x16 qa[DH / 32];
#pragma unroll
  for (int dt = 0; dt < DH / 32; ++dt) qa[dt] = f32x16{};
  const uint8_t* xb = lds + P::XS + (32 * wave + (lane & 31)) * PJ_PITCH + 16 * g;
  const uint8_t* wb = lds + P::WS + (lane & 31) * PJ_PITCH + 16 * g;
#pragma unroll
  for (int k0 = 0; k0 < PJ_PC / 2; k0 += 4) {
    u32x4 bx[4], aw[4][DH / 32];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      bx[j] = *(const u32x4*)(xb + (k0 + j) * 32);
#pragma unroll
      for (int dt = 0; dt < DH / 32; ++dt) aw[j][dt] = *(const u32x4*)(wb + dt * 32 * PJ_PITCH + (k0 + j) * 32);
    }
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int dt = 0; dt < DH / 32; ++dt) qa[dt] = mfma32(aw[j][dt], bx[j], qa[dt]);
  }
  // Lane l holds query l%32 at d = 8*(r/4) + 4*(l/32) + r%4 of each block;
  // the B operand of the logits needs d = 16*ks + 8*(l/32) + 0..7.  One
  // v_permlane32_swap per register pair moves the quads into place: the low
  // half keeps its quad of r%8 < 4 and takes the high half's, the high half
  // takes the low half's quad of r%8 >= 4 and keeps its own.
#pragma unroll
  for (int dt = 0; dt < DH / 32; ++dt)
#pragma unroll
    for (int hf = 0; hf < 2; ++hf) {
      const f32x16& v = qa[dt];
      const int r = 8 * hf;
      const uint32_t p0 = pack_bf16x2(v[r] * qs, v[r + 1] * qs), p1 = pack_bf16x2(v[r + 2] * qs, v[r + 3] * qs);
      const uint32_t q0 = pack_bf16x2(v[r + 4] * qs, v[r + 5] * qs), q1 = pack_bf16x2(v[r + 6] * qs, v[r + 7] * qs);
      const auto s0 = __builtin_amdgcn_permlane32_swap(p0, q0, false, false);
      const auto s1 = __builtin_amdgcn_permlane32_swap(p1, q1, false, false);
      qreg[2 * dt + hf] = u32x4{s0[0], s1[0], s0[1], s1[1]};
    }
  // every wave is done with the staged operands before the DMA reuses them
  lds_barrier();
}

constexpr float RESCALE_LOG2 = 8.0f;

// S^T (32 keys x 32 queries) of one half tile: K rows from LDS (kp points at
// this lane's row and lane-group chunk), Q~ columns from registers.  CH = 2:
// two accumulation chains (even / odd 16-deep steps) keep the MFMA pipe busy
// when one half tile is scored at a time; CH = 1 when two independent half
// tiles are scored together (no VALU sum of the chains).
template <int DH, int CH = 2>
__device__ __forceinline__ f32x16 attn_scores(const uint8_t* kp, const u32x4* qreg) {
  constexpr int NKS = DH / 16;
  constexpr int KG = NKS < 8 ? NKS : 8;
  f32x16 s0 = f32x16{}, s1 = f32x16{};
#pragma unroll
  for (int k0 = 0; k0 < NKS; k0 += KG) {
    u32x4 ka[KG];
#pragma unroll
    for (int j = 0; j < KG; ++j) ka[j] = *(const u32x4*)(kp + (k0 + j) * 32);
#pragma unroll
    for (int j = 0; j < KG; ++j) {
      if (CH == 2 && (j & 1))
        s1 = mfma32(ka[j], qreg[k0 + j], s1);
      else
        s0 = mfma32(ka[j], qreg[k0 + j], s0);
    }
  }
  if constexpr (CH == 2) return s0 + s1;
  return s0;
}

// Logits of two half tiles: all K operand reads are issued before the
// MFMAs, so that the chain waits for LDS once rather than once per step.
template <int DH>
__device__ __forceinline__ void attn_scores_pair(const uint8_t* ka, const uint8_t* kb, const u32x4* qreg,
                                                 f32x16& sa, f32x16& sb) {
  constexpr int NKS = DH / 16;
  u32x4 ra[NKS], rb[NKS];
#pragma unroll
  for (int j = 0; j < NKS; ++j) {
    ra[j] = *(const u32x4*)(ka + j * 32);
    rb[j] = *(const u32x4*)(kb + j * 32);
  }
  __builtin_amdgcn_sched_barrier(0);
  sa = f32x16{};
  sb = f32x16{};
#pragma unroll
  for (int j = 0; j < NKS; ++j) {
    sa = mfma32(ra[j], qreg[j], sa);
    sb = mfma32(rb[j], qreg[j], sb);
  }
}

// Maximum that propagates NaN (the logits hold none): v_maximum3_f32 needs
// no canonicalising of its inputs, unlike fmaxf.
__device__ __forceinline__ float max3f(float a, float b, float c) {
  return __builtin_elementwise_maximum(__builtin_elementwise_maximum(a, b), c);
}

// Sum of the two bf16 values of a packed pair added to acc (v_dot2 with 1,1):
// the row sums then add exactly the rounded probabilities the PV product uses.
__device__ __forceinline__ float add_bf16x2(uint32_t p, float acc) {
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  const bf16x2_t one = {(__bf16)1.0f, (__bf16)1.0f};
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, p), one, acc, false);
}

// grid 8*n_qt*ceil(G/8) with G = n_obj*H*S key groups, block 256 (4 waves x
// 32 queries).  Block b -> key group 8*((b>>3)/n_qt) + (b&7), query tile
// (b>>3) % n_qt, so all query tiles of one key group share an XCD (and its L2).
// PROJ: the queries are projected here from X[sel] and W_q (heads of width
// <= 64); otherwise they are read from the projected buffer Q.
// DEEP (launches of at most one work-group per CU, heads of width <= 64):
// 8 stages and a loop over pairs of half tiles (two independent chains per
// iteration for the one wave per SIMD); otherwise 4 stages and a loop over
// single half tiles, which keeps the registers of several work-groups per CU.
// NG = 2 (deep form with the projection only): eight waves, two groups of
// four on the same 128 queries, each group taking every other pair of half
// tiles, so that two waves share each SIMD; their partials are merged at the
// end through LDS.
template <int DH, bool PROJ, bool DEEP, int NG = 1>
__global__ __launch_bounds__(256 * NG) void k_attn(Rs3ReadoutArgs a, int G) {
  static_assert(NG == 1 || (NG == 2 && DEEP && PROJ), "two wave groups need the deep form");
  constexpr int NT = 256 * NG;
  using L = AttnLds<DH>;
  constexpr int nst = DEEP ? 8 : 4;   // LDS stages
  extern __shared__ __attribute__((aligned(1024))) uint8_t lds[];   // nst * L::STAGE bytes
  const int bid = blockIdx.x;
  const int rest = bid >> 3;
  const int qt = rest % a.n_qt;
  const int kvg = (rest / a.n_qt) * 8 + (bid & 7);
  if (kvg >= G) return;
  const int s = kvg % a.S, oh = kvg / a.S, h = oh % a.H, o = oh / a.H;
  const int tid = threadIdx.x, lane = tid & 63, g = lane >> 5;
  const int wave_all = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wave = wave_all & 3;                 // the wave's 32 queries: rows 32*wave of the tile
  const int grp = NG == 2 ? wave_all >> 2 : 0;   // its group of key pairs
  const int row0 = qt * 128;
  const int qrow = row0 + 32 * wave + (lane & 31);
  // Loads that need nothing but the arguments are issued before the chain
  // descriptor -> header -> tile list: the query operands (rows past the
  // selected count are clamped into the buffers and zeroed below), or for
  // PROJ the W_q chunks and the gathered row indices.
  const int qrow_c = min(qrow, a.max_sel - 1);
  u32x4 qreg[DH / 16];
  int src[PROJ ? PJ_XCH / NG : 1];
  u32x4 wv[PROJ ? AttnProj<DH>::WCH / NG : 1];
  if constexpr (PROJ) {
    // the row indices first: the X loads wait for them alone
    attn_proj_rows<NT>(a.sel_idx + (int64_t)o * a.sel_stride, row0, a.max_sel, tid, src);
    attn_proj_load_w<DH, NT>((const bf16_t*)a.WqT, h, tid, wv);
  } else {
    const bf16_t* Qp = (const bf16_t*)a.Q + ((int64_t)o * a.max_sel + qrow_c) * a.D + h * DH;
#pragma unroll
    for (int ks = 0; ks < DH / 16; ++ks) qreg[ks] = gload((const u32x4*)(Qp + 16 * ks + 8 * g));
  }
  // the bank descriptor's pointers (one cache line), by scalar loads
  const BankDev* bd = a.banks[o];
  const uint64_t p_hdr = sload((const uint64_t*)&bd->hdr);
  const uint64_t p_tiles = sload((const uint64_t*)&bd->tiles);
  const uint64_t p_kh = sload((const uint64_t*)&bd->Khat);
  const uint64_t p_vh = sload((const uint64_t*)&bd->Vhat);
  // the exits below keep every value loaded so far, so that the compiler
  // issues those loads before the exit tests instead of after them
  auto keep_loads = [&]() {
    keep_s(p_hdr);
    keep_s(p_tiles);
    keep_s(p_kh);
    keep_s(p_vh);
    if constexpr (PROJ) {
#pragma unroll
      for (int i = 0; i < PJ_XCH / NG; ++i) keep(src[i]);
#pragma unroll
      for (int j = 0; j < AttnProj<DH>::WCH / NG; ++j) keep(wv[j]);
    } else {
#pragma unroll
      for (int ks = 0; ks < DH / 16; ++ks) keep(qreg[ks]);
    }
  };
  int cnt = sload(a.sel_count + (a.sel_stride ? o : 0));   // out of range: reported by the merge
  cnt = cnt < 0 ? 0 : min(cnt, a.max_sel);
  if (row0 >= cnt) {
    keep_loads();
    return;
  }
  const int32_t* hdr = (const int32_t*)p_hdr;
  u32x4 xv[PROJ ? PJ_XCH / NG : 1];
  if constexpr (PROJ) {
    // the gathered X rows, in flight while the tile list arrives (invalid
    // list entries read row 0; the merge kernel skips their rows)
    attn_proj_load_x<NT>((const bf16_t*)a.X + (int64_t)o * a.x_stride, a.mn, tid, src, xv);
  }
  const int ntiles = sload(hdr + HDR_NTILES);
  const int tps = split_tiles(ntiles, a.S);
  const int tb = min(s * tps, ntiles), te = min(tb + tps, ntiles);
  if (tb >= te) {
    keep_loads();
    if constexpr (PROJ) {
#pragma unroll
      for (int i = 0; i < PJ_XCH / NG; ++i) keep(xv[i]);
    }
    // a split without tiles still holds a partial for each of its rows: the
    // empty one (m = -inf, l = 0), so that the merge reads every split
    if (g == 0 && grp == 0 && qrow < cnt) {
      float* ml = a.ML + ((((int64_t)o * a.S + s) * a.max_sel + qrow) * a.H + h) * 2;
      ml[0] = -INFINITY;
      ml[1] = 0.f;
    }
    return;
  }
  const int ub = 2 * tb, ue = 2 * te;   // half tiles

  // values loaded from the bank descriptor are wave-uniform scalar loads, so
  // load addresses are base (SGPR) + lane offset
  const bf16_t* Kh = (const bf16_t*)p_kh;
  const bf16_t* Vh = (const bf16_t*)p_vh;
  const TileEnt* tiles = (const TileEnt*)p_tiles;
  const int H = a.H;
  const AttnDmaOffsets<DH> doff = attn_dma_offsets<DH>(wave, lane);

  // Resident-tile entries of this split are cached one per lane (a window of
  // 64 tiles, read back with readlane), so the loop issues no metadata loads
  // that would drain the prefetch queue.
  // The half tiles of the split are visited starting at an offset that
  // depends on the query tile: the workgroups sharing a split (same XCD) then
  // fetch different tiles at any moment and later visitors hit in L2, rather
  // than all waiting on the same HBM misses.  (Only for splits that fit the
  // window; the visiting order changes nothing but fp rounding.)
  const int nh = ue - ub;
  const int rot = (te - tb <= 64) ? ((qt & 7) * nh) >> 3 : 0;
  int cbase = tb, c_tile = 0;
  uint32_t c_mlo = 0, c_mhi = 0;
  if (tb + lane < te) {
    c_tile = gload(&tiles[tb + lane].tile);
    const uint64_t m = gload(&tiles[tb + lane].mask);
    c_mlo = (uint32_t)m;
    c_mhi = (uint32_t)(m >> 32);
  }
  settle(c_tile, c_mlo, c_mhi);
  const bool qv = qrow < cnt;
  if constexpr (PROJ) attn_project<DH, NT>(lds, tid, wave, lane, a.qscale, wv, xv, qreg);
  // i-th visited half tile
  auto half_at = [&](int i) { int v = i + rot; return ub + (v >= nh ? v - nh : v); };
#pragma unroll
  for (int ks = 0; ks < DH / 16; ++ks)
    if (!qv) qreg[ks] = u32x4{0, 0, 0, 0};

  f32x16 acc[DH / 32];
#pragma unroll
  for (int dt = 0; dt < DH / 32; ++dt) acc[dt] = f32x16{};
  float m_run = -INFINITY, l_run = 0.f;
  const int kbase = (lane & 31) * L::KP + 16 * g;             // + ks*32
  const int vbase = L::KREG + (lane & 31) * L::VP + 16 * g;   // + dt*32*VP + q*32
  if constexpr (NG == 2) {
    // Group g takes the pairs p = g, g+2, ... (pair p = half tiles 2p, 2p+1
    // in stages 2(p&3), 2(p&3)+1), so each group has two stage pairs.
    // Iteration j: wait for this wave's DMA of its pair p = 2j+g (issued one
    // iteration earlier); barrier (the group's previous pair is done and its
    // stages free); issue pair p+2 into them; compute pair p.  Every wave runs
    // the same iterations, so the barriers match.
    const int npair = nh >> 1;
    auto issue_pair = [&](int p) {
#pragma unroll
      for (int k = 0; k < 2; ++k) {
        const int v = half_at(2 * p + k);
        if ((v >> 1) - cbase >= 64) {
          // (unrotated splits longer than the window) slide it to this tile;
          // the masks of the pair being computed were read before
          wait_vmcnt<0>();
          cbase = v >> 1;
          c_tile = 0;
          if (cbase + lane < te) c_tile = gload(&tiles[cbase + lane].tile);
          const uint64_t mm = cbase + lane < te ? gload(&tiles[cbase + lane].mask) : 0ull;
          c_mlo = (uint32_t)mm;
          c_mhi = (uint32_t)(mm >> 32);
          settle(c_tile, c_mlo, c_mhi);
        }
        const int tl = __builtin_amdgcn_readlane(c_tile, (v >> 1) - cbase);
        attn_issue<DH>(Kh, Vh, tl, v & 1, h, H, lds + (2 * (p & 3) + k) * L::STAGE, wave, doff);
      }
    };
    if (grp < npair) issue_pair(grp);
    const int nit = (npair + 1) >> 1;
    for (int j = 0; j < nit; ++j) {
      const int p = 2 * j + grp;
      wait_vmcnt<0>();   // this wave's DMA of pair p, the only one in flight
      stage_barrier();
      uint32_t mA = 0, mB = 0;
      if (p < npair) {
        const int u0 = half_at(2 * p), u1 = half_at(2 * p + 1);
        const int t0 = (u0 >> 1) - cbase, t1 = (u1 >> 1) - cbase;
        mA = (u0 & 1) ? __builtin_amdgcn_readlane(c_mhi, t0) : __builtin_amdgcn_readlane(c_mlo, t0);
        mB = (u1 & 1) ? __builtin_amdgcn_readlane(c_mhi, t1) : __builtin_amdgcn_readlane(c_mlo, t1);
      }
      if (p + 2 < npair) issue_pair(p + 2);
      if ((mA | mB) == 0u) continue;
      const uint8_t* SA = lds + (2 * (p & 3)) * L::STAGE;
      const uint8_t* SB = SA + L::STAGE;
      f32x16 sA, sB;
      attn_scores_pair<DH>(SA + kbase, SB + kbase, qreg, sA, sB);
      if (mA != 0xffffffffu) {   // partial or empty half tile (frame boundary)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (!(mA >> c_row(r, lane) & 1u)) sA[r] = -INFINITY;
      }
      if (mB != 0xffffffffu) {
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (!(mB >> c_row(r, lane) & 1u)) sB[r] = -INFINITY;
      }
      float mx = __builtin_elementwise_maximum(sA[0], sB[0]);
#pragma unroll
      for (int r = 1; r < 16; ++r) mx = max3f(mx, sA[r], sB[r]);
      mx = max_with_partner(mx);
      const bool need = mx > m_run + RESCALE_LOG2;   // lazy rescale, as below
      if (__any(need)) {
        const float m_new = need ? mx : m_run;
        const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
        l_run *= alpha;
#pragma unroll
        for (int dt = 0; dt < DH / 32; ++dt) acc[dt] *= alpha;
        m_run = m_new;
      }
      float psum = 0.f;
      u32x4 pkA[2], pkB[2];
#pragma unroll
      for (int hf = 0; hf < 2; ++hf)
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
          const float a0 = __builtin_amdgcn_exp2f(sA[8 * hf + 2 * jj] - m_run);
          const float a1 = __builtin_amdgcn_exp2f(sA[8 * hf + 2 * jj + 1] - m_run);
          const float b0 = __builtin_amdgcn_exp2f(sB[8 * hf + 2 * jj] - m_run);
          const float b1 = __builtin_amdgcn_exp2f(sB[8 * hf + 2 * jj + 1] - m_run);
          pkA[hf][jj] = pack_bf16x2(a0, a1);
          pkB[hf][jj] = pack_bf16x2(b0, b1);
          psum = add_bf16x2(pkB[hf][jj], add_bf16x2(pkA[hf][jj], psum));
        }
      l_run += psum;
#pragma unroll
      for (int dt = 0; dt < DH / 32; ++dt) {
        u32x4 va[4];
#pragma unroll
        for (int q = 0; q < 2; ++q) {
          va[q] = *(const u32x4*)(SA + vbase + dt * 32 * L::VP + q * 32);
          va[2 + q] = *(const u32x4*)(SB + vbase + dt * 32 * L::VP + q * 32);
        }
#pragma unroll
        for (int q = 0; q < 2; ++q) acc[dt] = mfma32(va[q], pkA[q], acc[dt]);
#pragma unroll
        for (int q = 0; q < 2; ++q) acc[dt] = mfma32(va[2 + q], pkB[q], acc[dt]);
      }
    }
    // Group 1 hands its (m, l, O^T) per lane to its partner wave of group 0
    // through LDS (past the epilogue's row stage), then ends; group 0 merges
    // the two partials to the larger reference maximum.
    constexpr int SW = 2 + 16 * (DH / 32);   // floats per lane
    float* xs = (float*)(lds + 4 * 32 * (DH * 2 + 16)) + wave * SW * 64 + lane;
    __syncthreads();   // every wave is done with the stages
    if (grp == 1) {
      xs[0] = m_run;
      xs[64] = l_run;
#pragma unroll
      for (int dt = 0; dt < DH / 32; ++dt)
#pragma unroll
        for (int r = 0; r < 16; ++r) xs[(2 + 16 * dt + r) * 64] = acc[dt][r];
    }
    __syncthreads();
    if (grp == 1) return;
    const float m1 = xs[0], l1 = xs[64];
    const float mm = __builtin_elementwise_maximum(m_run, m1);
    const float s0 = mm == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m_run - mm);
    const float s1 = mm == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m1 - mm);
    l_run = l_run * s0 + l1 * s1;
#pragma unroll
    for (int dt = 0; dt < DH / 32; ++dt)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[dt][r] = acc[dt][r] * s0 + xs[(2 + 16 * dt + r) * 64] * s1;
    m_run = mm;
  } else if constexpr (DEEP) {
    // the first nst-2 half tiles; each pair iteration prefetches two more
#pragma unroll
    for (int j = 0; j < nst - 2; ++j)
      if (j < nh) {
        const int v = half_at(j);
        const int tl = __builtin_amdgcn_readlane(c_tile, (v >> 1) - cbase);
        attn_issue<DH>(Kh, Vh, tl, v & 1, h, H, lds + j * L::STAGE, wave, doff);
      }

    // Pairs of visited half tiles (nh is even; pair i/2 sits in stages i, i+1
    // mod nst).  Iteration i: wait until its pair landed; barrier (the
    // previous pair's stages are free); prefetch half tiles i+nst-2, i+nst-1
    // into them; the logits of both halves (independent MFMA chains), one
    // softmax update over the 64 keys, then O^T += V^T P^T for both.
    const int smask = nst - 1;
    for (int i = 0; i < nh; i += 2) {
      wait_stages<L::PER_WAVE, nst - 2>(min(i + nst - 2, nh) - (i + 2));
      stage_barrier();
      const int u0 = half_at(i), u1 = half_at(i + 1);
#pragma unroll
      for (int k = 0; k < 2; ++k)
        if (i + nst - 2 + k < nh) {
          const int v = half_at(i + nst - 2 + k);
          if ((v >> 1) - cbase >= 64) {
            // (unrotated splits longer than the window, whose pairs are whole
            // tiles) slide it to the tile being computed
            wait_vmcnt<0>();
            cbase = u0 >> 1;
            c_tile = 0;
            if (cbase + lane < te) c_tile = gload(&tiles[cbase + lane].tile);
            const uint64_t mm = cbase + lane < te ? gload(&tiles[cbase + lane].mask) : 0ull;
            c_mlo = (uint32_t)mm;
            c_mhi = (uint32_t)(mm >> 32);
            settle(c_tile, c_mlo, c_mhi);
          }
          const int tl = __builtin_amdgcn_readlane(c_tile, (v >> 1) - cbase);
          attn_issue<DH>(Kh, Vh, tl, v & 1, h, H, lds + ((i + nst - 2 + k) & smask) * L::STAGE, wave, doff);
        }
      const uint8_t* SA = lds + (i & smask) * L::STAGE;
      const uint8_t* SB = lds + ((i + 1) & smask) * L::STAGE;
      const int t0 = (u0 >> 1) - cbase, t1 = (u1 >> 1) - cbase;
      const uint32_t mA = (u0 & 1) ? __builtin_amdgcn_readlane(c_mhi, t0) : __builtin_amdgcn_readlane(c_mlo, t0);
      const uint32_t mB = (u1 & 1) ? __builtin_amdgcn_readlane(c_mhi, t1) : __builtin_amdgcn_readlane(c_mlo, t1);
      if ((mA | mB) == 0u) continue;
      f32x16 sA = attn_scores<DH, 1>(SA + kbase, qreg);
      f32x16 sB = attn_scores<DH, 1>(SB + kbase, qreg);
      if (mA != 0xffffffffu) {   // partial or empty half tile (frame boundary)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (!(mA >> c_row(r, lane) & 1u)) sA[r] = -INFINITY;
      }
      if (mB != 0xffffffffu) {
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (!(mB >> c_row(r, lane) & 1u)) sB[r] = -INFINITY;
      }
      float mx = __builtin_elementwise_maximum(sA[0], sB[0]);
#pragma unroll
      for (int r = 1; r < 16; ++r) mx = max3f(mx, sA[r], sB[r]);
      mx = max_with_partner(mx);
      // Lazy rescale: the reference max only moves when a pair exceeds it by
      // more than RESCALE_LOG2 (probabilities stay <= 2^RESCALE_LOG2); the
      // accumulators are touched only when some lane of the wave moves.
      const bool need = mx > m_run + RESCALE_LOG2;
      if (__any(need)) {
        const float m_new = need ? mx : m_run;
        const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);   // 0 on the first pair
        l_run *= alpha;
#pragma unroll
        for (int dt = 0; dt < DH / 32; ++dt) acc[dt] *= alpha;
        m_run = m_new;
      }
      float psum = 0.f;
      u32x4 pkA[2], pkB[2];
#pragma unroll
      for (int hf = 0; hf < 2; ++hf)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const float a0 = __builtin_amdgcn_exp2f(sA[8 * hf + 2 * j] - m_run);
          const float a1 = __builtin_amdgcn_exp2f(sA[8 * hf + 2 * j + 1] - m_run);
          const float b0 = __builtin_amdgcn_exp2f(sB[8 * hf + 2 * j] - m_run);
          const float b1 = __builtin_amdgcn_exp2f(sB[8 * hf + 2 * j + 1] - m_run);
          pkA[hf][j] = pack_bf16x2(a0, a1);
          pkB[hf][j] = pack_bf16x2(b0, b1);
          psum = add_bf16x2(pkB[hf][j], add_bf16x2(pkA[hf][j], psum));
        }
      l_run += psum;
      // O^T += V^T P^T over the 64 keys (two 16-key MFMA steps per half and d block)
#pragma unroll
      for (int dt = 0; dt < DH / 32; ++dt) {
        u32x4 va[4];
#pragma unroll
        for (int q = 0; q < 2; ++q) {
          va[q] = *(const u32x4*)(SA + vbase + dt * 32 * L::VP + q * 32);
          va[2 + q] = *(const u32x4*)(SB + vbase + dt * 32 * L::VP + q * 32);
        }
#pragma unroll
        for (int q = 0; q < 2; ++q) acc[dt] = mfma32(va[q], pkA[q], acc[dt]);
#pragma unroll
        for (int q = 0; q < 2; ++q) acc[dt] = mfma32(va[2 + q], pkB[q], acc[dt]);
      }
    }
  } else {
#pragma unroll
    for (int j = 0; j < nst - 1; ++j)
      if (j < nh) {
        const int v = half_at(j);
        const int tl = __builtin_amdgcn_readlane(c_tile, (v >> 1) - cbase);
        attn_issue<DH>(Kh, Vh, tl, v & 1, h, H, lds + j * L::STAGE, wave, doff);
      }

    // stage 0 must land before its scores: later stages issued = min(nst-2, nh-1)
    wait_stages<L::PER_WAVE, nst - 2>(min(nst - 2, nh - 1));
    stage_barrier();

    // Software pipeline over the visited half tiles i = 0 .. nh-1 (stage i%NST):
    //   iteration i: wait until stage i+1 landed; barrier (stage i-1 free);
    //   prefetch i+nst-1 into it; S^T(i+1) on the MFMA pipe while the VALU
    //   does the softmax of i; then O^T += V^T(i) P(i).
    const int smask = nst - 1;
    f32x16 sc = attn_scores<DH>(lds + kbase, qreg);
    for (int i = 0; i < nh; ++i) {
      const int st = i & smask;
      const int u = half_at(i);
      if (i + 1 < nh) wait_stages<L::PER_WAVE, nst - 2>(min(i + nst - 2, nh - 1) - (i + 1));
      stage_barrier();
      if (i + nst - 1 < nh) {
        const int v = half_at(i + nst - 1);
        if ((v >> 1) - cbase >= 64) {
          // (unrotated splits longer than the window) slide it to the tile
          // being computed
          wait_vmcnt<0>();
          cbase = u >> 1;
          c_tile = 0;
          if (cbase + lane < te) c_tile = gload(&tiles[cbase + lane].tile);
          const uint64_t mm = cbase + lane < te ? gload(&tiles[cbase + lane].mask) : 0ull;
          c_mlo = (uint32_t)mm;
          c_mhi = (uint32_t)(mm >> 32);
          settle(c_tile, c_mlo, c_mhi);
        }
        const int tl = __builtin_amdgcn_readlane(c_tile, (v >> 1) - cbase);
        attn_issue<DH>(Kh, Vh, tl, v & 1, h, H, lds + ((st + nst - 1) & smask) * L::STAGE, wave, doff);
      }
      const uint8_t* Sb = lds + st * L::STAGE;
      const int tu = (u >> 1) - cbase;
      const uint32_t msk = (u & 1) ? __builtin_amdgcn_readlane(c_mhi, tu) : __builtin_amdgcn_readlane(c_mlo, tu);

      // S^T of the next half tile (independent of the softmax below).  In the
      // last iteration the stage holds an earlier tile and the result is unused.
      const f32x16 sc_next = attn_scores<DH>(lds + ((st + 1) & smask) * L::STAGE + kbase, qreg);

      if (msk != 0u) {
        if (msk != 0xffffffffu) {  // partial half tile (frame boundary)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            if (!(msk >> c_row(r, lane) & 1u)) sc[r] = -INFINITY;
        }
        float mx = __builtin_elementwise_maximum(sc[0], sc[1]);
#pragma unroll
        for (int r = 2; r < 16; r += 2) mx = max3f(mx, sc[r], sc[r + 1]);
        mx = max_with_partner(mx);
        // Lazy rescale: the reference max only moves when a half tile exceeds
        // it by more than RESCALE_LOG2 (probabilities stay <= 2^RESCALE_LOG2);
        // the accumulators are touched only when some lane of the wave moves.
        const bool need = mx > m_run + RESCALE_LOG2;
        if (__any(need)) {
          const float m_new = need ? mx : m_run;
          const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);   // 0 on the first tile
          l_run *= alpha;
#pragma unroll
          for (int dt = 0; dt < DH / 32; ++dt) acc[dt] *= alpha;
          m_run = m_new;
        }
        float psum = 0.f;
        u32x4 pk[2];
#pragma unroll
        for (int hf = 0; hf < 2; ++hf)
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const float p0 = __builtin_amdgcn_exp2f(sc[8 * hf + 2 * j] - m_run);
            const float p1 = __builtin_amdgcn_exp2f(sc[8 * hf + 2 * j + 1] - m_run);
            pk[hf][j] = pack_bf16x2(p0, p1);
            psum = add_bf16x2(pk[hf][j], psum);
          }
        l_run += psum;
        // O^T += V^T P^T over the 32 keys (two 16-key MFMA steps per d block)
        constexpr int DB = DH / 32 >= 2 ? 2 : 1;   // d blocks whose operands are fetched together
#pragma unroll
        for (int dt = 0; dt < DH / 32; dt += DB) {
          u32x4 va[2 * DB];
#pragma unroll
          for (int q = 0; q < 2 * DB; ++q)
            va[q] = *(const u32x4*)(Sb + vbase + (dt + (q >> 1)) * 32 * L::VP + (q & 1) * 32);
#pragma unroll
          for (int q = 0; q < 2 * DB; ++q) acc[dt + (q >> 1)] = mfma32(va[q], pk[q & 1], acc[dt + (q >> 1)]);
        }
      }
      sc = sc_next;
    }
  }
  const float l_tot = sum_with_partner(l_run);
  const float inv = l_tot > 0.f ? __builtin_amdgcn_rcpf(l_tot) : 0.f;
  // Epilogue: stage this wave's 32 normalized rows in LDS as [query][d] bf16,
  // then write whole rows with 16-byte stores.
  constexpr int OP = DH * 2 + 16;
  __syncthreads();   // every wave is done with the stages
  uint8_t* ow = lds + wave * 32 * OP;
#pragma unroll
  for (int dt = 0; dt < DH / 32; ++dt)
#pragma unroll
    for (int q4 = 0; q4 < 4; ++q4) {
      const int d = 32 * dt + 8 * q4 + 4 * g;
      u32x2 w;
      w[0] = pack_bf16x2(acc[dt][4 * q4] * inv, acc[dt][4 * q4 + 1] * inv);
      w[1] = pack_bf16x2(acc[dt][4 * q4 + 2] * inv, acc[dt][4 * q4 + 3] * inv);
      *(u32x2*)(ow + (lane & 31) * OP + d * 2) = w;
    }
  if (g == 0 && qv) {
    const int64_t prow = ((int64_t)o * a.S + s) * a.max_sel + qrow;
    float* ml = a.ML + (prow * a.H + h) * 2;
    if (a.stream_parts) {
      pstore(ml, m_run);
      pstore(ml + 1, l_tot);
    } else {
      ml[0] = m_run;
      ml[1] = l_tot;
    }
  }
  __syncthreads();
  constexpr int CH = DH / 8;   // 16-byte chunks per row
  bf16_t* obase = (bf16_t*)a.Opart + (((int64_t)o * a.S + s) * a.max_sel) * a.D + h * DH;
#pragma unroll
  for (int q = lane; q < 32 * CH; q += 64) {
    const int rr = q / CH, c = q - rr * CH;
    const int row = row0 + 32 * wave + rr;
    if (row < cnt) {
      u32x4* dst = (u32x4*)(obase + (int64_t)row * a.D + 8 * c);
      const u32x4 v = *(const u32x4*)(ow + rr * OP + 16 * c);
      if (a.stream_parts)
        pstore(dst, v);
      else
        *dst = v;
    }
  }
}

// ---------------------------------------------------------------------------
// The attention of launches whose heads are 64 wide at d_model 256, that
// project their queries inside (no rotary table) and that fit the chip once
// (at most one work-group per CU): 512 threads, two groups of four waves on
// the same 128 queries, group g taking the pairs of half tiles g, g+2, ... of
// the split.  Split s holds the resident tiles s, s+S, s+2S, ... of the bank
// (interleaved rather than a contiguous range), so its tile entries can be
// loaded before the resident tile count is known.  The bank pointers come in
// the arguments.  The prologue issues every load as soon as its inputs exist:
//   1. from the arguments alone: the 128 row indices, the head's 64 rows of
//      W_q^T (coalesced), the split's tile entries (one per lane), the
//      resident tile count, the selected count;
//   2. the gathered X rows once the indices land, and each group's first pair
//      of half tiles (DMA into stages 0-3) once the entries and the count land;
//   3. the query projection in two passes over the channel halves (the X and
//      W_q halves are staged in LDS above stages 0-3, each thread writing its
//      chunks in one of the passes): group g computes d = 32g .. 32g+31 of
//      its wave's 32 queries (8 MFMAs per pass), and the partner waves of the
//      two groups swap their halves through LDS.
// The key loop and the merge of the two groups' partials follow the
// two-group form of k_attn.
constexpr int G2_DH = 64;
constexpr int G2_HC = PJ_PC / 2;                 // 16-byte chunks per row half

// A 16-byte LDS store the compiler does not see as one: after direct-to-LDS
// loads it orders every LDS store behind all of them (a full wait for the
// vector memory counter), while these stores touch none of their stages and
// need only their own data, which the register operand makes it wait for.
__device__ __forceinline__ void ds_store16(const uint8_t* p, const u32x4& v) {
  const uint32_t off = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) uint8_t*)p;
  asm volatile("ds_write_b128 %0, %1" ::"v"(off), "v"(v) : "memory");
}
constexpr int G2_PITCH = (G2_HC + 1) * 16;       // odd chunk count: conflict-free operand reads
struct G2Lds {
  static constexpr int STAGE = AttnLds<G2_DH>::STAGE;
  static constexpr int XOFF = 4 * STAGE;               // X row halves [128][G2_PITCH] during the projection
  static constexpr int WOFF = XOFF + 128 * G2_PITCH;   // W_q^T row halves [64][G2_PITCH]
  static constexpr int XCH = WOFF + G2_DH * G2_PITCH;  // halves of Q~: [8 waves][64 lanes][2] u32x4
  static constexpr int BYTES = XCH + 8 * 64 * 32;
};
static_assert(G2Lds::BYTES >= 8 * G2Lds::STAGE, "the eight stages fit");
static_assert(G2Lds::BYTES <= 160 * 1024, "one CU's LDS");

// QPRE (rs3_frame): the queries of every cell were projected by the energy
// launch (a.Qall); each lane gathers its query's projected row instead, and
// the projection steps 2-3 fall away.  ONE: a one-object launch (o = 0), so
// the bank table entries are at fixed offsets and join the first batch of
// argument loads.
template <bool QPRE, bool ONE>
__global__ __launch_bounds__(512) void k_attn_g2(Rs3ReadoutArgs a, int G, Rs3AttnBanks ab) {
  constexpr int DH = G2_DH, NT = 512;
  using L = AttnLds<DH>;
  extern __shared__ __attribute__((aligned(1024))) uint8_t lds[];   // G2Lds::BYTES
  // 0. the arguments of the prologue in one batch of scalar loads: the
  //    argument block is memory the host wrote just before the launch, so
  //    each batch that waits on an earlier one (a value tested by a branch,
  //    an index into a table) costs a memory round trip before the first
  //    data load
  int n_qt = a.n_qt, S = a.S, Harg = a.H, Gv = G, max_sel = a.max_sel, sel_stride = a.sel_stride, mn = a.mn;
  const int32_t* sel_idx = a.sel_idx;
  const int32_t* sel_count = a.sel_count;
  const void* Qall = a.Qall;
  int64_t qall_stride = a.qall_stride;
  const TileEnt* tiles0 = ab.tiles[0];
  const int32_t* hdr0 = ab.hdr[0];
  const void* kh0 = ab.kh[0];
  const void* vh0 = ab.vh[0];
  int ntcap0 = ab.ntcap[0];
  const void* WqT = a.WqT;
  const void* Xarg = a.X;
  int64_t x_stride = a.x_stride;
  int y_fp32 = a.y_fp32;
  // (one asm statement: each asm is a scheduling barrier, so separate ones
  // would split the batch; the table entries are read whatever ONE says.
  // y_fp32 shares a four-dword load with n_qt: held here, its register is
  // not reused by a later load of the batch, which would wait for the first)
  asm volatile(""
               : "+s"(n_qt), "+s"(S), "+s"(Harg), "+s"(Gv), "+s"(max_sel), "+s"(sel_stride), "+s"(mn),
                 "+s"(sel_idx), "+s"(sel_count), "+s"(Qall), "+s"(qall_stride), "+s"(WqT), "+s"(Xarg),
                 "+s"(x_stride), "+s"(tiles0), "+s"(hdr0), "+s"(kh0), "+s"(vh0), "+s"(ntcap0), "+s"(y_fp32));
  const int bid = blockIdx.x;
  const int rest = bid >> 3;
  const int qt = rest % n_qt;
  const int kvg = (rest / n_qt) * 8 + (bid & 7);
  if (kvg >= Gv) return;
  const int s = kvg % S, oh = kvg / S, h = oh % Harg, o = ONE ? 0 : oh / Harg;
  const int tid = threadIdx.x, lane = tid & 63, g = lane >> 5;
  const int wave_all = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wave = wave_all & 3;    // the wave's 32 queries: rows 32*wave of the tile
  const int grp = wave_all >> 2;    // its group: pairs grp, grp+2, ...; d-block grp of the projection
  const int row0 = qt * 128;
  const int qrow = row0 + 32 * wave + (lane & 31);

  // 1. loads that need only the arguments (the row indices first: the X loads
  //    wait for them alone).  Group g holds channel half g of the operands:
  //    thread lt = tid % 256 of the group holds chunk 16g + lt%16 of X rows
  //    lt/16 + 16 i and of W_q^T rows h*64 + lt/16 + 16 j.
  constexpr int NX = QPRE ? 1 : 8, NW = QPRE ? 1 : 4;
  const int lt = tid & 255, hchunk = G2_HC * grp + (lt & 15);
  int src[NX];
  u32x4 wreg[NW];
  const int32_t* sel = sel_idx + (int64_t)o * sel_stride;
  if constexpr (QPRE) {
    src[0] = gload(sel + min(qrow, max_sel - 1));   // this lane's query cell
  } else {
#pragma unroll
    for (int i = 0; i < NX; ++i) src[i] = gload(sel + min(row0 + (lt >> 4) + 16 * i, max_sel - 1));
    const u32x4* wb = (const u32x4*)((const bf16_t*)WqT + (int64_t)h * DH * PJ_PC * 8) + hchunk;
#pragma unroll
    for (int j = 0; j < NW; ++j) wreg[j] = gload(wb + ((lt >> 4) + 16 * j) * PJ_PC);
  }
  const TileEnt* tiles = ONE ? tiles0 : ab.tiles[o];
  const int ntcap = ONE ? ntcap0 : ab.ntcap[o];
  int c_tile;
  uint32_t c_mlo, c_mhi;
  {
    const int e = s + S * lane;   // entries past the list are read clamped and discarded
    const int ec = max(min(e, ntcap - 1), 0);
    c_tile = gload(&tiles[ec].tile);
    const uint64_t m = gload(&tiles[ec].mask);
    c_mlo = (uint32_t)m;
    c_mhi = (uint32_t)(m >> 32);
  }
  const int ntiles = sload((ONE ? hdr0 : ab.hdr[o]) + HDR_NTILES);
  int cnt = sload(sel_count + (sel_stride ? o : 0));   // out of range: reported by the merge
  cnt = cnt < 0 ? 0 : min(cnt, max_sel);
  auto keep_loads = [&]() {
#pragma unroll
    for (int i = 0; i < NX; ++i) keep(src[i]);
    if constexpr (!QPRE) {
#pragma unroll
      for (int j = 0; j < NW; ++j) keep(wreg[j]);
    }
    keep(c_tile);
    keep(c_mlo);
    keep(c_mhi);
  };
  if (row0 >= cnt) {
    keep_loads();
    return;
  }
  // 2. the gathered X rows (invalid list entries read row 0; the merge skips
  //    their rows)
  u32x4 xv[NX];
  if constexpr (!QPRE) {
    const bf16_t* X = (const bf16_t*)Xarg + (int64_t)o * x_stride;
#pragma unroll
    for (int i = 0; i < NX; ++i) {
      const int r = (src[i] < 0 || src[i] >= mn) ? 0 : src[i];
      xv[i] = gload((const u32x4*)(X + (int64_t)r * PJ_PC * 8) + hchunk);
    }
  }
  const int nts = ntiles > s ? (ntiles - s + S - 1) / S : 0;   // tiles of this split
  if (nts == 0) {
    keep_loads();
    if constexpr (!QPRE) {
#pragma unroll
      for (int i = 0; i < NX; ++i) keep(xv[i]);
    }
    // the empty partial (m = -inf, l = 0), so that the merge reads every split
    if (g == 0 && grp == 0 && qrow < cnt) {
      float* ml = a.ML + ((((int64_t)o * S + s) * max_sel + qrow) * Harg + h) * 2;
      ml[0] = -INFINITY;
      ml[1] = 0.f;
    }
    return;
  }
  if (c_tile < 0) c_tile = 0;   // (entries are tile indices; keeps the DMA in the ring)
  const int nh = 2 * nts;   // half tiles, visited from an offset that depends on the query tile
  const int rot = nts <= 64 ? ((qt & 7) * nh) >> 3 : 0;
  auto half_at = [&](int i) { int v = i + rot; return v >= nh ? v - nh : v; };
  const bf16_t* Kh = (const bf16_t*)(ONE ? kh0 : ab.kh[o]);
  const bf16_t* Vh = (const bf16_t*)(ONE ? vh0 : ab.vh[o]);
  const int H = Harg;
  const AttnDmaOffsets<DH> doff = attn_dma_offsets<DH>(wave, lane);
  int cbase = 0;   // local tile of lane 0's cached entry
  const int npair = nts;   // pairs of half tiles (nh is even)
  // DMA of pair p into stage slot `slot` (stages 2*slot, 2*slot+1)
  auto issue_pair = [&](int p, int slot) {
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      const int v = half_at(2 * p + k);
      if ((v >> 1) - cbase >= 64) {
        // (splits of more than 64 tiles, which are not rotated) slide the
        // window of cached entries to this tile; the masks of the pair being
        // computed were read before
        wait_vmcnt<0>();
        cbase = v >> 1;
        const int j = min(cbase + lane, nts - 1);
        c_tile = gload(&tiles[s + S * j].tile);
        const uint64_t mm = gload(&tiles[s + S * j].mask);
        c_mlo = (uint32_t)mm;
        c_mhi = (uint32_t)(mm >> 32);
        settle(c_tile, c_mlo, c_mhi);
      }
      const int tl = __builtin_amdgcn_readlane(c_tile, (v >> 1) - cbase);
      attn_issue<DH>(Kh, Vh, tl, v & 1, h, H, lds + (2 * slot + k) * L::STAGE, wave, doff);
    }
  };
  u32x4 qreg[DH / 16];
  if constexpr (QPRE) {
    // each group's first pair (as below), then this lane's projected query
    // row (invalid list entries read row 0; the merge skips their rows)
    const int p0 = min(grp, npair - 1);
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      const int v = half_at(2 * p0 + k);
      const int tl = __builtin_amdgcn_readlane(c_tile, v >> 1);
      attn_issue<DH>(Kh, Vh, tl, v & 1, h, H, lds + (2 * grp + k) * L::STAGE, wave, doff);
    }
    const int cell = (src[0] < 0 || src[0] >= mn) ? 0 : src[0];
    const bf16_t* qp = (const bf16_t*)Qall + (int64_t)o * qall_stride + (int64_t)cell * DH + 8 * g;
#pragma unroll
    for (int ks = 0; ks < DH / 16; ++ks) qreg[ks] = gload((const u32x4*)(qp + 16 * ks));
    // both in: the loop's first wait then finds nothing outstanding, and the
    // empty asm hands the rows on as settled values
    wait_vmcnt<0>();
#pragma unroll
    for (int ks = 0; ks < DH / 16; ++ks) asm volatile("" : "+v"(qreg[ks]));
  } else {
  // 3. query projection, d-block grp of the wave's 32 queries, in two passes
  //    over the channel halves: group p writes half p of the operands in pass
  //    p.  Pass 0's operands are stored before the first key/value DMA is
  //    issued: with ordinary loads and direct-to-LDS loads in flight together
  //    the compiler waits for all of them, so the X rows (which land last of
  //    the ordinary loads) are waited for first.
  f32x16 qa = f32x16{};
  const int cpos = (lt & 15) * 16;   // the thread's chunk within the row half
  // every wave's operands have landed before any DMA goes out (the empty
  // asm hands them on as settled values)
#pragma unroll
  for (int i = 0; i < NX; ++i) asm volatile("" : "+v"(xv[i]));
#pragma unroll
  for (int j = 0; j < NW; ++j) asm volatile("" : "+v"(wreg[j]));
#pragma unroll
  for (int pass = 0; pass < 2; ++pass) {
    if (pass == 1) lds_barrier();   // every wave is done with pass 0's operands
    if (grp == pass) {
#pragma unroll
      for (int i = 0; i < NX; ++i) ds_store16(lds + G2Lds::XOFF + ((lt >> 4) + 16 * i) * G2_PITCH + cpos, xv[i]);
#pragma unroll
      for (int j = 0; j < NW; ++j) ds_store16(lds + G2Lds::WOFF + ((lt >> 4) + 16 * j) * G2_PITCH + cpos, wreg[j]);
    }
    if (pass == 0) {
      // each group's first pair (a group without one loads the last pair into
      // its own slot, never computed); it lies in the window of cached entries
      // (a split of more than 64 tiles is not rotated)
      const int p0 = min(grp, npair - 1);
#pragma unroll
      for (int k = 0; k < 2; ++k) {
        const int v = half_at(2 * p0 + k);
        const int tl = __builtin_amdgcn_readlane(c_tile, v >> 1);
        attn_issue<DH>(Kh, Vh, tl, v & 1, h, H, lds + (2 * grp + k) * L::STAGE, wave, doff);
      }
    }
    lds_barrier();
    const uint8_t* xb = lds + G2Lds::XOFF + (32 * wave + (lane & 31)) * G2_PITCH + 16 * g;
    const uint8_t* wb = lds + G2Lds::WOFF + (32 * grp + (lane & 31)) * G2_PITCH + 16 * g;
    u32x4 bx[G2_HC / 2], aw[G2_HC / 2];
#pragma unroll
    for (int ks = 0; ks < G2_HC / 2; ++ks) {
      bx[ks] = *(const u32x4*)(xb + ks * 32);
      aw[ks] = *(const u32x4*)(wb + ks * 32);
    }
#pragma unroll
    for (int ks = 0; ks < G2_HC / 2; ++ks) qa = mfma32(aw[ks], bx[ks], qa);
  }
  // Lane l holds query l%32 at d = 32*grp + 8*(r/4) + 4*(l/32) + r%4; the B
  // operand of the logits needs d = 16*ks + 8*(l/32) + 0..7: one
  // v_permlane32_swap per register pair (as in attn_project).
  u32x4 mine[2];
  const float qs = a.qscale;
#pragma unroll
  for (int hf = 0; hf < 2; ++hf) {
    const int r = 8 * hf;
    const uint32_t p0 = pack_bf16x2(qa[r] * qs, qa[r + 1] * qs), p1 = pack_bf16x2(qa[r + 2] * qs, qa[r + 3] * qs);
    const uint32_t q0 = pack_bf16x2(qa[r + 4] * qs, qa[r + 5] * qs), q1 = pack_bf16x2(qa[r + 6] * qs, qa[r + 7] * qs);
    const auto s0 = __builtin_amdgcn_permlane32_swap(p0, q0, false, false);
    const auto s1 = __builtin_amdgcn_permlane32_swap(p1, q1, false, false);
    mine[hf] = u32x4{s0[0], s1[0], s0[1], s1[1]};
  }
  const uint8_t* xw = lds + G2Lds::XCH + (wave_all * 64 + lane) * 32;
  ds_store16(xw, mine[0]);
  ds_store16(xw + 16, mine[1]);
  lds_barrier();
  const u32x4* xr = (const u32x4*)(lds + G2Lds::XCH) + ((wave_all ^ 4) * 64 + lane) * 2;
  if (grp == 0) {
    qreg[0] = mine[0];
    qreg[1] = mine[1];
    qreg[2] = xr[0];
    qreg[3] = xr[1];
  } else {
    qreg[0] = xr[0];
    qreg[1] = xr[1];
    qreg[2] = mine[0];
    qreg[3] = mine[1];
  }
  }   // !QPRE
  const bool qv = qrow < cnt;
#pragma unroll
  for (int ks = 0; ks < DH / 16; ++ks)
    if (!qv) qreg[ks] = u32x4{0, 0, 0, 0};

  // key loop: iteration j waits for this wave's DMA of its pair p = 2j+grp
  // (issued one iteration earlier, or in the prologue), passes one barrier
  // (the group's previous pair is done and its stages free; in the first
  // iteration: every wave is done with the projection's LDS), issues pair
  // p+2 and computes pair p.
  // The logits come out of the MFMA already shifted by the running reference
  // maximum: the accumulator input is -m_run (one tile per lane, whose 16
  // values all belong to its query), so the common pair needs no
  // subtraction before the exponentials; only a pair that moves the
  // reference (the first one, then rarely) shifts its own logits.
  f32x16 acc[DH / 32];
#pragma unroll
  for (int dt = 0; dt < DH / 32; ++dt) acc[dt] = f32x16{};
  float m_run = -INFINITY, l_run = 0.f;
  f32x16 negm = f32x16{};   // -reference (0 until the first pair sets it)
  bool first = true;
  const int kbase = (lane & 31) * L::KP + 16 * g;
  const int vbase = L::KREG + (lane & 31) * L::VP + 16 * g;
  const int nit = (npair + 1) >> 1;
  for (int j = 0; j < nit; ++j) {
    const int p = 2 * j + grp;
    wait_vmcnt<0>();
    stage_barrier();
    uint32_t mA = 0, mB = 0;
    if (p < npair) {
      const int u0 = half_at(2 * p), u1 = half_at(2 * p + 1);
      const int t0 = (u0 >> 1) - cbase, t1 = (u1 >> 1) - cbase;
      mA = (u0 & 1) ? __builtin_amdgcn_readlane(c_mhi, t0) : __builtin_amdgcn_readlane(c_mlo, t0);
      mB = (u1 & 1) ? __builtin_amdgcn_readlane(c_mhi, t1) : __builtin_amdgcn_readlane(c_mlo, t1);
    }
    if (p + 2 < npair) issue_pair(p + 2, (p + 2) & 3);
    if ((mA | mB) == 0u) continue;
    const uint8_t* SA = lds + (2 * (p & 3)) * L::STAGE;
    const uint8_t* SB = SA + L::STAGE;
    f32x16 sA, sB;
    {
      u32x4 ra[DH / 16], rb[DH / 16];
#pragma unroll
      for (int jj = 0; jj < DH / 16; ++jj) {
        ra[jj] = *(const u32x4*)(SA + kbase + jj * 32);
        rb[jj] = *(const u32x4*)(SB + kbase + jj * 32);
      }
      __builtin_amdgcn_sched_barrier(0);
      sA = mfma32(ra[0], qreg[0], negm);
      sB = mfma32(rb[0], qreg[0], negm);
#pragma unroll
      for (int jj = 1; jj < DH / 16; ++jj) {
        sA = mfma32(ra[jj], qreg[jj], sA);
        sB = mfma32(rb[jj], qreg[jj], sB);
      }
    }
    if (mA != 0xffffffffu) {   // partial or empty half tile (frame boundary)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        if (!(mA >> c_row(r, lane) & 1u)) sA[r] = -INFINITY;
    }
    if (mB != 0xffffffffu) {
#pragma unroll
      for (int r = 0; r < 16; ++r)
        if (!(mB >> c_row(r, lane) & 1u)) sB[r] = -INFINITY;
    }
    float mx = __builtin_elementwise_maximum(sA[0], sB[0]);
#pragma unroll
    for (int r = 1; r < 16; ++r) mx = max3f(mx, sA[r], sB[r]);
    mx = max_with_partner(mx);   // relative to the reference
    // lazy rescale as in k_attn: the reference moves when a pair exceeds it
    // by more than RESCALE_LOG2 (and at the first pair, to its maximum)
    const bool need = first || mx > RESCALE_LOG2;
    if (__any(need)) {
      const float d = need ? mx : 0.f;
      const float alpha = first ? 0.f : __builtin_amdgcn_exp2f(-d);
      l_run *= alpha;
#pragma unroll
      for (int dt = 0; dt < DH / 32; ++dt) acc[dt] *= alpha;
      m_run = first ? d : m_run + d;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        sA[r] -= d;
        sB[r] -= d;
        negm[r] = -m_run;
      }
    }
    first = false;
    float psum = 0.f;
    u32x4 pkA[2], pkB[2];
#pragma unroll
    for (int hf = 0; hf < 2; ++hf)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        const float a0 = __builtin_amdgcn_exp2f(sA[8 * hf + 2 * jj]);
        const float a1 = __builtin_amdgcn_exp2f(sA[8 * hf + 2 * jj + 1]);
        const float b0 = __builtin_amdgcn_exp2f(sB[8 * hf + 2 * jj]);
        const float b1 = __builtin_amdgcn_exp2f(sB[8 * hf + 2 * jj + 1]);
        pkA[hf][jj] = pack_bf16x2(a0, a1);
        pkB[hf][jj] = pack_bf16x2(b0, b1);
        psum = add_bf16x2(pkB[hf][jj], add_bf16x2(pkA[hf][jj], psum));
      }
    l_run += psum;
#pragma unroll
    for (int dt = 0; dt < DH / 32; ++dt) {
      u32x4 va[4];
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        va[q] = *(const u32x4*)(SA + vbase + dt * 32 * L::VP + q * 32);
        va[2 + q] = *(const u32x4*)(SB + vbase + dt * 32 * L::VP + q * 32);
      }
#pragma unroll
      for (int q = 0; q < 2; ++q) acc[dt] = mfma32(va[q], pkA[q], acc[dt]);
#pragma unroll
      for (int q = 0; q < 2; ++q) acc[dt] = mfma32(va[2 + q], pkB[q], acc[dt]);
    }
  }
  // Group 1 hands its (m, l, O^T) per lane to its partner wave of group 0
  // through LDS, then ends; group 0 merges the two partials to the larger
  // reference maximum and stores the split's partial rows.
  constexpr int SW = 2 + 16 * (DH / 32);   // floats per lane
  float* xs = (float*)(lds + 4 * 32 * (DH * 2 + 16)) + wave * SW * 64 + lane;
  wait_vmcnt<0>();   // (a group without its last pair left a DMA in flight)
  __syncthreads();   // every wave is done with the stages
  if (grp == 1) {
    xs[0] = m_run;
    xs[64] = l_run;
#pragma unroll
    for (int dt = 0; dt < DH / 32; ++dt)
#pragma unroll
      for (int r = 0; r < 16; ++r) xs[(2 + 16 * dt + r) * 64] = acc[dt][r];
  }
  __syncthreads();
  if (grp == 1) return;
  {
    const float m1 = xs[0], l1 = xs[64];
    const float mm = __builtin_elementwise_maximum(m_run, m1);
    const float s0 = mm == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m_run - mm);
    const float s1 = mm == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m1 - mm);
    l_run = l_run * s0 + l1 * s1;
#pragma unroll
    for (int dt = 0; dt < DH / 32; ++dt)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[dt][r] = acc[dt][r] * s0 + xs[(2 + 16 * dt + r) * 64] * s1;
    m_run = mm;
  }
  const float l_tot = sum_with_partner(l_run);
  const float inv = l_tot > 0.f ? __builtin_amdgcn_rcpf(l_tot) : 0.f;
  // stage the wave's 32 normalised rows in LDS as [query][d] bf16 (below the
  // handed-over partials), then whole rows with 16-byte stores
  constexpr int OP = DH * 2 + 16;
  uint8_t* ow = lds + wave * 32 * OP;
#pragma unroll
  for (int dt = 0; dt < DH / 32; ++dt)
#pragma unroll
    for (int q4 = 0; q4 < 4; ++q4) {
      const int d = 32 * dt + 8 * q4 + 4 * g;
      u32x2 w;
      w[0] = pack_bf16x2(acc[dt][4 * q4] * inv, acc[dt][4 * q4 + 1] * inv);
      w[1] = pack_bf16x2(acc[dt][4 * q4 + 2] * inv, acc[dt][4 * q4 + 3] * inv);
      *(u32x2*)(ow + (lane & 31) * OP + d * 2) = w;
    }
  if (g == 0 && qv) {
    float* ml = a.ML + ((((int64_t)o * S + s) * max_sel + qrow) * H + h) * 2;
    pstore(ml, m_run);
    pstore(ml + 1, l_tot);
  }
  // the staged rows of this wave are written by this wave alone: a wave-local
  // wait for its LDS stores suffices
  __builtin_amdgcn_s_waitcnt(0xc07f);   // lgkmcnt(0)
  __builtin_amdgcn_wave_barrier();
  constexpr int CH = DH / 8;   // 16-byte chunks per row
  bf16_t* obase = (bf16_t*)a.Opart + (((int64_t)o * S + s) * a.max_sel) * a.D + h * DH;
#pragma unroll
  for (int q = lane; q < 32 * CH; q += 64) {
    const int rr = q / CH, c = q - rr * CH;
    const int row = row0 + 32 * wave + rr;
    if (row < cnt) pstore((u32x4*)(obase + (int64_t)row * a.D + 8 * c), *(const u32x4*)(ow + rr * OP + 16 * c));
  }
}

// ---------------------------------------------------------------------------
// grid (n_obj, ceil(max_sel/cb_rows_for(D, n_obj, max_sel))), block CB_THREADS: one merge block each.
template <typename OutT>
__global__ __launch_bounds__(CB_THREADS) void k_combine(Rs3ReadoutArgs a) {
  extern __shared__ __attribute__((aligned(16))) uint8_t cl[];
  combine_block<OutT>(a, blockIdx.x, blockIdx.y, cl);
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
// fp32 path: grid (n_obj, max_sel), block 256, one selected row per
// work-group; its four waves split the resident tiles (wave w takes tiles
// w, w+4, ...) and merge their softmax states at the end.  For row i:
//   q = qscale * x W_q              threads over the attention columns
//   per head and tile of a wave:    lanes over the tile's 64 keys: logits,
//     wave max / sum (online softmax); lanes over the head's columns:
//     o = alpha*o + sum_k p_k v_k   (weights broadcast from LDS)
//   merge of the four waves' (m, l, o) per head, then
//   y = x + (o / l) W_o             threads over the output channels
// Every load that needs only the arguments (count, header, the first tile
// entries, the list entries, W_q rows) is issued first, and a wave's first
// key and value rows (heads of at most 64 columns) before the query is
// ready, so that the row's chain of dependent loads stays short.
// LDS: x [C], q [D], o [4][D], p [4][64], (m, l) [4][H] floats.
__global__ __launch_bounds__(256) void k_readout_f32(Rs3ReadoutArgs a, Rs3AttnBanks ab) {
  extern __shared__ float sm[];
  const int o = blockIdx.x, r = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int C = a.C, D = a.D, H = a.H, d_h = a.d_h;
  float* xs = sm;
  float* q = xs + C;
  float* ow = q + D + wave * D;        // this wave's o
  float* pr = q + 5 * D + wave * 64;   // this wave's weights of one tile
  float* ml = q + 5 * D + 256;         // [4][H][2]
  int32_t* hdr = (int32_t*)ab.hdr[o];
  const TileEnt* tiles = ab.tiles[o];
  const int ntcap = ab.ntcap[o];
  int cnt = gload(a.sel_count + (a.sel_stride ? o : 0));
  const int ntiles = gload(hdr + HDR_NTILES);
  // tile entries t = wave + 4*lane (a wave's first 64 tiles)
  int c_tile = 0;
  uint32_t c_lo = 0, c_hi = 0;
  if (wave + 4 * lane < ntcap) {
    c_tile = gload(&tiles[wave + 4 * lane].tile);
    const uint64_t mm = gload(&tiles[wave + 4 * lane].mask);
    c_lo = (uint32_t)mm;
    c_hi = (uint32_t)(mm >> 32);
  }
  const int32_t* sel = a.sel_idx + (int64_t)o * a.sel_stride;
  const int rc = min(r, a.max_sel - 1);
  const int i_raw = gload(sel + rc), i_prev = rc > 0 ? gload(sel + rc - 1) : -1;
  if (cnt < 0 || cnt > a.max_sel) {
    if (r == 0 && tid == 0) set_err(hdr, RS3_E_INVALID);
    cnt = cnt < 0 ? 0 : a.max_sel;
  }
  if (r >= cnt) return;
  if (!(i_raw >= 0 && i_raw < a.mn && i_prev < i_raw)) {
    if (tid == 0) set_err(hdr, RS3_E_INVALID);
    return;
  }
  const int i = i_raw;
  const float* x = (const float*)a.X + (int64_t)o * a.x_stride + (int64_t)i * C;
  float* y = (float*)a.Y + (int64_t)o * a.y_stride + (int64_t)i * C;
  if (ntiles == 0) {
    for (int c = tid; c < C; c += 256) gstore(y + c, gload(x + c));
    return;
  }
  const float* Kh = (const float*)ab.kh[o];
  const float* Vh = (const float*)ab.vh[o];
  const bool fast = d_h <= 64 && (d_h & 3) == 0 && ntiles <= 256;
  // fast path: the key row (lane = key) and value row (lane = column) of a
  // tile of this wave, first tile in flight before the query is ready
  f32x4 kc[16], vc[16];
  auto load_tile = [&](int j, int h) {   // j: the wave's j-th tile
    const int tl = __builtin_amdgcn_readlane(c_tile, j);
    const f32x4* kr = (const f32x4*)(Kh + (((int64_t)tl * H + h) * KT + lane) * d_h);
    const f32x4* vr = (const f32x4*)(Vh + (((int64_t)tl * H + h) * d_h + min(lane, d_h - 1)) * KT);
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      if (4 * u < d_h) kc[u] = gload(kr + u);
      vc[u] = gload(vr + u);
    }
  };
  const int nmine = ntiles > wave ? (ntiles - wave + 3) / 4 : 0;   // this wave's tiles
  if (fast && nmine > 0) load_tile(0, 0);
  for (int c = tid; c < C; c += 256) xs[c] = gload(x + c);
  __syncthreads();
  const float* WqT = (const float*)a.WqT;
  for (int d = tid; d < D; d += 256) {
    const f32x4* wr = (const f32x4*)(WqT + (int64_t)d * C);
    float s0 = 0.f, s1 = 0.f;
    for (int c4 = 0; c4 < C / 4; c4 += 2) {
      const f32x4 w0 = gload(wr + c4), x0 = *(const f32x4*)(xs + 4 * c4);
      s0 = fmaf(x0[0], w0[0], fmaf(x0[1], w0[1], fmaf(x0[2], w0[2], fmaf(x0[3], w0[3], s0))));
      if (c4 + 1 < C / 4) {
        const f32x4 w1 = gload(wr + c4 + 1), x1 = *(const f32x4*)(xs + 4 * c4 + 4);
        s1 = fmaf(x1[0], w1[0], fmaf(x1[1], w1[1], fmaf(x1[2], w1[2], fmaf(x1[3], w1[3], s1))));
      }
    }
    q[d] = (s0 + s1) * a.qscale;
  }
  __syncthreads();
  if (a.rope) {
    // Eq. 7: turn each head's channel pairs by the factors of cell i
    const float* f = a.rope + (int64_t)i * d_h;   // d_h/2 (cos, sin) pairs
    for (int pp = tid; pp < D / 2; pp += 256) {
      const int d = 2 * pp, fp = (d % d_h) & ~1;
      const float c = gload(f + fp), sn = gload(f + fp + 1), xe = q[d], xo = q[d + 1];
      q[d] = xe * c - xo * sn;
      q[d + 1] = xe * sn + xo * c;
    }
    __syncthreads();
  }
  for (int h = 0; h < H; ++h) {
    float m_run = -INFINITY, l_run = 0.f;
    const float* qh = q + h * d_h;
    for (int dd = lane; dd < d_h; dd += 64) ow[h * d_h + dd] = 0.f;
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    for (int j = 0; j < nmine; ++j) {
      const int t = wave + 4 * j;
      int etile;
      uint64_t emask;
      if (fast) {
        etile = __builtin_amdgcn_readlane(c_tile, j);
        emask = (uint64_t)__builtin_amdgcn_readlane(c_lo, j) | ((uint64_t)__builtin_amdgcn_readlane(c_hi, j) << 32);
        if (j > 0 || h > 0) load_tile(j, h);
      } else {
        etile = gload(&tiles[t].tile);
        emask = gload(&tiles[t].mask);
      }
      const bool valid = emask >> lane & 1ull;
      float s0 = 0.f, s1 = 0.f;
      if (fast) {
#pragma unroll
        for (int u = 0; u < 16; u += 2) {
          if (4 * u < d_h) {
            const f32x4 q0 = *(const f32x4*)(qh + 4 * u);
            s0 = fmaf(q0[0], kc[u][0], fmaf(q0[1], kc[u][1], fmaf(q0[2], kc[u][2], fmaf(q0[3], kc[u][3], s0))));
          }
          if (4 * u + 4 < d_h) {
            const f32x4 q1 = *(const f32x4*)(qh + 4 * u + 4);
            s1 = fmaf(q1[0], kc[u + 1][0], fmaf(q1[1], kc[u + 1][1], fmaf(q1[2], kc[u + 1][2], fmaf(q1[3], kc[u + 1][3], s1))));
          }
        }
      } else {
        const float* krow = Kh + (((int64_t)etile * H + h) * KT + lane) * d_h;
        for (int u = 0; u < d_h; ++u) s0 = fmaf(qh[u], gload(krow + u), s0);
      }
      const float s = valid ? s0 + s1 : -INFINITY;
      const float mx = wave_max(s);
      if (mx == -INFINITY) continue;   // no resident key in the tile
      const float m_new = fmaxf(m_run, mx);
      const float alpha = exp2f(m_run - m_new);   // 0 on the wave's first keys
      const float p = valid ? exp2f(s - m_new) : 0.f;
      l_run = l_run * alpha + wave_sum(p);
      m_run = m_new;
      pr[lane] = p;
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      // slot quad 4j of a V^ row holds the key quad vslot(4j) (the slot
      // permutation swaps whole quads and is its own inverse)
      if (fast) {
        if (lane < d_h) {
          float acc = ow[h * d_h + lane] * alpha;
#pragma unroll
          for (int u = 0; u < 16; ++u) {
            const f32x4 pk = *(const f32x4*)(pr + vslot(4 * u));
            acc = fmaf(pk[0], vc[u][0], fmaf(pk[1], vc[u][1], fmaf(pk[2], vc[u][2], fmaf(pk[3], vc[u][3], acc))));
          }
          ow[h * d_h + lane] = acc;
        }
      } else {
        for (int dd = lane; dd < d_h; dd += 64) {
          const float* vr = Vh + (((int64_t)etile * H + h) * d_h + dd) * KT;
          float acc = ow[h * d_h + dd] * alpha;
          for (int k = 0; k < KT; ++k) acc = fmaf(pr[vslot(k)], gload(vr + k), acc);
          ow[h * d_h + dd] = acc;
        }
      }
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    }
    if (lane == 0) {
      ml[(wave * H + h) * 2] = m_run;
      ml[(wave * H + h) * 2 + 1] = l_run;
    }
  }
  __syncthreads();
  // merge the waves' states into q's place: o = sum_w e^(m_w - M) o_w / sum_w e^(m_w - M) l_w
  float* of = q;
  for (int d = tid; d < D; d += 256) {
    const int h = d / d_h;
    float M = -INFINITY;
    for (int w = 0; w < 4; ++w) M = fmaxf(M, ml[(w * H + h) * 2]);
    float num = 0.f, den = 0.f;
    if (M != -INFINITY)
      for (int w = 0; w < 4; ++w) {
        const float mw = ml[(w * H + h) * 2];
        if (mw == -INFINITY) continue;
        const float sc = exp2f(mw - M);
        num = fmaf(sc, q[D + w * D + d], num);
        den = fmaf(sc, ml[(w * H + h) * 2 + 1], den);
      }
    of[d] = den > 0.f ? num / den : 0.f;
  }
  __syncthreads();
  const float* WoT = (const float*)a.WoT;
  for (int c = tid; c < C; c += 256) {
    const f32x4* wr = (const f32x4*)(WoT + (int64_t)c * D);
    float s0 = 0.f, s1 = 0.f;
    for (int d4 = 0; d4 < D / 4; d4 += 2) {
      const f32x4 w0 = gload(wr + d4), o0 = *(const f32x4*)(of + 4 * d4);
      s0 = fmaf(o0[0], w0[0], fmaf(o0[1], w0[1], fmaf(o0[2], w0[2], fmaf(o0[3], w0[3], s0))));
      if (d4 + 1 < D / 4) {
        const f32x4 w1 = gload(wr + d4 + 1), o1 = *(const f32x4*)(of + 4 * d4 + 4);
        s1 = fmaf(o1[0], w1[0], fmaf(o1[1], w1[1], fmaf(o1[2], w1[2], fmaf(o1[3], w1[3], s1))));
      }
    }
    gstore(y + c, xs[c] + (s0 + s1));
  }
}

}  // namespace rs3

using namespace rs3;

// Launches of at most one work-group per CU take the deep form of the
// attention where its 8 stages fit the LDS (heads of width <= 64).
constexpr int ATTN_DEEP_MAX_BLOCKS = 256;

template <int DH, bool PROJ, bool DEEP, int NG = 1>
static hipError_t launch_attn_dh(const Rs3ReadoutArgs& a, int G, int nblk, hipStream_t st) {
  size_t lds = (size_t)(DEEP ? 8 : 4) * AttnLds<DH>::STAGE;
  if constexpr (PROJ) lds = lds > (size_t)AttnProj<DH>::BYTES ? lds : (size_t)AttnProj<DH>::BYTES;
  RS3_LAUNCH(RS3_K_ATTN, st, (k_attn<DH, PROJ, DEEP, NG>), dim3(nblk), dim3(256 * NG), lds, st, a, G);
  return hipGetLastError();
}

// Launches of at most one work-group per CU with heads of width <= 64 at
// d_model 256 project their queries inside the attention (the staged
// operands would cost larger launches their occupancy); rotary layers
// project in k_qproj, which turns the rows.
static bool attn_projects(const Rs3ReadoutArgs& a) {
  const int G = a.n_obj * a.H * a.S;
  const int nblk = 8 * a.n_qt * ((G + 7) / 8);
  return a.d_h <= 64 && a.C == 8 * PJ_PC && nblk <= ATTN_DEEP_MAX_BLOCKS && !a.rope;
}

bool rs3_attn_projects(const Rs3ReadoutArgs& a) { return attn_projects(a); }

hipError_t rs3_launch_attn(const Rs3ReadoutArgs& a, const Rs3AttnBanks& ab, hipStream_t st, bool project) {
  const int G = a.n_obj * a.H * a.S;
  const int nblk = 8 * a.n_qt * ((G + 7) / 8);
  if (project && !attn_projects(a)) return hipErrorInvalidValue;
  const bool deep = nblk <= ATTN_DEEP_MAX_BLOCKS;
  switch (a.d_h) {
    case 32:
      if (project) return launch_attn_dh<32, true, true, 2>(a, G, nblk, st);
      return deep ? launch_attn_dh<32, false, true>(a, G, nblk, st) : launch_attn_dh<32, false, false>(a, G, nblk, st);
    case 64:
      if (project) {
        const bool one = a.n_obj == 1;
        if (a.Qall && one)
          RS3_LAUNCH(RS3_K_ATTN, st, (k_attn_g2<true, true>), dim3(nblk), dim3(512), 8 * G2Lds::STAGE, st, a, G, ab);
        else if (a.Qall)
          RS3_LAUNCH(RS3_K_ATTN, st, (k_attn_g2<true, false>), dim3(nblk), dim3(512), 8 * G2Lds::STAGE, st, a, G, ab);
        else if (one)
          RS3_LAUNCH(RS3_K_ATTN, st, (k_attn_g2<false, true>), dim3(nblk), dim3(512), G2Lds::BYTES, st, a, G, ab);
        else
          RS3_LAUNCH(RS3_K_ATTN, st, (k_attn_g2<false, false>), dim3(nblk), dim3(512), G2Lds::BYTES, st, a, G, ab);
        return hipGetLastError();
      }
      return deep ? launch_attn_dh<64, false, true>(a, G, nblk, st) : launch_attn_dh<64, false, false>(a, G, nblk, st);
    case 128: return launch_attn_dh<128, false, false>(a, G, nblk, st);
    case 256: return launch_attn_dh<256, false, false>(a, G, nblk, st);
    default: return hipErrorInvalidValue;
  }
}

hipError_t rs3_launch_readout(const Rs3ReadoutArgs& a, const Rs3AttnBanks& ab, int dtype, hipStream_t st, bool merge,
                              bool* pending) {
  if (pending) *pending = false;
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
    size_t lds = (size_t)(a.C + 5 * a.D + 256 + 8 * a.H) * 4;
    RS3_LAUNCH(RS3_K_READOUT_F32, st, k_readout_f32, dim3(a.n_obj, a.max_sel), dim3(256), lds, st, a, ab);
    return hipGetLastError();
  }
  const bool project = attn_projects(a);
  if (!project) {
    RS3_LAUNCH(RS3_K_QPROJ, st, k_qproj, dim3(a.n_obj, (a.max_sel + 63) / 64, a.D / 64), dim3(256), 0, st, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipError_t e = rs3_launch_attn(a, ab, st, project);
  if (e != hipSuccess) return e;
  if (!merge) {
    if (pending) *pending = true;
    return hipSuccess;
  }
  return rs3_launch_combine(a, st);
}

hipError_t rs3_launch_combine(const Rs3ReadoutArgs& a, hipStream_t st) {
  const size_t lds = combine_lds_bytes(a.D);
  const int rb = cb_rows_for(a.D, a.n_obj, a.max_sel);
  const dim3 cgrid(a.n_obj, (a.max_sel + rb - 1) / rb);
  if (a.y_fp32)
    RS3_LAUNCH(RS3_K_COMBINE, st, k_combine<float>, cgrid, dim3(CB_THREADS), lds, st, a);
  else
    RS3_LAUNCH(RS3_K_COMBINE, st, k_combine<bf16_t>, cgrid, dim3(CB_THREADS), lds, st, a);
  return hipGetLastError();
}

hipError_t rs3_readout_setup() {
  // D <= 1024 (checked on the host)
  size_t max_lds = 0;
  for (int D = 64; D <= 1024; D += 64) {
    const size_t b = combine_lds_bytes(D);
    if (b > max_lds) max_lds = b;
  }
  hipError_t e = hipFuncSetAttribute((const void*)k_combine<bf16_t>, hipFuncAttributeMaxDynamicSharedMemorySize,
                                     (int)max_lds);
  if (e != hipSuccess) return e;
  // the attention's stages: 8 for heads of width <= 64, else 4
  const struct {
    const void* f;
    int bytes;
  } attn[] = {{(const void*)k_attn<32, false, false>, 4 * AttnLds<32>::STAGE},
              {(const void*)k_attn<32, false, true>, 8 * AttnLds<32>::STAGE},
              {(const void*)k_attn<32, true, true, 2>, std::max(8 * AttnLds<32>::STAGE, AttnProj<32>::BYTES)},
              {(const void*)k_attn<64, false, false>, 4 * AttnLds<64>::STAGE},
              {(const void*)k_attn<64, false, true>, 8 * AttnLds<64>::STAGE},
              {(const void*)k_attn_g2<false, false>, G2Lds::BYTES},
              {(const void*)k_attn_g2<false, true>, G2Lds::BYTES},
              {(const void*)k_attn_g2<true, false>, 8 * G2Lds::STAGE},
              {(const void*)k_attn_g2<true, true>, 8 * G2Lds::STAGE},
              {(const void*)k_attn<128, false, false>, 4 * AttnLds<128>::STAGE},
              {(const void*)k_attn<256, false, false>, 4 * AttnLds<256>::STAGE}};
  for (const auto& k : attn) {
    e = hipFuncSetAttribute(k.f, hipFuncAttributeMaxDynamicSharedMemorySize, k.bytes);
    if (e != hipSuccess) return e;
  }
  return hipFuncSetAttribute((const void*)k_combine<float>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)max_lds);
}
