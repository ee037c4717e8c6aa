// Merge of the key splits, output projection and residual scatter of the
// readout (Sec. 3.1, Eq. 6), as a device function shared by the merge kernel
// and the fused merge + commit launch.
#pragma once

#include "device_util.h"

namespace rs3 {

// ---------------------------------------------------------------------------
template <typename OutT>
__device__ __forceinline__ void store_out(OutT* p, float v);
template <>
__device__ __forceinline__ void store_out<bf16_t>(bf16_t* p, float v) { gstore(p, f2bf(v)); }
template <>
__device__ __forceinline__ void store_out<float>(float* p, float v) { gstore(p, v); }

template <typename OutT>
__device__ __forceinline__ void copy_out(OutT* p, bf16_t x);
template <>
__device__ __forceinline__ void copy_out<bf16_t>(bf16_t* p, bf16_t x) { gstore(p, x); }
template <>
__device__ __forceinline__ void copy_out<float>(float* p, bf16_t x) { gstore(p, bf2f(x)); }

// grid (n_obj, ceil(max_sel/cb_rows_for(D, n_obj, max_sel))), block 512.  Every key split of the call
// holds a partial for every selected row (the attention writes l = 0 for
// splits without tiles), so the merge needs nothing from the bank.
// 1. the row indices are loaded and checked;
// 2. for each (row, 8-column chunk) item, each of the NG thread groups that
//    share it loads the (m, l) pairs and partial O chunks of its splits grp,
//    grp + NG, ... (PART_B per batch, the first batch together with the
//    residual inputs and W_o operands) and merges them by log-sum-exp in
//    registers; NG is as large as the threads allow but no larger than S
//    needs.  The NG groups are merged through LDS, and the normalised row
//    goes to LDS as bf16;
// 3. y = x + O W_o on a 32x32x16 MFMA whose rows past the block's are zero; a row with
//    no resident key (total weight 0) is returned as x, bit for bit.
// Rows per work-group, at most CB_ROWS (the W_o step maps them to
// accumulator rows r < 8).  8 at attention widths up to 64 when the call's
// 8-row blocks fit the chip's 256 CUs at once: the merge of many splits is
// VALU-bound per work-group, so the rows spread over more CUs.  Else 16,
// since every work-group reads all of W_o and larger grids gain nothing from
// smaller blocks.
constexpr int CB_ROWS = 16;
__host__ __device__ inline int cb_rows_for(int D, int n_obj, int max_sel) {
  return D <= 64 && (int64_t)n_obj * ((max_sel + 7) / 8) <= 256 ? 8 : CB_ROWS;
}
constexpr int CB_THREADS = 512;
constexpr int PART_B = 8;     // splits per batch of partial loads

__host__ __device__ constexpr int cb_groups(int D, int rows) {
  return CB_THREADS / (rows * (D / 8)) < 1 ? 1
         : (CB_THREADS / (rows * (D / 8)) > 8 ? 8 : CB_THREADS / (rows * (D / 8)));
}

struct PartBatch {
  float m[PART_B], l[PART_B];
  u32x4 v[PART_B];
};

// Batch j of one item's partials: splits grp + NG*(PART_B*j + i); indices
// past S re-read split S-1 (masked in the merge), rows past max_sel re-read
// row max_sel-1 (not stored): no branch around the loads.
__device__ __forceinline__ void part_load(const Rs3ReadoutArgs& a, int o, int row, int d0, int h, int grp, int NG,
                                          int j, PartBatch& pb) {
  const int64_t rows = a.max_sel;
  const int rw = min(row, a.max_sel - 1);
#pragma unroll
  for (int i = 0; i < PART_B; ++i) {
    const int sp = min(grp + NG * (PART_B * j + i), a.S - 1);
    const int64_t prow = ((int64_t)o * a.S + sp) * rows + rw;
    typedef float f32x2 __attribute__((ext_vector_type(2)));
    const f32x2 ml = pload((const f32x2*)(a.ML + (prow * a.H + h) * 2));
    pb.m[i] = ml[0];
    pb.l[i] = ml[1];
    pb.v[i] = pload((const u32x4*)((const bf16_t*)a.Opart + prow * a.D + d0));
  }
}

// Log-sum-exp merge of a batch into the running maximum M, weight W and sum
// acc: the batch's largest maximum is found first, so the running sums are
// rescaled once per batch instead of once per split.  Splits that are off
// (past S, or empty with l = 0) add nothing; their partial O words are
// replaced by zero before use, since an empty split leaves its O unwritten.
__device__ __forceinline__ void part_merge(const PartBatch& pb, int first, int NG, int S, float& M, float& W,
                                           float (&acc)[8]) {
  bool on[PART_B];
  float mb = -INFINITY;
#pragma unroll
  for (int i = 0; i < PART_B; ++i) {
    on[i] = first + NG * i < S && pb.l[i] > 0.f;
    mb = __builtin_elementwise_maximum(mb, on[i] ? pb.m[i] : -INFINITY);
  }
  if (mb == -INFINITY) return;
  const float Mn = __builtin_elementwise_maximum(M, mb);
  const float sc = __builtin_amdgcn_exp2f(M - Mn);   // 0 while M = -inf
  W *= sc;
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] *= sc;
#pragma unroll
  for (int i = 0; i < PART_B; ++i) {
    const float w = on[i] ? __builtin_amdgcn_exp2f(pb.m[i] - Mn) * pb.l[i] : 0.f;
    W += w;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const uint32_t x = on[i] ? pb.v[i][e] : 0u;
      acc[2 * e] += w * __uint_as_float(x << 16);
      acc[2 * e + 1] += w * __uint_as_float(x & 0xffff0000u);
    }
  }
  M = Mn;
}

// The merge of rows [ry*RB, +RB) of object o, RB = cb_rows_for(D, n_obj, max_sel), by CB_THREADS threads
// (threadIdx.x < CB_THREADS), cl: combine_lds_bytes(D) bytes of LDS.
template <typename OutT>
__device__ __forceinline__ void combine_block(const Rs3ReadoutArgs& a, int o, int ry, uint8_t* cl) {
  const int RB = cb_rows_for(a.D, a.n_obj, a.max_sel);
  const int r0 = ry * RB;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, g = lane >> 5;
  const int D = a.D, C = a.C, d_h = a.d_h, S = a.S, OS = D + 8;
  const int cpr = D / 8, items = RB * cpr;
  const int NG = min(cb_groups(D, RB), max(1, (S + PART_B - 1) / PART_B));   // thread groups per item
  const int nb = (S + NG * PART_B - 1) / (NG * PART_B);   // batches per item
  const int32_t* sel = a.sel_idx + (int64_t)o * a.sel_stride;
  const bf16_t* X = (const bf16_t*)a.X + (int64_t)o * a.x_stride;
  const bf16_t* WoT = (const bf16_t*)a.WoT;

  // 1. The list entries of this lane's accumulator rows r < 8 (rows
  //    8*(r/4) + 4*g + r%4 < RB) and their predecessors (ascending
  //    check), and of row r0 + tid for the error report: the only loads
  //    before the row decisions, so waiting for them waits for nothing else.
  int srow[8], sprv[8];
#pragma unroll
  for (int r = 0; r < 8; ++r) {
    const int rc = min(r0 + c_row(r, lane), a.max_sel - 1);
    srow[r] = gload(sel + rc);
    sprv[r] = gload(sel + max(rc - 1, 0));
  }
  const int erc = min(r0 + (tid & (RB - 1)), a.max_sel - 1);
  const int e_cur = gload(sel + erc), e_prv = gload(sel + max(erc - 1, 0));
  BankDev& b = *a.banks[o];
  // the merge covers every selected row: it reports a count past max_sel and
  // invalid (out of range or not ascending) list entries, whose rows it skips
  const int cnt = sel_count_of(a, o, b, ry == 0 && tid == 0);
  if (r0 >= cnt) return;
  // entry i of row r is valid iff it is in range and above its predecessor
  auto entry_ok = [&](int i, int prev, int r) { return i >= 0 && i < a.mn && (r == 0 || prev < i); };
  // LDS: Os [CB_ROWS][D+8] bf16 | red [NG][items][10] f32 | kept [CB_ROWS] | sdst [CB_ROWS]
  bf16_t* Os = (bf16_t*)cl;
  float* red = (float*)(cl + ((CB_ROWS * OS * 2 + 15) & ~15));
  int* kept = (int*)(red + (size_t)NG * items * 10);
  int* sdst = kept + CB_ROWS;
  // destination cell of each row of the block (-1 = none), kept in LDS for
  // the output step rather than in registers across the merge
  if (tid < RB) {
    const bool ok = r0 + tid < cnt && entry_ok(e_cur, e_prv, r0 + tid);
    if (r0 + tid < cnt && !ok) set_err(b.hdr, RS3_E_INVALID);
    sdst[tid] = ok ? e_cur : -1;
  }
  int dst[8];   // destination cell of each accumulator row (-1 = none)
#pragma unroll
  for (int r = 0; r < 8; ++r) {
    const int row = r0 + c_row(r, lane);
    dst[r] = (c_row(r, lane) < RB && row < cnt && entry_ok(srow[r], sprv[r], row)) ? srow[r] : -1;
  }
  // 2. Every data load in one batch: residual inputs of the wave's first
  //    column block, its first W_o operands, and this thread's first item's
  //    first batch of partials (waves past the last column block, C < 256,
  //    re-read the last column).
  const int col0 = 32 * wave + (lane & 31);
  bf16_t xv0[8];
#pragma unroll
  for (int r = 0; r < 8; ++r) xv0[r] = gload(X + (int64_t)max(dst[r], 0) * C + min(col0, C - 1));
  constexpr int KB = 4;   // k steps per batch of W_o operands (D is a multiple of 64)
  u32x4 bv0[KB];
  {
    const bf16_t* wr = WoT + (int64_t)min(col0, C - 1) * D;
#pragma unroll
    for (int j = 0; j < KB; ++j) bv0[j] = gload((const u32x4*)(wr + 16 * j + 8 * g));
  }
  const int q0 = tid;
  PartBatch pb;
  {
    const int item0 = q0 % items, grp0 = q0 / items;
    const int rr = item0 / cpr, d0 = 8 * (item0 - rr * cpr);
    if (q0 < items * NG) part_load(a, o, r0 + rr, d0, d0 / d_h, grp0, NG, 0, pb);
  }

  // merge
  for (int q = q0; q < items * NG; q += CB_THREADS) {
    const int item = q % items, grp = q / items;
    const int rr = item / cpr, d0 = 8 * (item - rr * cpr), h = d0 / d_h;
    float M = -INFINITY, W = 0.f;
    float acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    for (int j = 0; j < nb; ++j) {
      if (q != q0 || j > 0) part_load(a, o, r0 + rr, d0, h, grp, NG, j, pb);
      part_merge(pb, grp + NG * PART_B * j, NG, S, M, W, acc);
    }
    float* dstp = red + (size_t)grp * 10 * items + item;   // [NG][10][items]
    dstp[0] = M;
    dstp[items] = W;
#pragma unroll
    for (int e = 0; e < 8; ++e) dstp[(2 + e) * items] = acc[e];
  }
  lds_barrier();
  for (int item = tid; item < items; item += CB_THREADS) {
    float M = -INFINITY;
    for (int grp = 0; grp < NG; ++grp) M = fmaxf(M, red[(size_t)grp * 10 * items + item]);
    float W = 0.f, acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    if (M != -INFINITY)
      for (int grp = 0; grp < NG; ++grp) {
        const float* sp = red + (size_t)grp * 10 * items + item;
        const float sc = __builtin_amdgcn_exp2f(sp[0] - M);   // 0 for empty groups
        W += sc * sp[items];
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[e] += sc * sp[(2 + e) * items];
      }
    const float inv = W > 0.f ? 1.f / W : 0.f;
    const int rr = item / cpr, d0 = 8 * (item - rr * cpr);
    u32x4 pk;
#pragma unroll
    for (int j = 0; j < 4; ++j) pk[j] = pack_bf16x2(acc[2 * j] * inv, acc[2 * j + 1] * inv);
    *(u32x4*)&Os[rr * OS + d0] = pk;
    if (d0 == 0) kept[rr] = W > 0.f;
  }
  lds_barrier();
  // 3. y = x + O W_o for the block's rows, columns split over the waves
  OutT* Y = (OutT*)a.Y + (int64_t)o * a.y_stride;
  const bool arow = (lane & 31) < RB;
  const bf16_t* orow = &Os[(arow ? (lane & 31) : 0) * OS + 8 * g];
  bool keys[8];
#pragma unroll
  for (int r = 0; r < 8; ++r) {
    keys[r] = c_row(r, lane) < RB && kept[c_row(r, lane)] != 0;
    dst[r] = c_row(r, lane) < RB ? sdst[c_row(r, lane)] : -1;
  }
  for (int nbk = wave; nbk < C / 32; nbk += CB_THREADS / 64) {
    const bool first = nbk == wave;
    const int col = 32 * nbk + (lane & 31);
    const bf16_t* wr = WoT + (int64_t)col * D + 8 * g;
    bf16_t xv[8];
#pragma unroll
    for (int r = 0; r < 8; ++r) xv[r] = first ? xv0[r] : gload(X + (int64_t)max(dst[r], 0) * C + col);
    f32x16 acc = {};
    for (int k0 = 0; k0 < D; k0 += 16 * KB) {
      u32x4 av[KB], bv[KB];
#pragma unroll
      for (int j = 0; j < KB; ++j) {
        av[j] = arow ? *(const u32x4*)(orow + k0 + 16 * j) : u32x4{0, 0, 0, 0};
        bv[j] = (first && k0 == 0) ? bv0[j] : gload((const u32x4*)(wr + k0 + 16 * j));
      }
#pragma unroll
      for (int j = 0; j < KB; ++j) acc = mfma32(av[j], bv[j], acc);
    }
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      if (dst[r] < 0) continue;
      const int64_t off = (int64_t)dst[r] * C + col;
      if (!keys[r])
        copy_out<OutT>(&Y[off], xv[r]);
      else
        store_out<OutT>(&Y[off], bf2f(xv[r]) + acc[r]);
    }
  }
}

__host__ __device__ inline size_t combine_lds_bytes(int D) {
  size_t red = 0;   // the larger of the two row counts' merge buffers
  for (int rb = 8; rb <= CB_ROWS; rb *= 2) {
    const size_t b = (size_t)cb_groups(D, rb) * rb * (D / 8) * 10 * 4;
    red = b > red ? b : red;
  }
  return (((size_t)CB_ROWS * (D + 8) * 2 + 15) & ~(size_t)15) + red + 2 * CB_ROWS * 4;
}

}  // namespace rs3
