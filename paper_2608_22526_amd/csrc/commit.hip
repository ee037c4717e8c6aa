// Store-sparse commit (Sec. 3.2, Eq. 8; sparse write of Algorithm 1).
//
// k_commit : grid (n_obj, 1 + ceil(mn/R)), block 1024, R = rows_per_wg.
//            Every work-group of an object compacts the mask to the ascending
//            kept list (ordered block scan, dense fall-through) and runs the
//            placement rule (documented in rs3.h; one wave) on its own LDS
//            copy of the frame table as it was before this commit (copy p of
//            the double-buffered table), so all of them know the new frame's
//            start row.  Work-group 0 writes the new state to copy 1-p, the
//            key count and the list of resident 64-row tiles with their row
//            masks; work-group 1 + b appends kept rows Rb .. Rb+R-1, 64 per
//            round (R = 64 unless a call would launch far more work-groups
//            than CUs): the raw K/V rows into the ring, their cells into
//            `pos`, and their projections K^ = K W_k, V^ = V W_v into the
//            tile-blocked attention layouts (bf16 MFMA with fp32
//            accumulation, or fp32 FMA loops; the raw rows re-laid in
//            absorbed mode).
// k_commit_append_* / k_bank_tiles : the same append and tile rebuild for a
//            bank restored from a snapshot (rows already in the ring).
#include "commit_body.h"

namespace rs3 {

// Bank restore: frame table from device memory, then the tile list and the
// key count (grid 1, block CP_THREADS, dynamic LDS f_max*16 bytes).
__global__ __launch_bounds__(CP_THREADS) void k_bank_tiles(Rs3CommitArgs a) {
  extern __shared__ __attribute__((aligned(16))) int32_t sfr[];
  __shared__ CpShared sh;
  const int tid = threadIdx.x;
  const BankDev& b = *a.banks[0];
  const int p = (int)(a.parity & 1);
  const int nf = b.hdr[HDR_NFRAMES + HDR_COPY * p];
  if (tid < 4 * nf) sfr[tid] = b.frames[4 * b.f_max * p + tid];
  __syncthreads();
  if (tid == 0) {
    int keys = 0;
    for (int f = 0; f < nf; ++f) keys += sfr[4 * f + 1];
    b.hdr[HDR_NKEYS] = keys;
    b.hdr[HDR_PLEN] = -1;
  }
  rebuild_tiles(b, sfr, nf, sh);
}

// Restored bank: rows [hdr PSTART, + PLEN) of bank 0 from the raw ring,
// 64 per work-group.
__global__ __launch_bounds__(256) void k_commit_append_bf16(Rs3CommitArgs a) {
  extern __shared__ __attribute__((aligned(16))) bf16_t rows_lds[];
  __shared__ int spos[64];
  const int o = blockIdx.x;
  const BankDev& b = *a.banks[o];
  const int L = b.hdr[HDR_PLEN];
  const int r0 = blockIdx.y * 64;
  if (L < 0 || r0 >= L) return;
  const int start = b.hdr[HDR_PSTART];
  const int rows = min(64, L - r0);
  if (threadIdx.x < 64) spos[threadIdx.x] = (int)threadIdx.x < rows ? b.pos[start + r0 + threadIdx.x] : 0;
  __syncthreads();
  append_bf16<256>(a, b, o, start, r0, rows, spos, rows_lds);
}

// Restored bank: rows [hdr PSTART, + PLEN) of bank 0 from the raw ring,
// 64 per work-group.
__global__ __launch_bounds__(256) void k_commit_append_f32(Rs3CommitArgs a) {
  __shared__ __attribute__((aligned(16))) float sK[64 * F32_SP], sV[64 * F32_SP], sW[64 * F32_WP];
  __shared__ int spos[64];
  const int o = blockIdx.x;
  const BankDev& b = *a.banks[o];
  const int L = b.hdr[HDR_PLEN];
  const int r0 = blockIdx.y * 64;
  if (L < 0 || r0 >= L) return;
  const int start = b.hdr[HDR_PSTART];
  const int rows = min(64, L - r0);
  if (threadIdx.x < 64) spos[threadIdx.x] = (int)threadIdx.x < rows ? b.pos[start + r0 + threadIdx.x] : 0;
  __syncthreads();
  append_f32<256>(a, b, o, start, r0, rows, spos, sK, sV, sW);
}

// grid (n_obj, 1 + ceil(kept rows / rows_per_wg)), block CP_THREADS.
template <bool BF16>
__global__ __launch_bounds__(CP_THREADS) void k_commit(Rs3CommitArgs a) {
  extern __shared__ __attribute__((aligned(16))) int32_t dyn[];
  commit_block<BF16>(a, blockIdx.x, blockIdx.y, dyn);
}

}  // namespace rs3

using namespace rs3;


hipError_t rs3_commit_setup() {
  hipError_t e = hipFuncSetAttribute((const void*)k_commit_append_bf16, hipFuncAttributeMaxDynamicSharedMemorySize,
                                     (int)commit_stage_bytes(RS3_BF16, 256));
  if (e == hipSuccess)
    e = hipFuncSetAttribute((const void*)k_commit<true>, hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)(CP_FMAX * 16 + commit_stage_bytes(RS3_BF16, 256)));
  if (e == hipSuccess)
    e = hipFuncSetAttribute((const void*)k_commit<false>, hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)(CP_FMAX * 16 + commit_stage_bytes(RS3_F32, 256)));
  return e;
}

hipError_t rs3_launch_commit(const Rs3CommitArgs& a, int dtype, int d_kv, int D, int H, int d_h,
                             hipStream_t st) {
  (void)D;
  (void)H;
  (void)d_h;
  const int mn = a.m * a.n;
  Rs3CommitArgs b = a;
  b.rows_per_wg = commit_rows_per_wg(a.n_obj, mn);
  const dim3 grid(a.n_obj, 1 + (mn + b.rows_per_wg - 1) / b.rows_per_wg);
  const size_t lds = CP_FMAX * 16 + commit_stage_bytes(dtype, d_kv);
  if (dtype == RS3_BF16)
    RS3_LAUNCH(RS3_K_COMMIT, st, k_commit<true>, grid, dim3(CP_THREADS), lds, st, b);
  else
    RS3_LAUNCH(RS3_K_COMMIT, st, k_commit<false>, grid, dim3(CP_THREADS), lds, st, b);
  return hipGetLastError();
}

hipError_t rs3_launch_bank_restore(const Rs3CommitArgs& a, int dtype, int d_kv, int rebuild, hipStream_t st) {
  if (rebuild) {
    hipLaunchKernelGGL(k_bank_tiles, dim3(1), dim3(CP_THREADS), CP_FMAX * 16, st, a);
    return hipGetLastError();
  }
  const int mn = a.m * a.n;   // upper bound on the rows of the span
  dim3 grid(1, (mn + 63) / 64);
  if (dtype == RS3_BF16)
    hipLaunchKernelGGL(k_commit_append_bf16, grid, dim3(256), commit_stage_bytes(RS3_BF16, d_kv), st, a);
  else
    hipLaunchKernelGGL(k_commit_append_f32, grid, dim3(256), 0, st, a);
  return hipGetLastError();
}
