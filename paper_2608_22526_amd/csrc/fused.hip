// One launch for the tail of a frame: the merge of the readout's key splits
// (output projection and residual scatter, Sec. 3.1, Eq. 6) and the commit
// of the frame's memory tokens (Sec. 3.2, Eq. 8).  The two touch disjoint
// data -- the merge reads the attention partials, X and W_o and writes Y;
// the commit reads the memory tokens and the bank state and writes the bank
// -- so their work-groups run side by side in one grid instead of one launch
// after the other.
//
// Block b < n_cb is merge block (b % n_obj, b / n_obj) of the readout; the
// others are commit blocks in the same flattened order.  The block size is
// the commit's; a merge block uses its first CB_THREADS threads and the rest
// end at once (a work-group barrier waits only for the waves still running).
#include "combine.h"
#include "commit_body.h"

namespace rs3 {

// The argument block is memory the host wrote just before the launch: every
// argument that either kind of block reads before its first data load, and
// the first entries of the bank tables (the table lines of one-object
// launches), are loaded in one batch at the start (one memory round trip),
// so that the later loads behind the block-kind test and the table index
// find them in the scalar cache.
template <typename OutT, bool BF16>
__global__ __launch_bounds__(CP_THREADS) void k_merge_commit(Rs3ReadoutArgs ra, Rs3CommitArgs ca, int n_cb) {
  extern __shared__ __attribute__((aligned(16))) uint8_t dyn[];
  asm volatile("" ::"s"(n_cb), "s"(ra.n_obj), "s"(ra.D), "s"(ra.max_sel), "s"(ra.sel_idx), "s"(ra.sel_stride),
               "s"(ra.X), "s"(ra.x_stride), "s"(ra.WoT), "s"(ra.sel_count), "s"(ra.S), "s"(ra.C),
               "s"(ca.n_obj), "s"(ca.masks), "s"(ca.m), "s"(ca.n), "s"(ca.s), "s"(ca.parity), "s"(ca.t),
               "s"(ca.fall_min), "s"(ca.fall_max), "s"(ca.banks[0]), "s"(ra.banks[0]));
  const int b = blockIdx.x;
  if (b < n_cb) {
    if (threadIdx.x >= CB_THREADS) return;
    combine_block<OutT>(ra, b % ra.n_obj, b / ra.n_obj, dyn);
  } else {
    const int c = b - n_cb;
    commit_block<BF16>(ca, c % ca.n_obj, c / ca.n_obj, (int32_t*)dyn);
  }
}

}  // namespace rs3

using namespace rs3;

static size_t merge_commit_lds(int D, int d_kv) {
  const size_t cb = combine_lds_bytes(D), cp = CP_FMAX * 16 + commit_stage_bytes(RS3_BF16, d_kv);
  return cb > cp ? cb : cp;
}

hipError_t rs3_fused_setup() {
  // D <= 1024, d_kv <= 256 (checked on the host)
  size_t max_lds = 0;
  for (int D = 64; D <= 1024; D += 64) {
    const size_t b = merge_commit_lds(D, 256);
    if (b > max_lds) max_lds = b;
  }
  const void* fs[] = {(const void*)k_merge_commit<bf16_t, true>, (const void*)k_merge_commit<float, true>};
  for (const void* f : fs) {
    hipError_t e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, (int)max_lds);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// Work-groups of the fused launch beyond which the merge and the commit run
// as two launches: a fused work-group has the commit's 1,024 threads, whose
// register count (126) allows one per CU, while the merge's 512-thread
// blocks fit two per CU on their own (149 us fused against 75 + 34 us
// separate at 64 objects of 898 selected rows).
constexpr int FUSE_MAX_WGS = 1024;

hipError_t rs3_launch_merge_commit(const Rs3ReadoutArgs& ra, const Rs3CommitArgs& ca, int d_kv, hipStream_t st) {
  const int rb = cb_rows_for(ra.D, ra.n_obj, ra.max_sel), n_cb = ra.n_obj * ((ra.max_sel + rb - 1) / rb);
  const int mn = ca.m * ca.n;
  Rs3CommitArgs c = ca;
  c.rows_per_wg = commit_rows_per_wg(ca.n_obj, mn);
  const int n_cp = ca.n_obj * (1 + (mn + c.rows_per_wg - 1) / c.rows_per_wg);
  if (n_cb + n_cp > FUSE_MAX_WGS) {
    hipError_t e = rs3_launch_combine(ra, st);
    return e == hipSuccess ? rs3_launch_commit(ca, RS3_BF16, d_kv, 0, 0, 0, st) : e;
  }
  const size_t lds = merge_commit_lds(ra.D, d_kv);
  const dim3 grid(n_cb + n_cp), blk(CP_THREADS);
  if (ra.y_fp32)
    RS3_LAUNCH(RS3_K_MERGE_COMMIT, st, (k_merge_commit<float, true>), grid, blk, lds, st, ra, c, n_cb);
  else
    RS3_LAUNCH(RS3_K_MERGE_COMMIT, st, (k_merge_commit<bf16_t, true>), grid, blk, lds, st, ra, c, n_cb);
  return hipGetLastError();
}
