// Internal definitions shared by the HIP kernels and the host side of the
// rs3 library (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <hip/hip_ext.h>
#include <stdint.h>

#include "rs3.h"

namespace rs3 {

// ---- bank layout -----------------------------------------------------------
// Device header words of a bank.  The frame count and pin end exist twice,
// like the frame table: a commit of parity p (the bank's commit count mod 2,
// kept by the host) reads copy p and writes copy 1-p, so that every
// work-group of the commit reads the state from before it.
enum : int {
  HDR_NFRAMES = 0,   // resident frames (copy 0; copy 1 at + HDR_COPY)
  HDR_PINEND = 1,    // rows occupied by pinned frames (copy 0; copy 1 at + HDR_COPY)
  HDR_ERR = 2,       // sticky error word (first error wins)
  HDR_PSTART = 3,    // row where the pending append starts
  HDR_PLEN = 4,      // rows of the pending append, -1 when none
  HDR_NTILES = 5,    // entries in the resident tile list
  HDR_NKEYS = 6,     // resident rows (N)
  HDR_COPY = 8,
  HDR_WORDS = 16
};

constexpr int KT = 64;  // keys per bank tile

// Resident tile: ring rows [64*tile, 64*tile+64), bit j set iff row 64*tile+j
// belongs to a resident frame.
struct TileEnt {
  int32_t tile;
  int32_t pad;
  uint64_t mask;
};

// Device-resident descriptor of one bank.
//  Kraw, Vraw : [cap][d_kv] (dtype), raw rows as committed
//  pos        : [cap] int32, kept cell index of each row
//  Khat       : [n_tiles_cap][H][64][d_h]   rows = keys, d contiguous
//  Vhat       : [n_tiles_cap][H][d_h][64]   keys contiguous in the slot
//               order of vslot() (see below)
//  hdr        : [HDR_WORDS] int32
//  frames     : [2][f_max][4] int32 {start, len, t, pinned} in key order
//               (copy p current for a bank of commit parity p)
//  tiles      : [n_tiles_cap] TileEnt, ascending tile index
struct BankDev {
  int32_t cap, f_max, n_pin, d_kv, H, d_h, dtype, n_tiles_cap;
  void* Kraw;
  void* Vraw;
  int32_t* pos;
  void* Khat;
  void* Vhat;
  int32_t* hdr;
  int32_t* frames;
  TileEnt* tiles;
};

// Slot of key j (0..63) inside a V^ tile.  Within each 16-key group the two
// middle quads swap places ([0-3, 8-11, 4-7, 12-15]), so the eight keys that
// one lane feeds to a 16-deep bf16 MFMA step after the key-major logits are
// contiguous (see the attention kernel).
__host__ __device__ inline int vslot(int j) {
  int w = j & 15;
  return (j & ~15) | (((w >> 2) & 1) << 3) | ((w >> 3) << 2) | (w & 3);
}

// ---- layer -----------------------------------------------------------------
// Device weights, transposed so that every MFMA operand reads contiguous
// 16-byte runs along the contraction dimension.
// The attention runs at width Da over Ha heads of width dah:
//   projected: Da = D, Ha = H, dah = d_h; WqT = W_q^T [D][C], WoT = W_o^T [C][D]
//   absorbed : Da = d_kv, Ha = 1, dah = d_kv; WqT = (W_q W_k^T)^T [d_kv][C],
//              WoT = (W_v W_o)^T [C][d_kv]; WkT/WvT unused (null)
// Optional rotary table (projected mode): rope [rope_m*rope_n][d_h/2] of
// (cos, sin) fp32 pairs, null when absent.
struct LayerDev {
  int32_t C, H, d_h, D, d_kv, dtype, absorb;
  int32_t Da, Ha, dah;
  void* WqT;
  void* WkT;  // [D][d_kv] (projected mode)
  void* WvT;  // [D][d_kv] (projected mode)
  void* WoT;
  float* rope;
  int32_t rope_m, rope_n;
};

struct Launch {
  hipStream_t stream;
};

// ---- bf16 helpers ----------------------------------------------------------
typedef uint16_t bf16_t;

__device__ __forceinline__ float bf2f(bf16_t b) {
  return __uint_as_float(((uint32_t)b) << 16);
}

// fp32 -> bf16, round to nearest even (NaN stays NaN).
__device__ __forceinline__ bf16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (bf16_t)((u >> 16) | 0x40);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (bf16_t)(u >> 16);
}

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

// D = A(32x16) * B(16x32) + C.  Lane l supplies A row l%32 and B column l%32,
// each with the eight k values 8*(l/32) .. 8*(l/32)+7.  The 16 results of lane
// l are column l%32, rows 8*(r/4) + 4*(l/32) + (r%4) for r = 0..15.
__device__ __forceinline__ f32x16 mfma32(u32x4 a, u32x4 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(a), as_bf16x8(b), c, 0, 0, 0);
}

__device__ __forceinline__ int c_row(int r, int lane) { return 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3); }

// Two fp32 values -> packed bf16 pair (round to nearest even, v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  bf16x2_t v = {(__bf16)lo, (__bf16)hi};
  return __builtin_bit_cast(uint32_t, v);
}

// Key splits of a query tile: every split gets at least MIN_TILES_PER_SPLIT
// resident tiles, so with few tiles only the first splits are active.
constexpr int MIN_TILES_PER_SPLIT = 2;
// Key splits times heads per readout call (bounds the merge kernel's LDS).
#define RS3_MAX_SPLITS_X_HEADS 256
__host__ __device__ __forceinline__ int split_tiles(int ntiles, int S) {
  int tps = (ntiles + S - 1) / S;
  return tps < MIN_TILES_PER_SPLIT ? MIN_TILES_PER_SPLIT : tps;
}
__host__ __device__ __forceinline__ int active_splits(int ntiles, int S) {
  const int tps = split_tiles(ntiles, S);
  return (ntiles + tps - 1) / tps;
}

// Workgroup barrier for LDS traffic only: waits for this wave's LDS
// operations, not for its outstanding global loads (which the fence of
// __syncthreads would drain).
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

__device__ __forceinline__ void set_err(int32_t* hdr, int code) {
  atomicCAS(&hdr[HDR_ERR], 0, code);
}

}  // namespace rs3

// ---- kernel argument blocks (passed by value) ------------------------------
struct Rs3SelectArgs {
  const uint8_t* masks;   // [n_obj][m*s][n*s]
  int32_t* track;         // [n_obj][RS3_TRACK_WORDS]
  const double* e;        // [n_x][mn] energies
  const unsigned long long* erange;   // [n_x][ceil(mn/64)][2] min/max energy bits per 64 cells
  int32_t* sel_idx;       // [n_groups][mn]
  int32_t* sel_count;     // [n_groups]
  uint8_t* prior_out;     // [n_groups][mn] or null
  uint64_t* prior_bits;   // [n_groups][64][4] prior rows computed beside the energies, or null
  int m, n, s, n_obj, union_objects, seed_box, r_s, c, x_per_obj;
  int k[RS3_MAX_OBJ];
};

// Query projection of every grid row inside the energy launch (rs3_frame
// with a single 64-wide attention head at d_model 256): the launch reads
// every row of X anyway, and the attention then gathers projected rows.
//   Qall[xi][i] = bf16(qscale * x_i W_q)  (W_q the attention's query weights)
struct Rs3QProjArgs {
  const rs3::bf16_t* WqT;   // [64][256] (W_q^T of the one head)
  rs3::bf16_t* Qall;        // [n_x][mn][64]
  float qscale;             // log2(e) / sqrt(d_h)
};

struct Rs3CommitArgs {
  rs3::BankDev* banks[RS3_MAX_OBJ];
  const uint8_t* masks;   // [n_obj][m*s][n*s]
  const void* Kmem;       // [n_obj][mn][d_kv]
  const void* Vmem;
  int64_t kv_stride;      // elements between objects
  int32_t* kept_count;    // [n_obj] or null
  const void* WkT;        // [D][d_kv] (projected mode)
  const void* WvT;
  int m, n, s, t, pin, fall_min, fall_max, n_obj, absorb;
  int from_ring;          // append: rows are already in the raw ring (bank import)
  uint64_t parity;        // bit o: current copy of bank o's frame table and frame count
  int rows_per_wg;        // commit: kept rows appended per work-group (a multiple of 64)
  const float* rope;      // [rope_mn][d_h/2][2] rotary table for the keys, or null
  int rope_mn;
};

struct Rs3ReadoutArgs {
  rs3::BankDev* banks[RS3_MAX_OBJ];
  const void* X;
  int64_t x_stride;       // elements between objects' grids (0 = shared)
  void* Y;
  int64_t y_stride;
  const int32_t* sel_idx;
  const int32_t* sel_count;
  int sel_stride;         // elements between objects' lists (0 = shared)
  const void* WqT;        // [D][C]
  const void* WoT;        // [C][D]
  void* Q;                // [n_obj][max_sel][D] bf16 workspace
  void* Opart;            // [n_obj][S][max_sel][D] bf16 workspace
  float* ML;              // [n_obj][S][max_sel][H][2] workspace
  float qscale;           // log2(e) / sqrt(d_h)
  int mn, C, H, d_h, D, n_obj, max_sel, S, n_qt, y_fp32;
  const float* rope;      // [mn][d_h/2][2] rotary table for the queries, or null
  const void* Qall;       // queries of every cell projected by the energy launch (rs3_frame), or null:
  int64_t qall_stride;    //   [n_x][mn][64] bf16, elements between objects' grids (0 = shared)
  int stream_parts;       // 1: the split partials are stored non-temporally (the readout's merge
                          //   reads them once, non-temporally); 0: plain stores (stack, attend)
};

// The attention-side pointers of every object's bank, handed to the
// attention launch by value: its first loads (header word, tile entries, key
// and value tiles) then need no read of the bank descriptor first.
struct Rs3AttnBanks {
  const int32_t* hdr[RS3_MAX_OBJ];
  const rs3::TileEnt* tiles[RS3_MAX_OBJ];
  const void* kh[RS3_MAX_OBJ];
  const void* vh[RS3_MAX_OBJ];
  int32_t ntcap[RS3_MAX_OBJ];   // entries of the tile list (n_tiles_cap)
};

// Bare attention core: the tensors of rs3_attend laid out as a one-frame
// bank in the caller's workspace.
struct AttendPrepArgs {
  const rs3::bf16_t* Q;        // [n_q][H][d_h]
  const rs3::bf16_t* K;        // [n_kv][H][d_h]
  const rs3::bf16_t* V;
  rs3::bf16_t* Qs;             // [n_q][D], Q * log2(e)/sqrt(d_h)
  rs3::bf16_t* Khat;           // [ntile][H][64][d_h]
  rs3::bf16_t* Vhat;           // [ntile][H][d_h][64] (slot order)
  rs3::TileEnt* tiles;         // [ntile]
  rs3::BankDev* desc;
  int32_t* hdr;           // [HDR_WORDS]
  int32_t* count;         // selected-query count read by the attention
  int64_t n_kv;
  float qscale;
  int n_q, H, d_h, ntile;
};

// Arguments of the memory-attention stack's launches (stack.hip); every
// launch reads the fields it needs.  n = the device count, clamped into
// [0, M]; row-indexed buffers hold M rows.
struct StkArgs {
  const int32_t* count;       // kept rows (device)
  int32_t* err_hdr;           // header of the bank whose error word takes the reports
  const int32_t* sel;         // kept cells (gather, scatter)
  int M, mn;
  const void* X;              // bf16 grid [mn][256]
  void* Y;                    // bf16 or fp32 grid [mn][256]
  int y_f32;
  float* Z;                   // [M][256] residual stream
  float* Zp;                  // [M][256] stream after the cross-attention
  float* P;                   // [NC][M][256] MLP partials, one per 256 hidden units
  int NC, F;
  rs3::bf16_t* A1;            // [M][256] LN1 rows, the QKV product's input
  const float* ln_g;          // the norm of k_stk_rows (LN1 of the layer it feeds)
  const float* ln_b;
  const float* ln2_g;
  const float* ln2_b;
  const float* ln3_g;
  const float* ln3_b;
  rs3::bf16_t* Qs;            // [M][256] self-attention queries, then its merged output
  rs3::bf16_t* Qc;            // [M][64] cross-attention queries, then its merged output
  // packed weights (MFMA B-operand order, see pack_b)
  const rs3::bf16_t* Wqkv;    // [256][768]
  const rs3::bf16_t* Wos;     // [256][256]
  const rs3::bf16_t* Wqc;     // [256][64]   W_q W_k^T
  const rs3::bf16_t* Wvo;     // [64][256]   W_v W_o
  const rs3::bf16_t* W1;      // [256][F]
  const rs3::bf16_t* W2;      // [F][256]
  float qscale_s, qscale_c;   // log2(e) / sqrt(head width)
  // split merge (k_stk_merge): Opart [S][M][D_att], ML [S][M][H_att][2]
  const rs3::bf16_t* Opart;
  const float* ML;
  int S, H_att, d_att, D_att;
  rs3::bf16_t* mout;          // [M][D_att]
  // the self-attention's one-frame bank
  rs3::bf16_t* Kh;            // [ntile_cap][Hs][64][dhs]
  rs3::bf16_t* Vh;            // [ntile_cap][Hs][dhs][64] (slot order)
  rs3::TileEnt* tiles;        // [ntile_cap]
  rs3::BankDev* desc;
  int32_t* shdr;              // [HDR_WORDS]
  int Hs, dhs, ntile_cap, write_bank;
};

// Launchers (all enqueue on `st` and return the launch status).
// qp (optional, bf16 grids of 256 channels only): the launch also projects
// every row (Rs3QProjArgs).
hipError_t rs3_launch_energy(const void* X, int64_t x_stride, int n_x, int mn, int C, int dtype,
                             double* e, unsigned long long* range, hipStream_t st,
                             const Rs3QProjArgs* qp = nullptr);
hipError_t rs3_launch_select(const Rs3SelectArgs& a, int n_groups, hipStream_t st);
// Grids for which the prior runs beside the energies (one wave per group).
bool rs3_select_prior_beside(int m, int n, int s);
// Energies and the one-wave priors (written to a.prior_bits) in one launch.
hipError_t rs3_launch_energy_prior(const void* X, int64_t x_stride, int n_x, int mn, int C, int dtype, double* e,
                                   unsigned long long* range, const Rs3SelectArgs& a, int n_groups, hipStream_t st,
                                   const Rs3QProjArgs* qp = nullptr);
hipError_t rs3_launch_commit(const Rs3CommitArgs& a, int dtype, int d_kv, int D, int H, int d_h,
                             hipStream_t st);
// merge = false leaves the split merge of the bf16 path to the caller (the
// fused merge + commit launch); returns whether a merge is pending in *pending.
hipError_t rs3_launch_readout(const Rs3ReadoutArgs& a, const Rs3AttnBanks& ab, int dtype, hipStream_t st,
                              bool merge = true, bool* pending = nullptr);
// The readout's split merge and a commit in one launch (bf16 layers).
hipError_t rs3_launch_merge_commit(const Rs3ReadoutArgs& ra, const Rs3CommitArgs& ca, int d_kv, hipStream_t st);
// The readout's split merge, output projection and residual scatter alone.
hipError_t rs3_launch_combine(const Rs3ReadoutArgs& a, hipStream_t st);
hipError_t rs3_fused_setup();
// Split-KV attention only; project: the queries are projected from X[sel]
// inside the kernel (heads of width <= 64), else read from a.Q.
hipError_t rs3_launch_attn(const Rs3ReadoutArgs& a, const Rs3AttnBanks& ab, hipStream_t st, bool project);
// Whether the attention of this launch projects its queries inside (then a
// frame may hand it the energy launch's projection of every cell instead).
bool rs3_attn_projects(const Rs3ReadoutArgs& a);
hipError_t rs3_launch_attend_prep(const AttendPrepArgs& p, hipStream_t st);
hipError_t rs3_launch_attend_merge(const Rs3ReadoutArgs& a, int SA, float* O, hipStream_t st);
hipError_t rs3_launch_attend_f32(const float* Q, const float* K, const float* V, int n_q, int64_t n_kv, int H,
                                 int d_h, float qscale, float* O, hipStream_t st);
// Projects the raw ring rows [hdr PSTART, + PLEN) of bank 0 of `a` into its
// attention tiles (a.from_ring = 1), or, with rebuild = 1, rebuilds the
// resident tile list and key count from the frame table.
hipError_t rs3_launch_bank_restore(const Rs3CommitArgs& a, int dtype, int d_kv, int rebuild, hipStream_t st);
hipError_t rs3_readout_setup();
// The fixed write keep-set (see rs3_write_keepset); D is already clamped.
hipError_t rs3_launch_write_keepset(const uint8_t* seed, int n_obj, int m, int n, int s, int D, int fall_min,
                                    int fall_max, int n_copies, uint8_t* keep, int32_t* counts, hipStream_t st);
// Closure of decoded masks and the palette (see rs3_close_masks).
size_t rs3_post_workspace_bytes(int n_obj, int H, int W);
hipError_t rs3_launch_close_masks(int n_obj, int H, int W, const void* logits, int dtype, int k, uint8_t* closed,
                                  uint8_t* palette, void* ws, hipStream_t st);
// Fills the axial rotary table (see rs3_layer_set_rope_axial).
hipError_t rs3_launch_rope_axial(float* table, int m, int n, int d_h, double theta, hipStream_t st);
// While profiling is on: the next free pair of the event pool for a launch
// of kernel ID (false when profiling is off or the pool is full).
bool rs3_prof_events(int id, hipEvent_t* start, hipEvent_t* stop);

// Launch a kernel; while profiling is on, through hipExtLaunchKernelGGL with
// a start and a stop event, which the runtime stamps with the kernel's own
// begin and end (the dispatch gap before it is not counted).  ST is the
// stream, also passed in the launch arguments.
#define RS3_LAUNCH(ID, ST, K, G, B, SHM, S, ...)                                   \
  do {                                                                            \
    hipEvent_t rs3_e0_, rs3_e1_;                                                  \
    if (rs3_prof_events((ID), &rs3_e0_, &rs3_e1_))                                \
      hipExtLaunchKernelGGL(K, G, B, SHM, S, rs3_e0_, rs3_e1_, 0u, __VA_ARGS__);  \
    else                                                                          \
      hipLaunchKernelGGL(K, G, B, SHM, S, __VA_ARGS__);                           \
  } while (0)
// The stack's launches (stack.hip): k_stk_rows (mode 0 gather + LN1,
// 1 partial sum + LN1, 2 partial sum + scatter), the QKV product, the
// post-self-attention block, the MLP chunks, the split merge and the
// X -> Y copy before the scatter.
hipError_t rs3_launch_stack_rows(const StkArgs& p, int mode, hipStream_t st);
hipError_t rs3_launch_stack_qkv(const StkArgs& p, hipStream_t st);
hipError_t rs3_launch_stack_post_sa(const StkArgs& p, hipStream_t st);
hipError_t rs3_launch_stack_mlp(const StkArgs& p, hipStream_t st);
hipError_t rs3_launch_stack_merge(const StkArgs& p, hipStream_t st);
hipError_t rs3_launch_stack_copy(const void* X, void* Y, int64_t elems, int y_f32, hipStream_t st);
hipError_t rs3_stack_setup();
hipError_t rs3_select_setup();
hipError_t rs3_commit_setup();
