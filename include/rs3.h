/*
 * rs3.h -- C ABI of the read-sparse memory readout and store-sparse commit
 * (RS^3-Prune, Sec. 3.1 and Sec. 3.2) on AMD Instinct MI355X (gfx950).
 *
 * Three calls make up one frame of the method's hot path:
 *   rs3_select_queries : per-object spatial prior from the previous masks
 *                        (Eqs. 1, 2, 5) and the energy top-k keep-set inside
 *                        it (Eq. 4)  -> ascending selected-query lists;
 *   rs3_readout        : gather the selected query tokens, cross-attend them
 *                        to the object's memory bank (Eq. 6) and scatter the
 *                        result back; unselected rows pass through unchanged;
 *   rs3_commit         : compact the memory-encoder tokens inside the mask
 *                        (Eq. 8) into the object's ring memory bank.
 *
 * Conventions (every call):
 *  - Tensor pointers are DEVICE pointers unless marked [host].  The caller
 *    owns every tensor it passes and the stream; the library owns the memory
 *    behind its handles (weights copy, banks, tracker state).
 *  - Work is enqueued asynchronously on `stream` (a hipStream_t; NULL = the
 *    null stream).  Only the *_export, *_import and rs3_bank_error calls
 *    synchronise.  Nothing is allocated inside select/readout/commit.
 *  - Grids are m x n token cells, cell index i = y*n + x.  Per-object masks
 *    are uint8 [(m*s) x (n*s)] pixel grids; cell (y, x) samples pixel
 *    (y*s, x*s).  Any nonzero byte counts as set.
 *  - Float tensors are bf16 (stored as 16-bit patterns) or fp32, one dtype per
 *    layer: query tokens X, outputs Y, weights and the bank share it.  All
 *    accumulation is fp32; token energies are fp64.
 *  - Errors are return codes, never exceptions.  Problems visible on the host
 *    (null pointers, bad sizes, dtype mismatches, pin misuse, workspace too
 *    small) return RS3_E_INVALID before any device work and change no state.
 *    Problems only the device can see (a bank frame that does not fit, a
 *    selection list that is out of range or not ascending) set a sticky error
 *    word in the affected bank; the failing operation leaves that bank
 *    unchanged (commit) or skips the offending rows (readout).  The word keeps
 *    the first error; rs3_bank_error reads it.  HIP failures map to
 *    RS3_E_DEVICE (launch/copy) or RS3_E_OOM (allocation).
 *  - Token tensors (X, Y, the memory tokens, the rs3_attend operands) and
 *    workspaces are moved in 16-byte vectors: their base pointers must be
 *    16-byte aligned and per-object strides whole multiples of 16 bytes, else
 *    RS3_E_INVALID (torch allocations and contiguous slices of whole grids
 *    meet this).
 *  - A handle must not be used from two streams at once.
 */
#ifndef RS3_H
#define RS3_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  RS3_OK = 0,
  RS3_E_INVALID = 1,
  RS3_E_CAPACITY = 2,
  RS3_E_DEVICE = 3,
  RS3_E_OOM = 4
} rs3_status;

typedef enum { RS3_F32 = 0, RS3_BF16 = 1 } rs3_dtype;

/* Token grid m x n; masks are (m*s) x (n*s) pixels (s = encoder stride). */
typedef struct {
  int32_t m, n, s;
} rs3_grid;

/* Prior parameters (Sec. 3.1, Algorithm 1 hyper-parameters):
 *   r_s            dilation radius in cells of the previous-mask prior (Eq. 2)
 *   c              cap on the extra radius of the lost-object box fallback (Eq. 5)
 *   seed_box       1: a non-empty mask contributes its dilated filled bounding
 *                  box (the frame-0 seed prior, Eq. 1); 0: the dilated mask
 *   union_objects  1: one keep-set for the union of all objects' priors (as in
 *                  the paper); 0: one keep-set per object */
typedef struct {
  int32_t r_s, c, seed_box, union_objects;
} rs3_select_params;

#define RS3_MAX_OBJ 64          /* objects per call */
#define RS3_MAX_MN 32768        /* token cells per grid */
#define RS3_TRACK_WORDS 6       /* y0, x0, y1, x1, streak, has_box (pixels) */
#define RS3_BANK_HDR_WORDS 8    /* exported header: n_frames, pin_end, err, ... */

typedef struct rs3_track rs3_track; /* per-object tracker state, device resident */
typedef struct rs3_layer rs3_layer; /* cross-attention weights and shape */
typedef struct rs3_bank rs3_bank;   /* one object's ring memory bank */

const char* rs3_status_str(rs3_status s);

/* ---- tracker state (Sec. 3.1, streak-counted box fallback, Eq. 5) --------
 * Holds, per object, the most recent non-empty box (pixel coordinates,
 * inclusive), the count of consecutive empty frames and whether a box was
 * ever seen.  Created zeroed (no box).  export/import copy
 * int32 [n_obj][RS3_TRACK_WORDS] host arrays and synchronise the device
 * (checkpoint and resume).  import accepts only states the tracker update
 * reaches, else RS3_E_INVALID with the state unchanged: has_box 0 or 1;
 * streak in [0, 2^30]; with has_box = 1, 0 <= y0 <= y1 < 2^30 and
 * 0 <= x0 <= x1 < 2^30; with has_box = 0, a zero box.  (The tracker does not
 * know the grid: a box past the pixel grid of a later select is clipped to
 * the grid when the prior is drawn.) */
rs3_status rs3_track_create(int32_t n_obj, rs3_track** out);
void rs3_track_destroy(rs3_track* t);
rs3_status rs3_track_export(const rs3_track* t, int32_t* state /*[host]*/);
rs3_status rs3_track_import(rs3_track* t, const int32_t* state /*[host]*/);

/* ---- layer (one cross-attention of the memory readout, Eq. 6) -------------
 * C: query token width; H heads of width d_h with D = H*d_h = C; d_kv: width
 * of the bank's raw key/value tokens.  Weights are [host] row-major arrays in
 * dtype `dt`: Wq [C][D], Wk [d_kv][D], Wv [d_kv][D], Wo [D][C]; the library
 * copies them (into its own device layouts).
 * absorb = 0 (projected): banks store K^ = K W_k and V^ = V W_v (width D) and
 *   the attention runs per head at width d_h.  d_h must be 32, 64, 128 or
 *   256 for bf16 (at most 256 for fp32).
 * absorb = 1 (H = 1 only): the attention runs directly on the raw bank rows
 *   (width d_kv) with q' = x W_q W_k^T and y = x + o' W_v W_o, the same
 *   function with the projections re-associated; the products W_q W_k^T and
 *   W_v W_o are formed once here in fp64 and rounded to `dt`.  bf16 needs
 *   d_kv in {64, 128, 256}.
 * C <= 1024 (a multiple of 64 for bf16); d_kv <= 256, a multiple of 16. */
rs3_status rs3_layer_create(int32_t C, int32_t H, int32_t d_kv, rs3_dtype dt, int32_t absorb,
                            const void* Wq, const void* Wk, const void* Wv,
                            const void* Wo, rs3_layer** out);
void rs3_layer_destroy(rs3_layer* L);

/* ---- rotary positions on the gathered subset (Sec. 3.1, Eq. 7) ------------
 * Attaches a rotary table to a projected layer (absorb = 0) whose attention
 * then turns each head's channel pairs (2p, 2p+1), read as the complex number
 * x_2p + i x_2p+1, by the table row of the token's grid cell: a selected query
 * by the row of the cell it was gathered from (f~ = f[K_r], not the first
 * |K_r| rows), a bank key by the row of the cell it was kept from.  Values
 * are not turned.  The heads share the table, which has d_h/2 columns.  The
 * grid of every later rs3_readout and rs3_commit with this layer must be
 * m x n (else RS3_E_INVALID).  Keys are turned once, when they are committed
 * (or restored by rs3_bank_import), so the table must be set before the
 * first bank is created from the layer: with a bank alive the call returns
 * RS3_E_INVALID and changes nothing.  Both calls are synchronous.
 *
 * rs3_layer_set_rope: table [host] fp32 [m*n][d_h/2][2] holding (cos, sin)
 *   of each factor, copied to the device; table = NULL with m = n = 0
 *   removes the table.
 * rs3_layer_set_rope_axial: builds the axial two-dimensional table on the
 *   device: for p < d_h/4 the angle of cell (row, col) = (i / n, i % n) is
 *   col * theta^(-4p/d_h), for the other d_h/4 factors it is
 *   row * theta^(-4(p - d_h/4)/d_h) (computed in fp64, stored as fp32).
 *   Requires theta > 1 and d_h divisible by 4.
 * Both require 1 <= m*n <= RS3_MAX_MN and an even d_h. */
rs3_status rs3_layer_set_rope(rs3_layer* L, int32_t m, int32_t n, const float* table /*[host]*/);
rs3_status rs3_layer_set_rope_axial(rs3_layer* L, int32_t m, int32_t n, double theta);

/* ---- bank (Sec. 3.2; placement rule below) --------------------------------
 * A ring of `cap` token rows holding at most `f_max` frames, of which the
 * first commits (at most n_pin, all before any unpinned commit) may be pinned.
 * Pinned frames are laid out from row 0 and never evicted.  An unpinned frame
 * of L kept tokens: (1) L > cap - pin_end -> RS3_E_CAPACITY, bank unchanged;
 * (2) while f_max frames are resident evict the oldest unpinned frame;
 * (3) start = end of the newest unpinned frame (pin_end if none), or pin_end
 * if start + L > cap; (4) evict unpinned frames oldest first until none
 * overlaps [start, start+L); (5) store rows and record (start, L, t, pinned).
 * Zero-length frames are recorded.  The bank stores the raw K/V rows, the
 * kept cell index (`pos`) per row, and the rows projected by W_k / W_v of
 * the layer it was created for (which must outlive it).
 * Requires 0 <= n_pin < f_max <= 256, 1 <= cap <= 2^26. */
rs3_status rs3_bank_create(const rs3_layer* L, int32_t cap, int32_t f_max,
                           int32_t n_pin, rs3_bank** out);
void rs3_bank_destroy(rs3_bank* b);

/* Bank snapshot in key order (pinned frames, then unpinned oldest->newest).
 * hdr [host, RS3_BANK_HDR_WORDS]: n_frames, pin_end, err, n_keys, rest 0.
 * frames [host, f_max][4]: start, length, t, pinned (first n_frames rows).
 * K, V [host, cap][d_kv] (dtype bytes) and pos [host, cap]: resident rows
 * concatenated in key order (first n_keys rows); any may be NULL.
 * Synchronises the device. */
rs3_status rs3_bank_export(const rs3_bank* b, int32_t* hdr, int32_t* frames,
                           void* K, void* V, int32_t* pos);
/* Restore a bank from a snapshot in the rs3_bank_export format (checkpoint
 * and resume).  The bank must have been created for a layer of the same
 * shape and dtype, with at least the snapshot's capacity, frame count and
 * pinned frames.  hdr uses words n_frames, pin_end, err and n_keys; frames,
 * K, V and pos are as exported (rows concatenated in key order).  The
 * snapshot must be a state the placement rule reaches: pinned frames first,
 * packed from row 0 and adding up to pin_end, unpinned frames inside
 * [pin_end, cap), non-empty frames disjoint, lengths adding up to n_keys;
 * otherwise RS3_E_INVALID and the bank is unchanged.  The attention tiles
 * are recomputed from the raw rows with this bank's layer, and the host-side
 * pin bookkeeping follows the snapshot.  Synchronises the device. */
rs3_status rs3_bank_import(rs3_bank* b, const int32_t* hdr /*[host]*/, const int32_t* frames /*[host]*/,
                           const void* K /*[host]*/, const void* V /*[host]*/, const int32_t* pos /*[host]*/);

/* Read (and optionally clear) the sticky device error word.  Synchronises. */
rs3_status rs3_bank_error(rs3_bank* b, int32_t* err /*[host]*/, int32_t clear);

/* ---- select_queries (Sec. 3.1: Eqs. 1, 2, 4, 5; Algorithm 1) --------------
 * masks  : uint8 [n_obj][m*s][n*s], each object's previous-frame mask
 * tr     : tracker state for n_obj objects, updated in place (box, streak)
 * X      : [n_x][m*n][C] query tokens in `dt`; x_obj_stride (elements) = 0
 *          when all objects share one grid, else the per-object stride (then
 *          p->union_objects must be 0 or n_obj 1)
 * k      : [host][n_groups] keep budgets floor(rho*mn), computed exactly by
 *          the caller; n_groups = 1 if union_objects else n_obj
 * ws     : device workspace of at least rs3_select_workspace_size() bytes
 * sel_idx: out int32 [n_groups][m*n]; the first sel_count[g] entries of row g
 *          are the kept cells in ascending order: all of the prior P_g if
 *          |P_g| <= k[g], otherwise the k[g] cells of P_g with the largest
 *          energy sum_c x_{i,c}^2 (fp64, channels added in ascending order),
 *          ties to the lower cell index
 * sel_count : out int32 [n_groups]
 * prior_out : optional out uint8 [n_groups][m*n], the prior bitmap P_g */
rs3_status rs3_select_workspace_size(const rs3_grid* g, int32_t n_obj,
                                     int64_t x_obj_stride, size_t* bytes);
rs3_status rs3_select_queries(const rs3_grid* g, int32_t n_obj, const uint8_t* masks,
                              rs3_track* tr, const void* X, int64_t x_obj_stride,
                              int32_t C, rs3_dtype dt, const int32_t* k,
                              const rs3_select_params* p, void* ws, size_t ws_bytes,
                              int32_t* sel_idx, int32_t* sel_count, uint8_t* prior_out,
                              void* stream);

/* ---- readout (Sec. 3.1, Eq. 6 with the residual reading) -------------------
 * For object o with selection list sel (row o of sel_idx, or row 0 when
 * sel_stride == 0) and bank banks[o] of N resident keys:
 *   y_i = x_i + [softmax(q_h K^_h^T / sqrt(d_h)) V^_h]_h W_o,  q = x_i W_q,
 *         for every selected cell i;
 *   y_i = x_i bit for bit for every other cell, and for all cells if N = 0.
 * X      : [n_x][m*n][C] (x_obj_stride as in select)
 * sel_idx/sel_count : as produced by rs3_select_queries; sel_stride = m*n
 *          for per-object lists or 0 for one shared list
 * max_sel: upper bound on every sel_count used (host grid size), <= m*n
 * n_splits: key splits per query tile (0 = automatic); n_splits*H <= 256
 * Y      : [n_obj][m*n][C] with stride y_obj_stride (elements); may equal X
 *          (in place) only when n_obj == 1 or X is per object with the same
 *          stride.  y_fp32 = 1 writes Y as fp32 for diagnostics (never in
 *          place), otherwise Y has the layer dtype.
 * ws     : device workspace of at least rs3_readout_workspace_size() bytes (a
 *          size queried for max_sel also serves every smaller max_sel) */
rs3_status rs3_readout_workspace_size(const rs3_layer* L, int32_t n_obj, int32_t max_sel,
                                      int32_t n_splits, size_t* bytes);
rs3_status rs3_readout(const rs3_layer* L, const rs3_grid* g, int32_t n_obj,
                       const void* X, int64_t x_obj_stride, rs3_bank* const* banks /*[host]*/,
                       const int32_t* sel_idx, const int32_t* sel_count, int32_t sel_stride,
                       int32_t max_sel, int32_t n_splits, void* Y, int64_t y_obj_stride,
                       int32_t y_fp32, void* ws, size_t ws_bytes, void* stream);

/* ---- readout for callers that cannot allocate ------------------------------
 * For code that may not call hipMalloc or take a workspace (work recorded
 * under HIP graph capture, fixed serving loops, hosts that forbid device
 * allocation): rs3_readout with the same arguments and results, minus
 * ws/ws_bytes.  The split partials and projected queries go to a fixed
 * device array of RS3_NOALLOC_SCRATCH_BYTES inside the library, one copy per
 * GPU, held until the process ends; the call allocates nothing.
 * n_splits = 0 takes the automatic key-split count, reduced until the
 * partials fit the array (the results then differ from rs3_readout's only in
 * rounding); a call whose layout does not fit even with one split (or with
 * the n_splits given) returns RS3_E_INVALID and launches nothing.  The bf16
 * partials of one call need about
 *   n_obj*max_sel*Da*2 + S*n_obj*max_sel*(Da*2 + H*8) bytes
 * for S key splits, Da the attention width (D, or d_kv in the absorbed form)
 * and H its heads.  E.g. one object on a 64x64 grid with one head of 256 fits
 * every max_sel up to 4096, with at most 6 key splits projected and 29
 * absorbed.  fp32 layers use no scratch.
 * Every call on one GPU shares that GPU's array, and no call clears it
 * (nothing in it must start at zero): calls that overlap in time on one GPU
 * (two streams, or two host threads) race and give undefined results. */
#define RS3_NOALLOC_SCRATCH_BYTES (16u << 20)
rs3_status rs3_readout_noalloc(const rs3_layer* L, const rs3_grid* g, int32_t n_obj, const void* X,
                               int64_t x_obj_stride, rs3_bank* const* banks /*[host]*/, const int32_t* sel_idx,
                               const int32_t* sel_count, int32_t sel_stride, int32_t max_sel, int32_t n_splits,
                               void* Y, int64_t y_obj_stride, int32_t y_fp32, void* stream);

/* ---- commit (Sec. 3.2, Eq. 8 and the sparse write of Algorithm 1) ----------
 * For each object o: kept = ascending cells set in masks[o] (sampled at
 * stride s); if kept_count < fall_min or > fall_max all m*n cells are kept
 * (the dense fall-through; pass 0 and m*n to disable).  The kept rows of
 * Kmem[o], Vmem[o] ([m*n][d_kv] each, object stride kv_obj_stride elements)
 * are appended to banks[o] as frame t by the placement rule of
 * rs3_bank_create, together with their projections by W_k and W_v.
 * pin = 1 marks a pinned frame (host-checked: only before any unpinned commit
 * and at most n_pin times per bank).  kept_count: optional device out
 * int32 [n_obj]. */
rs3_status rs3_commit(rs3_bank* const* banks /*[host]*/, int32_t n_obj, const rs3_grid* g,
                      const void* Kmem, const void* Vmem, int64_t kv_obj_stride,
                      const uint8_t* masks, int32_t t, int32_t pin, int32_t fall_min,
                      int32_t fall_max, int32_t* kept_count, void* stream);

/* ---- readout and commit of one frame in one call ---------------------------
 * Exactly rs3_readout(...) followed by rs3_commit(...) on the same stream
 * and banks (arguments as there; the commit's banks are the readout's), with
 * the readout's split merge and the commit in one launch for bf16 layers:
 * the merge reads the attention partials, X and W_o and writes Y, the commit
 * writes the banks, so their work-groups run side by side (Algorithm 1 writes
 * a frame to memory right after its readout).  Calls whose two parts come to
 * more than 1,024 work-groups (many objects) run them as two launches, which
 * fit the chip better at that size.  Both argument sets are checked
 * before any device work; either failing returns RS3_E_INVALID with no state
 * changed.  When the selection list and the commit both find device errors,
 * the bank's sticky word keeps whichever is recorded first. */
rs3_status rs3_readout_commit(const rs3_layer* L, const rs3_grid* g, int32_t n_obj, const void* X,
                              int64_t x_obj_stride, rs3_bank* const* banks /*[host]*/, const int32_t* sel_idx,
                              const int32_t* sel_count, int32_t sel_stride, int32_t max_sel, int32_t n_splits,
                              void* Y, int64_t y_obj_stride, int32_t y_fp32, void* ws, size_t ws_bytes,
                              const void* Kmem, const void* Vmem, int64_t kv_obj_stride, const uint8_t* masks,
                              int32_t t, int32_t pin, int32_t fall_min, int32_t fall_max, int32_t* kept_count,
                              void* stream);

/* ---- one frame of the path in one call (Algorithm 1's per-frame body) -------
 * rs3_select_queries, then rs3_readout_commit, on the same stream, for one
 * frame of every object: the previous masks select the queries (Eqs. 1, 2,
 * 4, 5), the selected queries read the banks (Eq. 6), and the frame's memory
 * tokens are committed (Eq. 8).  The results are those of the separate calls
 * with the same arguments (bit for bit).  C and the dtype are the layer's;
 * the selection lists are per group with sel_stride 0 (one union group) or
 * m*n (one group per object), as in rs3_select_queries.
 * Because one call sees the whole frame, it may fuse across the calls: with
 * one attention head of width 64 at d_model 256 (the absorbed form, d_kv =
 * 64, no rotary table), the energy launch also projects the query of every
 * cell (it reads every row of X anyway) and the attention gathers projected
 * rows; the projection then runs for all m*n cells rather than the selected
 * ones (2*m*n*256*64 flops per grid).
 * ws: device workspace of at least rs3_frame_workspace_size() bytes (a size
 * queried for max_sel also serves every smaller max_sel).  Errors as in the
 * separate calls; every argument is checked before any device work. */
typedef struct {
  /* selection (rs3_select_queries) */
  const uint8_t* read_masks;   /* [n_obj][m*s][n*s] masks of the previous frame */
  const void* X;               /* [n_x][m*n][C] query tokens */
  int64_t x_obj_stride;        /* 0 = one grid shared by all objects */
  const int32_t* k;            /* [host][n_groups] keep budgets */
  rs3_select_params params;
  int32_t* sel_idx;            /* out [n_groups][m*n] */
  int32_t* sel_count;          /* out [n_groups] */
  uint8_t* prior_out;          /* optional out [n_groups][m*n] */
  /* readout (rs3_readout) */
  int32_t max_sel, n_splits;
  void* Y;                     /* may equal X as in rs3_readout */
  int64_t y_obj_stride;
  int32_t y_fp32;
  /* commit (rs3_commit) */
  const void* Kmem;
  const void* Vmem;
  int64_t kv_obj_stride;
  const uint8_t* commit_masks; /* [n_obj][m*s][n*s] masks of this frame */
  int32_t t, pin, fall_min, fall_max;
  int32_t* kept_count;         /* optional out [n_obj] */
} rs3_frame_io;
rs3_status rs3_frame_workspace_size(const rs3_layer* L, const rs3_grid* g, int32_t n_obj, int64_t x_obj_stride,
                                    int32_t max_sel, int32_t n_splits, size_t* bytes);
rs3_status rs3_frame(const rs3_layer* L, const rs3_grid* g, int32_t n_obj, rs3_track* tr,
                     rs3_bank* const* banks /*[host]*/, const rs3_frame_io* io /*[host]*/, void* ws,
                     size_t ws_bytes, void* stream);

/* ---- the paper's fixed write keep-set (Sec. 3.2, Eq. 8) -------------------
 * K_w = union over the n_obj objects of dilate_{D_w}(down_s(seed_masks[o])),
 * where seed_masks[o] is object o's mask at its first frame ([n_obj][m*s][n*s]
 * u8, nonzero = set; cell (y, x) samples pixel (y*s, x*s)) and the dilation is
 * the Chebyshev radius D_w in grid cells.  If the undilated footprint (the
 * union of the down-sampled seeds) has fewer than fall_min or more than
 * fall_max cells, K_w is every cell (the dense fall-through; 0 and m*n turn
 * it off).  K_w is computed once and passed unchanged to every later
 * rs3_commit of the sequence (with the grid {m, n, 1}: the keep-set is at
 * grid resolution), so every stored frame holds |K_w| rows: a constant
 * per-frame stride, and fixed ring slots when the bank holds the pinned rows
 * plus a multiple of |K_w|.
 * keep   : device out u8 [n_copies][m*n], 1 = kept; the keep-set is written
 *          n_copies times so that it serves as the mask of n_copies objects.
 * counts : optional device out int32 [2]: footprint cells, |K_w|.
 * Asynchronous on `stream`, allocates nothing.  Requires a valid grid,
 * 1 <= n_obj <= RS3_MAX_OBJ, 1 <= n_copies <= RS3_MAX_OBJ, D_w >= 0 (radii
 * beyond the grid act as max(m, n)). */
rs3_status rs3_write_keepset(const rs3_grid* g, int32_t n_obj, const uint8_t* seed_masks, int32_t D_w,
                             int32_t fall_min, int32_t fall_max, int32_t n_copies, uint8_t* keep,
                             int32_t* counts, void* stream);

/* ---- closure of the decoded masks and the palette (Sec. 3.3) ----------------
 * The steps after the mask decoder in Algorithm 1.  For each object o its
 * binary mask is logits[o] > 0 at decoder resolution H x W; it is closed
 * with a k x k square (k odd, 9 in the paper): a dilation for which pixels
 * outside the image are unset, then an erosion for which they are set, so
 * the closing never removes a pixel.  The palette is, per pixel, 1 + the
 * object with the largest logit among the objects whose closed mask covers
 * the pixel (the lowest index on ties), or 0 where none does.  The closed
 * masks are what the next frame's tracker update reads: with H = m*s and
 * W = n*s they are the `masks` argument of rs3_select_queries.
 * logits  : device [n_obj][H][W] in `dt` (bf16 or fp32).
 * closed  : optional device out u8 [n_obj][H][W] (1 = set).
 * palette : optional device out u8 [H][W].
 * ws      : device workspace of at least rs3_close_workspace_size() bytes.
 * Asynchronous on `stream`, allocates nothing.  Requires 1 <= n_obj <=
 * RS3_MAX_OBJ, 1 <= H <= 16384, 1 <= W <= 4096, k odd in [1, 15]. */
rs3_status rs3_close_workspace_size(int32_t n_obj, int32_t H, int32_t W, size_t* bytes);
rs3_status rs3_close_masks(int32_t n_obj, int32_t H, int32_t W, const void* logits, rs3_dtype dt, int32_t k,
                           uint8_t* closed, uint8_t* palette, void* ws, size_t ws_bytes, void* stream);

/* ---- bare attention core (Sec. 3.1, Eq. 6 without the projections) ---------
 * O_h = softmax(Q_h K_h^T / sqrt(d_h)) V_h for every head h on tensors that
 * are already projected: Qh [n_q][H][d_h], Kh and Vh [n_kv][H][d_h] in `dt`,
 * O [n_q][H][d_h] fp32 (all device).  n_kv = 0 gives O = 0.  This entry
 * exists to measure and check the attention kernel on its own: in bf16 the
 * keys and values are laid out as a one-frame bank in `ws` and the readout's
 * split-KV attention kernel runs on it unchanged (d_h in {32, 64, 128, 256},
 * H*d_h <= 1024, n_splits*H <= 256, n_splits 0 = automatic); in fp32 a direct
 * kernel runs (d_h <= 256, no workspace).  n_q <= RS3_MAX_MN, n_kv <= 2^26.
 * ws: at least rs3_attend_workspace_size() bytes (bf16; may be NULL for fp32). */
rs3_status rs3_attend_workspace_size(int32_t n_q, int32_t n_kv, int32_t H, int32_t d_h, rs3_dtype dt,
                                     int32_t n_splits, size_t* bytes);
rs3_status rs3_attend(const void* Qh, const void* Kh, const void* Vh, int32_t n_q, int32_t n_kv,
                      int32_t H, int32_t d_h, rs3_dtype dt, int32_t n_splits, float* O, void* ws,
                      size_t ws_bytes, void* stream);

/* ---- the L-layer memory-attention stack on the kept queries -----------------
 * Sec. 3.1 ("Sparse memory attention"): the memory module of the VOS models
 * consists of L layers, each with a self-attention and a cross-attention,
 * and the sparse readout applies at the input of every layer, so that each
 * runs on the kept queries only.  The paper gives no
 * layer, so the layer is this pre-norm residual one, in the shape of
 * SAM2-class memory attention (z the fp32 residual stream of a kept row):
 *   z += SA(LN1(z))    self-attention among the kept rows: H_s heads of
 *                      width C/H_s, q, k, v = a W_qs, a W_ks, a W_vs, logits
 *                      scaled by 1/sqrt(C/H_s), output o W_os
 *   z += CA(LN2(z))    the readout of Eq. 6 against the bank: one head,
 *                      q = b W_q, bank keys/values K W_k, V W_v, logits scaled
 *                      by 1/sqrt(C), output o W_o
 *   z += relu(LN3(z) W_1) W_2
 * LN(z) = (z - mean) / sqrt(biased variance + 1e-5) * gain + shift, per row;
 * no biases, no norm after the last layer.  The kept rows are gathered from
 * X once before the first layer and scattered to Y once after the last; every
 * other cell of Y is X's, bit for bit (a dropped row gets a zero update at
 * every layer, so one gather and one scatter equal one per layer).
 *
 * rs3_stack_create: n_layers in [1, 16]; C = 256; H_s in {1, 2, 4, 8};
 * d_kv = 64; F a multiple of 256 up to 8192; dt = RS3_BF16.  layers: host
 * array of n_layers weight sets; matrices row-major bf16 (input dimension
 * first): W_qs, W_ks, W_vs, W_os, W_q, W_o [C][C], W_k, W_v [d_kv][C],
 * W_1 [C][F], W_2 [F][C]; gains and shifts fp32 [C].  Everything is copied
 * to the device at create time (the caller keeps ownership of its arrays);
 * the cross-attention's products W_q W_k^T and W_v W_o are formed there in
 * fp64 and rounded to bf16 once.  Allocates device memory; synchronous.
 *
 * rs3_stack_readout: one object.  X: device bf16 grid [m*n][C]; bank: a bank
 * of a bf16 layer created with absorb = 1, C = 256, d_kv = 64 and no rotary
 * table (its raw rows serve every layer); sel_idx / sel_count / max_sel as in
 * rs3_readout (one list; entries out of range or not ascending, or a count
 * outside [0, max_sel], set the bank's error word, and the rows of such a
 * call are unspecified); n_splits: key splits of the cross-attention, 0 =
 * automatic; Y: device [m*n][C], bf16 or (y_fp32 = 1) fp32, may equal X when
 * bf16.  ws: device workspace of at least rs3_stack_workspace_size(max_sel,
 * n_splits) bytes, 16-byte aligned like X and Y.  Asynchronous on `stream`, allocates
 * nothing; the bank is read only. */
typedef struct rs3_stack rs3_stack;
typedef struct {
  const float* ln1_g;
  const float* ln1_b;
  const void* Wqs;
  const void* Wks;
  const void* Wvs;
  const void* Wos;
  const float* ln2_g;
  const float* ln2_b;
  const void* Wq;
  const void* Wk;
  const void* Wv;
  const void* Wo;
  const float* ln3_g;
  const float* ln3_b;
  const void* W1;
  const void* W2;
} rs3_stack_weights;
rs3_status rs3_stack_create(int32_t n_layers, int32_t C, int32_t H_s, int32_t d_kv, int32_t F, rs3_dtype dt,
                            const rs3_stack_weights* layers /*[host]*/, rs3_stack** out);
void rs3_stack_destroy(rs3_stack* S);
rs3_status rs3_stack_workspace_size(const rs3_stack* S, int32_t max_sel, int32_t n_splits, size_t* bytes);
rs3_status rs3_stack_readout(const rs3_stack* S, const rs3_grid* g, const void* X, rs3_bank* bank,
                             const int32_t* sel_idx, const int32_t* sel_count, int32_t max_sel, int32_t n_splits,
                             void* Y, int32_t y_fp32, void* ws, size_t ws_bytes, void* stream);

/* ---- per-kernel timing (diagnostics) ---------------------------------------
 * rs3_profile_enable(1, max_launches) creates a pool of HIP events; while
 * enabled, each kernel launched by the library is bracketed by two events on
 * its stream (event records only: nothing is allocated or synchronised in the
 * timed calls; launches beyond the pool are not timed and are counted as
 * dropped).  rs3_profile_report waits for the recorded events and fills
 * total_ms[RS3_K_COUNT] and launches[RS3_K_COUNT] (host arrays) with the
 * accumulated kernel durations per kernel id; rs3_profile_reset clears them. */
enum {
  RS3_K_ENERGY = 0,        /* token energies */
  RS3_K_SELECT = 1,        /* prior + top-k + compaction */
  RS3_K_COMMIT = 2,        /* commit: mask compaction, ring placement, tile list, row copy and K/V projection */
  RS3_K_COMMIT_APPEND = 3, /* row copy + K/V projection of a restored bank (rs3_bank_import) */
  RS3_K_COPY = 4,          /* X -> Y copy for out-of-place readout */
  RS3_K_QPROJ = 5,         /* gather + query projection */
  RS3_K_ATTN = 6,          /* split-KV attention */
  RS3_K_COMBINE = 7,       /* split merge + W_o + residual + scatter */
  RS3_K_READOUT_F32 = 8,   /* fp32 readout */
  RS3_K_MERGE_COMMIT = 9,  /* split merge and commit in one launch (rs3_readout_commit, rs3_frame) */
  RS3_K_STACK_GEMM = 10,   /* stack: QKV product, and W_os + LN2 + cross-attention queries */
  RS3_K_STACK_MERGE = 11,  /* stack: split merge of its attentions */
  RS3_K_STACK_MLP = 12,    /* stack: W_vo + LN3 + MLP chunk partials */
  RS3_K_STACK_ROWS = 13,   /* stack: gather / partial sum + LN1 / scatter */
  RS3_K_COUNT = 14
};
rs3_status rs3_profile_enable(int32_t on, int32_t max_launches);
rs3_status rs3_profile_report(double* total_ms, int64_t* launches, int64_t* dropped);
rs3_status rs3_profile_reset(void);

/* ---- read-only streaming rate (measurement) --------------------------------
 * Not part of the method: the reference that read-bound kernels (the
 * energies read each grid row once) are measured against, since a copy
 * kernel's rate counts reads and writes together.  Reads `bytes` bytes of
 * device memory at `src` once with 16-byte loads over RS3_STREAM_READ_THREADS
 * threads (grid-stride, four loads in flight per thread) and writes, for
 * thread i, the xor of every 32-bit word it read to out[i] (device, uint32,
 * RS3_STREAM_READ_THREADS entries).  src and bytes must be multiples of 16
 * (RS3_E_INVALID otherwise); nothing is allocated; enqueued on `stream`. */
#define RS3_STREAM_READ_THREADS (1024 * 256)
rs3_status rs3_stream_read(const void* src, size_t bytes, uint32_t* out, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* RS3_H */
