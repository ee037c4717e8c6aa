// Device helpers shared by the readout kernels and the fused merge + commit
// launch (gfx950 only).
#pragma once

#include "rs3_internal.h"

namespace rs3 {

// Loads through global (not generic) pointers: the compiler then counts
// them on the vector memory counter alone, and a wait for one of them does
// not have to drain every outstanding load.
#define RS3_GLOBAL __attribute__((address_space(1)))
template <class T>
__device__ __forceinline__ T gload(const T* p) {
  return *(const RS3_GLOBAL T*)p;
}

// Stores through global pointers, for the same reason: a generic (flat)
// store counts on the LDS counter too, so a later wait for an LDS read would
// also wait for the store to land.
template <class T>
__device__ __forceinline__ void gstore(T* p, const T& v) {
  *(RS3_GLOBAL T*)p = v;
}

// Non-temporal (streaming) accesses for data that is written once and read
// once: the readout's split partials.  The merge reads every partial with
// pload; k_attn_g2, and k_attn when the readout launches it, write them
// with pstore.  Measured on the 64x64 one-object frame: the stores gave
// 1.2-1.4 % more frames/s, the loads another 1.6 %, and the attention of the
// next frame got faster too (the partials, about 3.7 MB a frame, no longer
// crowd the bank's key/value tiles out of the L2); with k_attn's stores as
// well the projected 64x64 frame gained 5 %, the other readout workloads
// 0.2-0.9 %.  The same marking was slower for the energies and projected
// queries of the energy launch, which the next launch reads back, and for
// the partials of the stack's attentions, which its own merge reads.
template <class T>
__device__ __forceinline__ void pstore(T* p, const T& v) {
  __builtin_nontemporal_store(v, (RS3_GLOBAL T*)p);
}
template <class T>
__device__ __forceinline__ T pload(const T* p) {
  return __builtin_nontemporal_load((const RS3_GLOBAL T*)p);
}

// Loads of wave-uniform values that earlier launches wrote (bank headers,
// descriptors, selected counts): through the constant address space the
// compiler uses scalar loads, which are counted apart from the vector loads,
// so waiting for them does not wait for the operand loads issued before.
#define RS3_CONST __attribute__((address_space(4)))
template <class T>
__device__ __forceinline__ T sload(const T* p) {
  return *(const RS3_CONST T*)p;
}

// Waits for loaded values and hands them on as values the compiler did not
// see being loaded: a loop that uses them then carries no pending load to
// its head, where the compiler would otherwise wait for every outstanding
// load (the key/value DMA included) in each iteration.
__device__ __forceinline__ void settle(int& a, uint32_t& b, uint32_t& c) {
  asm volatile("s_waitcnt vmcnt(0)" : "+v"(a), "+v"(b), "+v"(c)::"memory");
}

// Keeps a loaded value alive on a path that does not use it, so the load is
// issued before the branch rather than sunk past it (an early exit would
// otherwise delay every load that only the main path uses).
template <class T>
__device__ __forceinline__ void keep(const T& v) {
  asm volatile("" ::"v"(v));
}
template <class T>
__device__ __forceinline__ void keep_s(const T& v) {
  asm volatile("" ::"s"(v));
}

__device__ __forceinline__ int sel_count_of(const Rs3ReadoutArgs& a, int o, BankDev& b,
                                            bool report) {
  int cnt = gload(a.sel_count + (a.sel_stride ? o : 0));
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

// Maximum over the 64 lanes by the same exchange pattern.
__device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, dppf<0xB1>(v));
  v = fmaxf(v, dppf<0x4E>(v));
  v = fmaxf(v, dppf<0x141>(v));
  v = fmaxf(v, dppf<0x140>(v));
  auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
  r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

}  // namespace rs3
