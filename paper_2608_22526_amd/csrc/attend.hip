// Bare attention core of the readout (Eq. 6 without the projections):
// O_h = softmax(Q_h K_h^T / sqrt(d_h)) V_h on already-projected tensors.
//
// bf16: the tensors are laid out as a one-frame bank in the caller's
// workspace (k_attend_prep), the readout's split-KV attention kernel runs on
// it unchanged, and k_attend_merge combines the key splits into fp32 O.
// fp32: k_attend_f32, one work-group per query row, FMA loops.
#include "rs3_internal.h"

namespace rs3 {

// grid (max(ntile*H, nqb), 2), block 256.
//  y = 0: block (tile t, head h) copies keys 64t..64t+63 of head h into the
//         K^ tile ([64][d_h]) and the V^ tile ([d_h][64] in slot order),
//         zero-filling past n_kv; (t, 0) writes the tile's list entry, and
//         block (0, 0) the bank descriptor, header and query count.
//  y = 1: block b scales 256 chunks of 8 query values by qscale into Qs.
__global__ __launch_bounds__(256) void k_attend_prep(AttendPrepArgs p) {
  const int tid = threadIdx.x;
  const int D = p.H * p.d_h;
  if (blockIdx.y == 1) {
    const int64_t chunk = (int64_t)blockIdx.x * 256 + tid;
    if (chunk * 8 >= (int64_t)p.n_q * D) return;
    const u32x4 v = *(const u32x4*)(p.Q + chunk * 8);
    u32x4 w;
#pragma unroll
    for (int e = 0; e < 4; ++e)
      w[e] = pack_bf16x2(__uint_as_float(v[e] << 16) * p.qscale, __uint_as_float(v[e] & 0xffff0000u) * p.qscale);
    *(u32x4*)(p.Qs + chunk * 8) = w;
    return;
  }
  if (blockIdx.x == 0 && tid == 0) {
    BankDev d = {};
    d.cap = p.ntile * KT;
    d.f_max = 1;
    d.n_pin = 0;
    d.d_kv = p.d_h;
    d.H = p.H;
    d.d_h = p.d_h;
    d.dtype = RS3_BF16;
    d.n_tiles_cap = p.ntile;
    d.Khat = p.Khat;
    d.Vhat = p.Vhat;
    d.hdr = p.hdr;
    d.tiles = p.tiles;
    *p.desc = d;
    for (int w = 0; w < HDR_WORDS; ++w) p.hdr[w] = 0;
    p.hdr[HDR_NTILES] = p.ntile;
    p.hdr[HDR_NKEYS] = (int)p.n_kv;
    p.hdr[HDR_PLEN] = -1;
    *p.count = p.n_q;
  }
  const int t = blockIdx.x / p.H, h = blockIdx.x - t * p.H;
  if (t >= p.ntile) return;
  const int d_h = p.d_h, cpr = d_h / 8;
  bf16_t* kt = p.Khat + ((int64_t)t * p.H + h) * KT * d_h;
  bf16_t* vt = p.Vhat + ((int64_t)t * p.H + h) * d_h * KT;
  for (int q = tid; q < KT * cpr; q += 256) {
    const int r = q / cpr, c = q - r * cpr;
    const int64_t j = (int64_t)t * KT + r;
    u32x4 kv = {0, 0, 0, 0}, vv = {0, 0, 0, 0};
    if (j < p.n_kv) {
      kv = *(const u32x4*)(p.K + (j * p.H + h) * d_h + 8 * c);
      vv = *(const u32x4*)(p.V + (j * p.H + h) * d_h + 8 * c);
    }
    *(u32x4*)(kt + r * d_h + 8 * c) = kv;
    const int slot = vslot(r);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      vt[(8 * c + 2 * e) * KT + slot] = (bf16_t)(vv[e] & 0xffffu);
      vt[(8 * c + 2 * e + 1) * KT + slot] = (bf16_t)(vv[e] >> 16);
    }
  }
  if (h == 0 && tid == 0) {
    const int64_t left = p.n_kv - (int64_t)t * KT;
    TileEnt e;
    e.tile = t;
    e.pad = 0;
    e.mask = left >= KT ? ~0ull : ((1ull << left) - 1ull);
    p.tiles[t] = e;
  }
}

// One thread per (query row, 8-column chunk): online log-sum-exp merge of
// the SA key splits into fp32 O [n_q][D].
__global__ __launch_bounds__(256) void k_attend_merge(Rs3ReadoutArgs a, int SA, float* O) {
  const int D = a.D, cpr = D / 8;
  const int64_t it = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (it >= (int64_t)a.max_sel * cpr) return;
  const int row = (int)(it / cpr), d0 = 8 * (int)(it - (int64_t)row * cpr), h = d0 / a.d_h;
  float M = -INFINITY, W = 0.f;
  float acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  for (int s = 0; s < SA; ++s) {
    const int64_t prow = (int64_t)s * a.max_sel + row;
    const float m = a.ML[(prow * a.H + h) * 2], l = a.ML[(prow * a.H + h) * 2 + 1];
    if (!(l > 0.f)) continue;
    const u32x4 v = *(const u32x4*)((const bf16_t*)a.Opart + prow * D + d0);
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
  float* out = O + (int64_t)row * D + d0;
  *(f32x4*)out = f32x4{acc[0] * inv, acc[1] * inv, acc[2] * inv, acc[3] * inv};
  *(f32x4*)(out + 4) = f32x4{acc[4] * inv, acc[5] * inv, acc[6] * inv, acc[7] * inv};
}

// fp32: grid n_q, block 256; per head, online softmax over 64-key tiles.
__global__ __launch_bounds__(256) void k_attend_f32(const float* Q, const float* K, const float* V, int n_q,
                                                    int64_t n_kv, int H, int d_h, float qscale, float* O) {
  __shared__ float q[256];
  __shared__ float pr[KT];
  __shared__ float st[4];   // running max, running sum, rescale factor
  const int r = blockIdx.x, tid = threadIdx.x, D = H * d_h;
  float* out = O + (int64_t)r * D;
  for (int h = 0; h < H; ++h) {
    for (int u = tid; u < d_h; u += 256) q[u] = Q[(int64_t)r * D + h * d_h + u] * qscale;
    if (tid == 0) {
      st[0] = -INFINITY;
      st[1] = 0.f;
    }
    float acc = 0.f;   // thread tid < d_h owns output column tid
    __syncthreads();
    for (int64_t j0 = 0; j0 < n_kv; j0 += KT) {
      if (tid < KT) {
        float s = -INFINITY;
        if (j0 + tid < n_kv) {
          const float* kr = K + ((j0 + tid) * H + h) * d_h;
          s = 0.f;
          for (int u = 0; u < d_h; ++u) s = fmaf(q[u], kr[u], s);
        }
        pr[tid] = s;
      }
      __syncthreads();
      if (tid == 0) {
        float mx = -INFINITY;
        for (int j = 0; j < KT; ++j) mx = fmaxf(mx, pr[j]);
        const float m_new = fmaxf(st[0], mx);
        const float alpha = exp2f(st[0] - m_new);
        float ps = 0.f;
        for (int j = 0; j < KT; ++j) {
          const float pj = exp2f(pr[j] - m_new);
          pr[j] = pj;
          ps += pj;
        }
        st[1] = st[1] * alpha + ps;
        st[0] = m_new;
        st[2] = alpha;
      }
      __syncthreads();
      if (tid < d_h) {
        acc *= st[2];
        const int64_t nk = n_kv - j0 < KT ? n_kv - j0 : KT;
        for (int j = 0; j < nk; ++j) acc = fmaf(pr[j], V[((j0 + j) * H + h) * d_h + tid], acc);
      }
      __syncthreads();
    }
    if (tid < d_h) out[h * d_h + tid] = st[1] > 0.f ? acc / st[1] : 0.f;
    __syncthreads();
  }
}

}  // namespace rs3

using namespace rs3;

hipError_t rs3_launch_attend_prep(const AttendPrepArgs& p, hipStream_t st) {
  const int D = p.H * p.d_h;
  const int64_t nqb = ((int64_t)p.n_q * D / 8 + 255) / 256;
  const int64_t nx = (int64_t)p.ntile * p.H > nqb ? (int64_t)p.ntile * p.H : nqb;
  if (nx == 0) {
    // nothing to lay out but the descriptor: one block writes it
    hipLaunchKernelGGL(k_attend_prep, dim3(1, 1), dim3(256), 0, st, p);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(k_attend_prep, dim3((unsigned)nx, 2), dim3(256), 0, st, p);
  return hipGetLastError();
}

hipError_t rs3_launch_attend_merge(const Rs3ReadoutArgs& a, int SA, float* O, hipStream_t st) {
  const int64_t items = (int64_t)a.max_sel * (a.D / 8);
  if (items == 0) return hipSuccess;
  hipLaunchKernelGGL(k_attend_merge, dim3((unsigned)((items + 255) / 256)), dim3(256), 0, st, a, SA, O);
  return hipGetLastError();
}

hipError_t rs3_launch_attend_f32(const float* Q, const float* K, const float* V, int n_q, int64_t n_kv, int H,
                                 int d_h, float qscale, float* O, hipStream_t st) {
  if (n_q == 0) return hipSuccess;
  hipLaunchKernelGGL(k_attend_f32, dim3(n_q), dim3(256), 0, st, Q, K, V, n_q, n_kv, H, d_h, qscale, O);
  return hipGetLastError();
}
