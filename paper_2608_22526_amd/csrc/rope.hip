// Axial rotary table for the sparse readout (Sec. 3.1, Eq. 7: the table f
// has one row of d_h/2 complex factors per grid cell; the readout gathers it
// with the keep-set).  Cell i = row * n + col; factor p < d_h/4 turns by
// col * theta^(-4p/d_h), factor d_h/4 + p by row * theta^(-4p/d_h).  Angles
// and their cosines and sines are evaluated in fp64 and stored as fp32
// (cos, sin) pairs: table [m*n][d_h/2][2].
#include "rs3_internal.h"

namespace rs3 {

__global__ __launch_bounds__(256) void k_rope_axial(float* table, int m, int n, int d_h, double theta) {
  const int half = d_h / 2, quarter = d_h / 4;
  const int64_t total = (int64_t)m * n * half;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < total; i += (int64_t)gridDim.x * 256) {
    const int cell = (int)(i / half), p = (int)(i - (int64_t)cell * half);
    const int row = cell / n, col = cell - row * n;
    const int e = p < quarter ? p : p - quarter;
    const double freq = pow(theta, -4.0 * e / d_h);
    const double angle = (p < quarter ? col : row) * freq;
    table[2 * i] = (float)cos(angle);
    table[2 * i + 1] = (float)sin(angle);
  }
}

}  // namespace rs3

using namespace rs3;

hipError_t rs3_launch_rope_axial(float* table, int m, int n, int d_h, double theta, hipStream_t st) {
  const int64_t total = (int64_t)m * n * (d_h / 2);
  const int64_t blocks = (total + 255) / 256;
  hipLaunchKernelGGL(k_rope_axial, dim3((unsigned)(blocks < 4096 ? blocks : 4096)), dim3(256), 0, st, table, m, n,
                     d_h, theta);
  return hipGetLastError();
}
