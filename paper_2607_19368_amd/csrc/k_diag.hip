// Diagnostics of the spectral step (section 5 kill test on spectral energy,
// rank ablation): per spectral window, the fraction of the operator's energy
// held by the kept Ritz values, sum(theta) / tr(Phi Phi^T), where
// tr(Phi Phi^T) = ||Phi_w||_F^2 (of the rows actually used, i.e. after the
// row normalisation when that option is on).  fp64, fixed summation order.
#include "slh_device.h"
#include "slh_internal.h"

namespace slh {

// rowsq[a][i] = ||phi_i||^2: one wave per row, lane = 4 columns of every
// 256-column slice, then a butterfly.
__global__ __launch_bounds__(256) void k_dg_rowsq(const float* __restrict__ Phi, int L, int m,
                                                  double* __restrict__ rowsq) {
  const int a = blockIdx.y, lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= L) return;                          // whole waves
  const float* P = Phi + ((int64_t)a * L + row) * m;
  const int nq = m >> 8;
  float4 v[8];
#pragma unroll
  for (int q = 0; q < 8; ++q) v[q] = *(const float4*)(P + 256 * min(q, nq - 1) + 4 * lane);
  double d = 0.0;
#pragma unroll
  for (int q = 0; q < 8; ++q) {
    if (q < nq) {
      d = fma((double)v[q].x, (double)v[q].x, d);
      d = fma((double)v[q].y, (double)v[q].y, d);
      d = fma((double)v[q].z, (double)v[q].z, d);
      d = fma((double)v[q].w, (double)v[q].w, d);
    }
  }
  d = wave_sum_f64(d);
  if (lane == 0) rowsq[(int64_t)a * L + row] = d;
}

// energy[a] = sum_c theta[a][c] / sum_i rowsq[a][i] (0 when the trace is 0):
// one 256-thread block per window.
__global__ __launch_bounds__(256) void k_dg_energy(const double* __restrict__ rowsq,
                                                   const double* __restrict__ theta, int L, int r,
                                                   double* __restrict__ energy) {
  const int a = blockIdx.x, tid = threadIdx.x;
  __shared__ double red[4];
  double t = 0.0;
  for (int i = tid; i < L; i += 256) t += rowsq[(int64_t)a * L + i];
  const double tr = block_sum_f64(t, red);
  double th = 0.0;
  if (tid == 0)
    for (int c = 0; c < r; ++c) th += theta[(int64_t)a * r + c];
  if (tid == 0) energy[a] = (tr > 0.0) ? th / tr : 0.0;
}

hipError_t launch_energy(const float* Phi, const double* theta, int n_act, int L, int m, int r,
                         double* rowsq, double* energy, hipStream_t s) {
  (void)hipGetLastError();
  if (n_act <= 0) return hipSuccess;
  if (m % 256 != 0) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_dg_rowsq, dim3((L + 3) / 4, n_act), dim3(256), 0, s, Phi, L, m, rowsq);
  hipLaunchKernelGGL(k_dg_energy, dim3(n_act), dim3(256), 0, s, rowsq, theta, L, r, energy);
  return hipGetLastError();
}

}  // namespace slh
