// Normalised operator (section 3.2, remark on row normalisation; appendix,
// softmax normalisation gap): per spectral window the row sums of the estimated
// kernel are s = Phi_w (Phi_w^T 1), and the rows of Phi_w are scaled in place by
// s_i^-1/2 (0 where s_i <= 0).  Lanczos then runs unchanged on
// diag(s)^-1/2 Phi Phi^T diag(s)^-1/2, which is similar to the normalised matvec
// diag(s)^-1 Phi Phi^T; its Ritz vectors differ from the normalised operator's by
// a positive row scaling, which SimHash does not see.
//
// Three passes, every sum in a fixed order (fp64): column partial sums over
// groups of rows, their reduction to Phi^T 1, and one wave per row forming
// s_i = phi_i . (Phi^T 1), then rewriting the row.  Work: two reads and one
// write of Phi (HBM-bound, 3 x 67 MB at N = 8192, m = 2048).
#include "slh_device.h"
#include "slh_internal.h"

#include <algorithm>

namespace slh {

// part[a][g][col] = sum of Phi[a][r][col] over rows r of group g (NR rows).
__global__ __launch_bounds__(256) void k_nm_colsum(const float* __restrict__ Phi, int L, int m,
                                                   int NR, double* __restrict__ part) {
  const int sl = blockIdx.x, g = blockIdx.y, a = blockIdx.z, tid = threadIdx.x;
  const int G = gridDim.y;
  const int col = sl * 256 + tid;
  const int r0 = g * NR, r1 = min(r0 + NR, L);
  const float* P = Phi + (int64_t)a * L * m + col;
  double acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  for (int r = r0; r < r1; r += 8) {
    // unconditional loads (rows clamped to the group, the surplus masked)
    float v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = P[(int64_t)min(r + e, r1 - 1) * m];
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] += (r + e < r1) ? (double)v[e] : 0.0;
  }
  part[((int64_t)a * G + g) * m + col] =
      ((acc[0] + acc[1]) + (acc[2] + acc[3])) + ((acc[4] + acc[5]) + (acc[6] + acc[7]));
}

// csum[a][col] = sum over the G groups of part[a][g][col], groups in order.
__global__ __launch_bounds__(256) void k_nm_colreduce(const double* __restrict__ part, int G, int m,
                                                      double* __restrict__ csum) {
  const int col = blockIdx.x * 256 + threadIdx.x, a = blockIdx.y;
  const double* p = part + (int64_t)a * G * m + col;
  double acc = 0.0;
  for (int g = 0; g < G; g += 8) {
    double v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = p[(int64_t)min(g + e, G - 1) * m];
#pragma unroll
    for (int e = 0; e < 8; ++e) acc += (g + e < G) ? v[e] : 0.0;
  }
  csum[(int64_t)a * m + col] = acc;
}

// One wave per row: s_i = phi_i . csum (lane = 4 columns of every 256-column
// slice, then a butterfly), w_i = s_i^-1/2 or 0, phi_i <- w_i phi_i.
__global__ __launch_bounds__(256) void k_nm_rowscale(float* __restrict__ Phi,
                                                     const double* __restrict__ csum, int L, int m,
                                                     double* __restrict__ s_out) {
  const int a = blockIdx.y, lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= L) return;                          // whole waves
  float* P = Phi + ((int64_t)a * L + row) * m;
  const double* ca = csum + (int64_t)a * m;
  const int nq = m >> 8;                         // 1..8 slices
  float4 v[8];
#pragma unroll
  for (int q = 0; q < 8; ++q) v[q] = *(const float4*)(P + 256 * min(q, nq - 1) + 4 * lane);
  double d = 0.0;
#pragma unroll
  for (int q = 0; q < 8; ++q) {
    if (q < nq) {
      const double* cq = ca + 256 * q + 4 * lane;
      d = fma((double)v[q].x, cq[0], d);
      d = fma((double)v[q].y, cq[1], d);
      d = fma((double)v[q].z, cq[2], d);
      d = fma((double)v[q].w, cq[3], d);
    }
  }
  d = wave_sum_f64(d);
  const double w = (d > 0.0) ? 1.0 / sqrt(d) : 0.0;
#pragma unroll
  for (int q = 0; q < 8; ++q) {
    if (q < nq) {
      float4 o;
      o.x = (float)(w * (double)v[q].x);
      o.y = (float)(w * (double)v[q].y);
      o.z = (float)(w * (double)v[q].z);
      o.w = (float)(w * (double)v[q].w);
      *(float4*)(P + 256 * q + 4 * lane) = o;
    }
  }
  if (lane == 0) s_out[(int64_t)a * L + row] = d;
}

int normalise_groups(int n_act, int L, int m, int n_cu) {
  const int64_t per = (int64_t)n_act * (m / 256);
  int G = (int)std::max<int64_t>(1, (4LL * n_cu + per - 1) / per);
  return std::max(1, std::min(G, (L + 7) / 8));
}

hipError_t launch_normalise(float* Phi, int n_act, int L, int m, int G, double* part, double* csum,
                            double* s_out, hipStream_t s) {
  (void)hipGetLastError();
  if (n_act <= 0 || m % 256 != 0 || G < 1) return n_act <= 0 ? hipSuccess : hipErrorInvalidValue;
  const int NR = (((L + G - 1) / G) + 7) / 8 * 8;
  const int Gr = (L + NR - 1) / NR;              // groups that hold rows
  hipLaunchKernelGGL(k_nm_colsum, dim3(m / 256, Gr, n_act), dim3(256), 0, s, Phi, L, m, NR, part);
  hipLaunchKernelGGL(k_nm_colreduce, dim3(m / 256, n_act), dim3(256), 0, s, part, Gr, m, csum);
  hipLaunchKernelGGL(k_nm_rowscale, dim3((L + 3) / 4, n_act), dim3(256), 0, s, Phi, csum, L, m,
                     s_out);
  return hipGetLastError();
}

}  // namespace slh
