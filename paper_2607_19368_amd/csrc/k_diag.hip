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

// Bucket purity (section 5 kill test on buckets): token pairs i < j of one
// bucket whose rows of X have cosine similarity above thresh.  Pairs are
// visited in 64 x 64 tiles of the merge's sorted member order, where each bucket
// is a run: tile (A, B), A <= B, covers sorted positions [64 A, 64 A + 64) x
// [64 B, 64 B + 64) and is listed (by the host) only where a bucket spans both
// blocks, so every pair lies in exactly one tile.  A thread owns 4 x 4 pairs;
// the Gram block is accumulated in fp64 (products of the given values are
// exact) 32 columns at a time through LDS; cos = dot / (|x_i| |x_j|) with the
// fp64 row norms, 0 for a zero row.  Counts leave through integer atomics.
template <int DT>
__global__ __launch_bounds__(256) void k_dg_purity(const void* __restrict__ X, int64_t ldx, int D,
                                                   const int* __restrict__ sval,
                                                   const int* __restrict__ sseg,
                                                   const double* __restrict__ nrm, int64_t N,
                                                   const int2* __restrict__ tiles, double thresh,
                                                   unsigned long long* __restrict__ counts) {
  const int2 tl = tiles[blockIdx.x];
  const int tid = threadIdx.x, ty = tid >> 4, tx = tid & 15;
  __shared__ double sA[32][65], sB[32][65];     // [column][row]
  __shared__ int tokA[64], tokB[64], segA[64], segB[64];
  __shared__ double nA[64], nB[64];
  const int64_t a0 = (int64_t)tl.x * 64, b0 = (int64_t)tl.y * 64;
  if (tid < 128) {
    const int r = tid & 63;
    const int64_t q = (tid < 64 ? a0 : b0) + r;
    const int64_t pq = min(q, N - 1);
    const int tok = sval[pq];
    const int seg = (q < N) ? sseg[pq] : -1;
    const double nv = nrm[tok];
    if (tid < 64) {
      tokA[r] = tok;
      segA[r] = seg;
      nA[r] = nv;
    } else {
      tokB[r] = tok;
      segB[r] = seg;
      nB[r] = nv;
    }
  }
  __syncthreads();
  double acc[4][4];
#pragma unroll
  for (int u = 0; u < 4; ++u)
#pragma unroll
    for (int v = 0; v < 4; ++v) acc[u][v] = 0.0;
  for (int c0 = 0; c0 < D; c0 += 32) {
    for (int e = tid; e < 2 * 64 * 32; e += 256) {
      const int side = e >> 11, r = (e >> 5) & 63, cc = e & 31;
      const int col = c0 + cc;
      const int tok = side ? tokB[r] : tokA[r];
      double x = 0.0;
      if constexpr (DT == 0) {
        const uint16_t b = ((const uint16_t*)X)[(int64_t)tok * ldx + min(col, D - 1)];
        x = (double)__uint_as_float(((uint32_t)b) << 16);
      } else {
        x = (double)((const float*)X)[(int64_t)tok * ldx + min(col, D - 1)];
      }
      if (col >= D) x = 0.0;
      if (side) sB[cc][r] = x;
      else sA[cc][r] = x;
    }
    __syncthreads();
#pragma unroll 8
    for (int k = 0; k < 32; ++k) {
      double av[4], bv[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) av[u] = sA[k][4 * ty + u];
#pragma unroll
      for (int v = 0; v < 4; ++v) bv[v] = sB[k][4 * tx + v];
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int v = 0; v < 4; ++v) acc[u][v] = fma(av[u], bv[v], acc[u][v]);
    }
    __syncthreads();
  }
  int sim = 0, tot = 0;
#pragma unroll
  for (int u = 0; u < 4; ++u)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int ra = 4 * ty + u, rb = 4 * tx + v;
      const int64_t i = a0 + ra, j = b0 + rb;
      if (i < j && segA[ra] >= 0 && segA[ra] == segB[rb]) {
        ++tot;
        const double den = nA[ra] * nB[rb];
        if (den > 0.0 && acc[u][v] / den > thresh) ++sim;
      }
    }
  sim = wave_sum_i32(sim);
  tot = wave_sum_i32(tot);
  if ((tid & 63) == 0) {
    atomicAdd(&counts[0], (unsigned long long)sim);
    atomicAdd(&counts[1], (unsigned long long)tot);
  }
}

hipError_t launch_purity(const void* X, int dtype, int64_t ldx, int D, const int* sval,
                         const int* sseg, const double* nrm, int64_t N, const int* tiles,
                         int ntiles, double thresh, unsigned long long* counts, hipStream_t s) {
  (void)hipGetLastError();
  if (ntiles <= 0) return hipSuccess;
  if (dtype == 0)
    hipLaunchKernelGGL(k_dg_purity<0>, dim3(ntiles), dim3(256), 0, s, X, ldx, D, sval, sseg, nrm,
                       N, (const int2*)tiles, thresh, counts);
  else
    hipLaunchKernelGGL(k_dg_purity<1>, dim3(ntiles), dim3(256), 0, s, X, ldx, D, sval, sseg, nrm,
                       N, (const int2*)tiles, thresh, counts);
  return hipGetLastError();
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
