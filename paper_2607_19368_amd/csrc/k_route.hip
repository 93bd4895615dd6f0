// Window redundancy score of the adaptive backend (section 3.6, Eq. 8):
//   score = (1/L) sum_i x_i . xbar / (|x_i| |xbar|),  xbar = S / |S|,  S = sum_i x_i
// computed in one pass as (U . S) / (L |S|) with U = sum_i x_i / |x_i| (zero rows
// contribute nothing).  Workgroup (window, slice of 1024 columns) accumulates
// S and U for its columns over the window's rows in fp64 and emits the partial
// dot U.S and |S|^2; a second kernel adds the slices in fixed order.
#include "slh_device.h"
#include "slh_internal.h"

namespace slh {

template <int DT>
__global__ __launch_bounds__(256) void k_route_part(const void* __restrict__ X, int64_t ldx,
                                                    const double* __restrict__ nrm_x, int L,
                                                    int D, double* __restrict__ part) {
  const int win = blockIdx.x, cs = blockIdx.y, tid = threadIdx.x;
  const int col = cs * 1024 + tid * 4;
  double S[4] = {0, 0, 0, 0}, U[4] = {0, 0, 0, 0};
  const int64_t r0 = (int64_t)win * L;
  if (col < D) {
    for (int i = 0; i < L; ++i) {
      const int64_t row = r0 + i;
      const double nx = nrm_x[row];
      const double inv = nx > 0.0 ? 1.0 / nx : 0.0;
      float x[4];
      if (DT == 0) {
        const uint2 v = *(const uint2*)((const uint16_t*)X + row * ldx + col);
        x[0] = __uint_as_float(v.x << 16);
        x[1] = __uint_as_float(v.x & 0xFFFF0000u);
        x[2] = __uint_as_float(v.y << 16);
        x[3] = __uint_as_float(v.y & 0xFFFF0000u);
      } else {
        const float4 v = *(const float4*)((const float*)X + row * ldx + col);
        x[0] = v.x; x[1] = v.y; x[2] = v.z; x[3] = v.w;
      }
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        S[e] += (double)x[e];
        U[e] = fma((double)x[e], inv, U[e]);
      }
    }
  }
  double dot = 0.0, ss = 0.0;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    dot = fma(U[e], S[e], dot);
    ss = fma(S[e], S[e], ss);
  }
  __shared__ double red[4];
  dot = block_sum_f64(dot, red);
  ss = block_sum_f64(ss, red);
  if (tid == 0) {
    part[((int64_t)win * gridDim.y + cs) * 2 + 0] = dot;
    part[((int64_t)win * gridDim.y + cs) * 2 + 1] = ss;
  }
}

__global__ void k_route_final(const double* __restrict__ part, int ncs, int L,
                              double* __restrict__ scores, int n_win) {
  const int win = blockIdx.x * 64 + threadIdx.x;
  if (win >= n_win) return;
  double dot = 0.0, ss = 0.0;
  for (int c = 0; c < ncs; ++c) {
    dot += part[((int64_t)win * ncs + c) * 2 + 0];
    ss += part[((int64_t)win * ncs + c) * 2 + 1];
  }
  scores[win] = ss > 0.0 ? dot / ((double)L * sqrt(ss)) : 0.0;
}

hipError_t launch_route_scores(const void* X, int dtype, int64_t ldx, const double* nrm_x,
                               int n_win, int L, int D, double* part, double* scores,
                               hipStream_t s) {
  (void)hipGetLastError();
  const int ncs = (D + 1023) / 1024;
  if (dtype == 0)
    hipLaunchKernelGGL(k_route_part<0>, dim3(n_win, ncs), dim3(256), 0, s, X, ldx, nrm_x, L, D,
                       part);
  else
    hipLaunchKernelGGL(k_route_part<1>, dim3(n_win, ncs), dim3(256), 0, s, X, ldx, nrm_x, L, D,
                       part);
  hipLaunchKernelGGL(k_route_final, dim3((n_win + 63) / 64), dim3(64), 0, s, part, ncs, L,
                     scores, n_win);
  return hipGetLastError();
}

}  // namespace slh
