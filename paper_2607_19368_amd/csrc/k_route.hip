// Window redundancy score of the adaptive backend (section 3.6, Eq. 8):
//   score = (1/L) sum_i x_i . xbar / (|x_i| |xbar|),  xbar = S / |S|,  S = sum_i x_i
// computed in one pass as (U . S) / (L |S|) with U = sum_i x_i / |x_i| (zero rows
// contribute nothing; 1 / |x_i| comes precomputed with the row norms).
// Workgroup (window, slice of 64 columns): thread (phase p = tid / 8, column
// group cg = tid % 8) accumulates S and U in fp64 for 8 columns over rows
// p, p + 32, ... of the window, 16-byte loads with 8 rows in flight; the 32
// phases are added in LDS in phase order and the workgroup emits the partial
// dot U.S and |S|^2 of its columns; a second kernel adds the slices in order.
#include "slh_device.h"
#include "slh_internal.h"

namespace slh {

constexpr int RT_COLS = 64;                    // columns per workgroup
constexpr int RT_PH = 32;                      // row phases per workgroup

template <int DT>
__device__ __forceinline__ void rt_load8(const void* X, int64_t ldx, int64_t row, int col,
                                         float (&x)[8]) {
  if constexpr (DT == 0) {
    const uint4 v = *(const uint4*)((const uint16_t*)X + row * ldx + col);
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      x[2 * e] = __uint_as_float(w[e] << 16);
      x[2 * e + 1] = __uint_as_float(w[e] & 0xFFFF0000u);
    }
  } else {
    const float4* p = (const float4*)((const float*)X + row * ldx + col);
    const float4 a = p[0], b = p[1];
    x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
    x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
  }
}

template <int DT>
__global__ __launch_bounds__(256) void k_route_part(const void* __restrict__ X, int64_t ldx,
                                                    const double* __restrict__ inv_x, int L,
                                                    int D, double* __restrict__ part) {
  const int win = blockIdx.x, cs = blockIdx.y, tid = threadIdx.x;
  const int ph = tid >> 3, cg = tid & 7;
  const int c0 = cs * RT_COLS + cg * 8;
  const int cc = min(c0, D - 8);                 // D % 8 == 0; columns past D masked below
  const int64_t r0 = (int64_t)win * L;
  const int nr = (L - ph + RT_PH - 1) / RT_PH;   // rows of this phase
  double S[8], U[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) S[k] = U[k] = 0.0;
  for (int b = 0; b < nr; b += 8) {
    // 8 rows in flight (index clamped to the phase's last row, the surplus masked)
    float x[8][8];
    double iv[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int64_t row = r0 + ph + (int64_t)RT_PH * min(b + e, nr - 1);
      rt_load8<DT>(X, ldx, row, cc, x[e]);
      iv[e] = inv_x[row];
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      if (b + e < nr) {
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          S[k] += (double)x[e][k];
          U[k] = fma((double)x[e][k], iv[e], U[k]);
        }
      }
    }
  }
  __shared__ double sS[RT_PH][RT_COLS + 1], sU[RT_PH][RT_COLS + 1];
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    sS[ph][cg * 8 + k] = S[k];
    sU[ph][cg * 8 + k] = U[k];
  }
  __syncthreads();
  if (tid < RT_COLS) {                           // wave 0: one column per lane
    double St = 0.0, Ut = 0.0;
#pragma unroll 8
    for (int q = 0; q < RT_PH; ++q) {
      St += sS[q][tid];
      Ut += sU[q][tid];
    }
    const bool in = cs * RT_COLS + tid < D;
    double dot = in ? Ut * St : 0.0, ss = in ? St * St : 0.0;
    dot = wave_sum_f64(dot);
    ss = wave_sum_f64(ss);
    if (tid == 0) {
      part[((int64_t)win * gridDim.y + cs) * 2 + 0] = dot;
      part[((int64_t)win * gridDim.y + cs) * 2 + 1] = ss;
    }
  }
}

// one wave per window: lane q adds slices q, q + 64, ... (in order), then a
// butterfly over the lanes (a fixed order)
__global__ __launch_bounds__(64) void k_route_final(const double* __restrict__ part, int ncs,
                                                    int L, double* __restrict__ scores) {
  const int win = blockIdx.x, lane = threadIdx.x;
  double dot = 0.0, ss = 0.0;
  for (int c = lane; c < ncs; c += 64) {
    dot += part[((int64_t)win * ncs + c) * 2 + 0];
    ss += part[((int64_t)win * ncs + c) * 2 + 1];
  }
  dot = wave_sum_f64(dot);
  ss = wave_sum_f64(ss);
  if (lane == 0) scores[win] = ss > 0.0 ? dot / ((double)L * sqrt(ss)) : 0.0;
}

int route_slices(int D) { return (D + RT_COLS - 1) / RT_COLS; }

hipError_t launch_route_scores(const void* X, int dtype, int64_t ldx, const double* inv_x,
                               int n_win, int L, int D, double* part, double* scores,
                               hipStream_t s) {
  (void)hipGetLastError();
  if (n_win <= 0) return hipSuccess;
  if (D % 8 != 0 || D < 8 || L < 1) return hipErrorInvalidValue;
  const int ncs = route_slices(D);
  if (dtype == 0)
    hipLaunchKernelGGL(k_route_part<0>, dim3(n_win, ncs), dim3(256), 0, s, X, ldx, inv_x, L, D,
                       part);
  else
    hipLaunchKernelGGL(k_route_part<1>, dim3(n_win, ncs), dim3(256), 0, s, X, ldx, inv_x, L, D,
                       part);
  hipLaunchKernelGGL(k_route_final, dim3(n_win), dim3(64), 0, s, part, ncs, L, scores);
  return hipGetLastError();
}

}  // namespace slh
