// Row norms of the prompt embeddings and the per-token feature-map scale.
//
// The random-feature map (section 3.2, Eq. 3) is multiplied per token by
// s(x) = exp(|x|^2 / (2 sqrt(D))) so that Phi Phi^T is unbiased for the
// unnormalised kernel exp(x.y / sqrt(D)) of section 3.2; the merge (Eq. 7)
// needs each member's norm |x_i| for the renormalisation target.  One wave per
// row; fp64 accumulation.  HBM-bound: one read of X (N*D*elem bytes).
#include "slh_device.h"
#include "slh_internal.h"

#include <algorithm>

namespace slh {

template <int DT>  // 0 = bf16, 1 = f32
__global__ __launch_bounds__(256) void k_rownorm(const void* __restrict__ Xv, int64_t ldx,
                                                 int64_t N, int D, double inv2sqrtD,
                                                 double sqrt2m, int gauss,
                                                 double* __restrict__ nrm2_fm,
                                                 double* __restrict__ nrm_x,
                                                 double* __restrict__ inv_x,
                                                 float* __restrict__ rowscale,
                                                 uint16_t* __restrict__ Xb) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= N) return;
  double s_fm = 0.0, s_x = 0.0;
  if (DT == 0) {
    const uint16_t* x = (const uint16_t*)Xv + row * ldx;
    // 8 bf16 (16 bytes) per lane per step
    for (int c = lane * 8; c < D; c += 512) {
      uint4 v = *(const uint4*)(x + c);
      uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        double a = (double)__uint_as_float(w[e] << 16);
        double b = (double)__uint_as_float(w[e] & 0xFFFF0000u);
        s_fm = fma(a, a, s_fm);
        s_fm = fma(b, b, s_fm);
      }
    }
    s_x = s_fm;
  } else {
    const float* x = (const float*)Xv + row * ldx;
    uint16_t* xb = Xb ? Xb + row * (int64_t)D : nullptr;
    for (int c = lane * 4; c < D; c += 256) {
      float4 v = *(const float4*)(x + c);
      float f[4] = {v.x, v.y, v.z, v.w};
      uint16_t hb[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        hb[e] = f32_to_bf16_rne(f[e]);
        double a = (double)bf16_to_f32(hb[e]);
        double g = (double)f[e];
        s_fm = fma(a, a, s_fm);
        s_x = fma(g, g, s_x);
      }
      if (Xb) {
        uint2 packed;
        packed.x = (uint32_t)hb[0] | ((uint32_t)hb[1] << 16);
        packed.y = (uint32_t)hb[2] | ((uint32_t)hb[3] << 16);
        *(uint2*)(xb + c) = packed;
      }
    }
  }
  s_fm = wave_sum_f64(s_fm);
  s_x = wave_sum_f64(s_x);
  if (lane == 0) {
    nrm2_fm[row] = s_fm;
    const double nx = sqrt(s_x);
    nrm_x[row] = nx;
    inv_x[row] = nx > 0.0 ? 1.0 / nx : 0.0;
    double sc = gauss ? 1.0 : exp(s_fm * inv2sqrtD);
    rowscale[row] = (float)(sc * sqrt2m);
  }
}

hipError_t launch_rownorm(const void* X, int dtype, int64_t ldx, int64_t N, int D, int m,
                          int gauss, double* nrm2_fm, double* nrm_x, double* inv_x,
                          float* rowscale, uint16_t* Xb, hipStream_t s) {
  (void)hipGetLastError();
  if (N <= 0) return hipSuccess;
  dim3 grid((unsigned)((N + 3) / 4));
  double inv2sqrtD = 1.0 / (2.0 * sqrt((double)D));
  double sqrt2m = sqrt(2.0 / (double)m);
  if (dtype == 0)
    hipLaunchKernelGGL(k_rownorm<0>, grid, dim3(256), 0, s, X, ldx, N, D, inv2sqrtD, sqrt2m,
                       gauss, nrm2_fm, nrm_x, inv_x, rowscale, Xb);
  else
    hipLaunchKernelGGL(k_rownorm<1>, grid, dim3(256), 0, s, X, ldx, N, D, inv2sqrtD, sqrt2m,
                       gauss, nrm2_fm, nrm_x, inv_x, rowscale, Xb);
  return hipGetLastError();
}

// dst[a][0..L) = src[winlist[a]][0..L) for the active windows (one launch for
// all of them, rather than a copy per window).
__global__ void k_gather_windows(double* __restrict__ dst, const double* __restrict__ src,
                                 const int* __restrict__ winlist, int64_t L) {
  const int a = blockIdx.y;
  const int64_t w = winlist[a];
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < L; i += (int64_t)gridDim.x * 256)
    dst[(int64_t)a * L + i] = src[w * L + i];
}

hipError_t launch_gather_windows(double* dst, const double* src, const int* winlist, int64_t L,
                                 int n_act, hipStream_t s) {
  (void)hipGetLastError();
  if (n_act <= 0 || L <= 0) return hipSuccess;
  const unsigned gx = (unsigned)std::min<int64_t>((L + 255) / 256, 64);
  hipLaunchKernelGGL(k_gather_windows, dim3(gx, n_act), dim3(256), 0, s, dst, src, winlist, L);
  return hipGetLastError();
}

}  // namespace slh
