// SimHash in the spectral subspace (Eq. 5): bit l of token i is
// [R[:, l] . z_i > 0], packed as code_i = sum_l bit_l 2^l.
//
// A wave covers 4 tokens x 16 hyperplanes: lane (q, l) computes the fp64
// projection of token q onto hyperplane l, and one wavefront ballot packs the
// 64 sign bits; token q's code is bits [16q, 16q + bits) of the ballot.
#include "slh_device.h"
#include "slh_internal.h"

namespace slh {

__global__ __launch_bounds__(256) void k_simhash(const double* __restrict__ Z,
                                                 const double* __restrict__ R,
                                                 const int* __restrict__ winlist, int L, int r,
                                                 int bits, uint32_t* __restrict__ codes,
                                                 double* __restrict__ proj) {
  __shared__ double sR[128 * 16];
  const int a = blockIdx.y, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  for (int k = tid; k < r * 16; k += 256) {
    const int c = k >> 4, l = k & 15;
    sR[k] = (l < bits) ? R[c * bits + l] : 0.0;
  }
  __syncthreads();
  const int q = lane >> 4, l = lane & 15;
  const int i = (blockIdx.x * 4 + wave) * 4 + q;   // token within the window
  double p = 0.0;
  if (i < L) {
    const double* z = Z + ((int64_t)a * L + i) * r;
    for (int c = 0; c < r; ++c) p = fma(z[c], sR[c * 16 + l], p);
  }
  const unsigned long long m = __ballot(i < L && l < bits && p > 0.0);
  if (i < L) {
    if (l < bits) proj[((int64_t)a * L + i) * bits + l] = p;
    if (l == 0) {
      const int64_t gi = (int64_t)(winlist ? winlist[a] : a) * L + i;
      codes[gi] = (uint32_t)((m >> (16 * q)) & 0xFFFFull);
    }
  }
}

__global__ void k_fill_u32(uint32_t* p, int64_t n, uint32_t v) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256)
    p[i] = v;
}

hipError_t launch_simhash(const double* Z, const double* R, const int* winlist, int n_act,
                          int L, int r, int bits, uint32_t* codes, double* proj,
                          hipStream_t s) {
  (void)hipGetLastError();
  const int blocks = (L + 15) / 16;
  hipLaunchKernelGGL(k_simhash, dim3(blocks, n_act), dim3(256), 0, s, Z, R, winlist, L, r, bits,
                     codes, proj);
  return hipGetLastError();
}

hipError_t launch_fill_u32(uint32_t* p, int64_t n, uint32_t v, hipStream_t s) {
  (void)hipGetLastError();
  if (n <= 0) return hipSuccess;
  int64_t b = (n + 255) / 256;
  if (b > 4096) b = 4096;
  hipLaunchKernelGGL(k_fill_u32, dim3((unsigned)b), dim3(256), 0, s, p, n, v);
  return hipGetLastError();
}

}  // namespace slh
