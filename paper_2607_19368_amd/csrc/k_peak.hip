// Measured ceilings for the roofline figures (measurement aids, no part of the
// method): the rate at which this device streams a buffer from memory, and the
// rate of its dense bf16 matrix cores.  Both are timed with HIP events around
// repeated launches on the caller's stream.
#include "slh.h"
#include "slh_device.h"

#include <algorithm>

namespace slh {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

// Every 16-byte word of the buffer read once per launch: grid-stride over
// float4 words, four non-temporal loads in flight per thread per round (the
// fastest of the shapes measured on this part: 16 blocks of 512 per CU,
// 6.6 TB/s over 1 GiB, 7.7 TB/s over 64 MiB).  The words are folded into one
// value per thread that is stored only if it equals a value no sum of these
// words takes in practice, so the loads cannot be dropped and nothing is
// written.
typedef float pk_f32x4 __attribute__((ext_vector_type(4)));
__global__ __launch_bounds__(512) void k_peak_read(const float4* __restrict__ src, int64_t n4,
                                                   float* __restrict__ sink) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const pk_f32x4* s4 = (const pk_f32x4*)src;
  float acc = 0.0f;
  for (; i + 3 * stride < n4; i += 4 * stride) {
    const pk_f32x4 a = __builtin_nontemporal_load(s4 + i);
    const pk_f32x4 b = __builtin_nontemporal_load(s4 + i + stride);
    const pk_f32x4 c = __builtin_nontemporal_load(s4 + i + 2 * stride);
    const pk_f32x4 d = __builtin_nontemporal_load(s4 + i + 3 * stride);
    acc += (a.x + b.y) + (c.z + d.w);
  }
  for (; i < n4; i += stride) acc += src[i].x;
  if (acc == -1.2345e-38f) sink[threadIdx.x & 3] = acc;
}

// Independent v_mfma_f32_32x32x16_bf16 chains, operands in registers: each wave
// issues NACC MFMAs per round, reps rounds.
constexpr int PK_NACC = 8;
__global__ __launch_bounds__(256) void k_peak_mfma(int rounds, float* __restrict__ sink) {
  const int lane = threadIdx.x & 63;
  bf16x8 a, b;
  for (int e = 0; e < 8; ++e) {
    a[e] = (__bf16)(1.0f + 0.001f * (float)((lane + e) & 15));
    b[e] = (__bf16)(0.5f - 0.001f * (float)((lane * 3 + e) & 15));
  }
  f32x16 acc[PK_NACC];
  for (int q = 0; q < PK_NACC; ++q)
    for (int v = 0; v < 16; ++v) acc[q][v] = 0.0f;
  for (int it = 0; it < rounds; ++it) {
#pragma unroll
    for (int q = 0; q < PK_NACC; ++q)
      acc[q] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[q], 0, 0, 0);
  }
  float t = 0.0f;
  for (int q = 0; q < PK_NACC; ++q) t += acc[q][lane & 15];
  if (t == -1.2345e-38f) sink[lane & 3] = t;
}

template <class F>
static hipError_t time_launches(hipStream_t s, int reps, float* ms, F&& launch) {
  hipEvent_t e0 = nullptr, e1 = nullptr;
  hipError_t e = hipEventCreate(&e0);
  if (e == hipSuccess) e = hipEventCreate(&e1);
  if (e == hipSuccess) {
    launch();                                      // warm-up
    e = hipEventRecord(e0, s);
  }
  for (int q = 0; q < reps && e == hipSuccess; ++q) {
    launch();
    e = hipGetLastError();
  }
  if (e == hipSuccess) e = hipEventRecord(e1, s);
  if (e == hipSuccess) e = hipEventSynchronize(e1);
  if (e == hipSuccess) e = hipEventElapsedTime(ms, e0, e1);
  if (e0) (void)hipEventDestroy(e0);
  if (e1) (void)hipEventDestroy(e1);
  return e;
}

}  // namespace slh

extern "C" {

int slh_peak_read(void* buf, int64_t bytes, int32_t reps, void* stream, double* gbs_out) {
  if (!buf || !gbs_out || bytes < 4096 || bytes % 16 != 0 || reps < 1 || reps > 1000 ||
      ((uintptr_t)buf) % 16 != 0)
    return SLH_EINVAL;
  int dev = 0, n_cu = 256;
  if (hipGetDevice(&dev) != hipSuccess) return SLH_EHIP;
  hipDeviceProp_t prop;
  if (hipGetDeviceProperties(&prop, dev) == hipSuccess) n_cu = prop.multiProcessorCount;
  const int64_t n4 = bytes / 16;
  const unsigned blocks = (unsigned)std::max<int64_t>(
      1, std::min<int64_t>((int64_t)16 * n_cu, (n4 + 4 * 512 - 1) / (4 * 512)));
  hipStream_t s = (hipStream_t)stream;
  (void)hipGetLastError();
  float ms = 0.f;
  const hipError_t e = slh::time_launches(s, reps, &ms, [&] {
    hipLaunchKernelGGL(slh::k_peak_read, dim3(blocks), dim3(512), 0, s, (const float4*)buf, n4,
                       (float*)buf);
  });
  if (e != hipSuccess || !(ms > 0.f)) return SLH_EHIP;
  *gbs_out = (double)bytes * reps / (1e-3 * ms) / 1e9;
  return SLH_OK;
}

int slh_peak_mfma(int32_t reps, void* sink, void* stream, double* tflops_out) {
  if (!tflops_out || !sink || reps < 1 || reps > 1000) return SLH_EINVAL;
  int dev = 0, n_cu = 256;
  if (hipGetDevice(&dev) != hipSuccess) return SLH_EHIP;
  hipDeviceProp_t prop;
  if (hipGetDeviceProperties(&prop, dev) == hipSuccess) n_cu = prop.multiProcessorCount;
  const int rounds = 4096;
  const unsigned blocks = (unsigned)(2 * n_cu);    // 8 waves per CU, two per SIMD
  hipStream_t s = (hipStream_t)stream;
  (void)hipGetLastError();
  float ms = 0.f;
  const hipError_t e = slh::time_launches(s, reps, &ms, [&] {
    hipLaunchKernelGGL(slh::k_peak_mfma, dim3(blocks), dim3(256), 0, s, rounds, (float*)sink);
  });
  if (e != hipSuccess || !(ms > 0.f)) return SLH_EHIP;
  const double flops = 2.0 * 32 * 32 * 16 * (double)slh::PK_NACC * rounds * (blocks * 4.0) * reps;
  *tflops_out = flops / (1e-3 * ms) / 1e12;
  return SLH_OK;
}

}  // extern "C"
