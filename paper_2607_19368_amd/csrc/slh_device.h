// Device-side helpers shared by the HIP kernels (gfx950, wave64).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#define SLH_WAVE 64

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __uint_as_float(((uint32_t)b) << 16);
}

// float -> bf16 bits, round to nearest even (finite inputs)
__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// Wave sums (every lane active; the same bits in every lane): the 32- and
// 16-lane trades of v_permlane32_swap / v_permlane16_swap, then DPP within each
// row of 16 lanes (lane ^ 8, 7 - i, lane ^ 2, lane ^ 1); each step adds the same
// two values in both lanes of a pair.  No LDS round trips.
__device__ __forceinline__ double wave_sum_f64(double v);

__device__ __forceinline__ float wave_sum_f32(float v) {
  auto t32 = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = __uint_as_float(t32[0]) + __uint_as_float(t32[1]);
  auto t16 = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = __uint_as_float(t16[0]) + __uint_as_float(t16[1]);
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x128, 0xF, 0xF, false));
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x141, 0xF, 0xF, false));
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x4E, 0xF, 0xF, false));
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xB1, 0xF, 0xF, false));
  return v;
}

__device__ __forceinline__ int wave_sum_i32(int v) {
  auto t32 = __builtin_amdgcn_permlane32_swap((uint32_t)v, (uint32_t)v, false, false);
  v = (int)t32[0] + (int)t32[1];
  auto t16 = __builtin_amdgcn_permlane16_swap((uint32_t)v, (uint32_t)v, false, false);
  v = (int)t16[0] + (int)t16[1];
  v += __builtin_amdgcn_update_dpp(0, v, 0x128, 0xF, 0xF, false);
  v += __builtin_amdgcn_update_dpp(0, v, 0x141, 0xF, 0xF, false);
  v += __builtin_amdgcn_update_dpp(0, v, 0x4E, 0xF, 0xF, false);
  v += __builtin_amdgcn_update_dpp(0, v, 0xB1, 0xF, 0xF, false);
  return v;
}

// Block-wide sum of one double per thread; every thread gets the result.
// `red` must hold blockDim.x/64 doubles of shared memory.
__device__ __forceinline__ double block_sum_f64(double v, double* red) {
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6, nw = blockDim.x >> 6;
  v = wave_sum_f64(v);
  __syncthreads();
  if (lane == 0) red[wid] = v;
  __syncthreads();
  double s = 0.0;
  for (int w = 0; w < nw; ++w) s += red[w];
  return s;
}

// Lane exchanges of doubles without an LDS round trip (gfx950): DPP moves
// within rows of 16 lanes, the 32- and 16-lane trades of v_permlane32_swap and
// v_permlane16_swap, and lane reads into scalar registers.
__device__ __forceinline__ uint32_t f64_lo(double v) {
  return (uint32_t)(uint64_t)__double_as_longlong(v);
}
__device__ __forceinline__ uint32_t f64_hi(double v) {
  return (uint32_t)((uint64_t)__double_as_longlong(v) >> 32);
}
__device__ __forceinline__ double f64_of(uint32_t lo, uint32_t hi) {
  return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

// DPP controls used here: quad_perm [1, 0, 3, 2] (lane ^ 1), quad_perm
// [2, 3, 0, 1] (lane ^ 2), row_half_mirror (7 - i within 8 lanes), row_mirror
// (15 - i within 16), row_ror:8 (lane ^ 8 within 16).
constexpr int DPP_XOR1 = 0xB1, DPP_XOR2 = 0x4E, DPP_HALF_MIRROR = 0x141, DPP_MIRROR = 0x140,
              DPP_ROR8 = 0x128;

// The value of lane dpp(l) in lane l (every lane active).
template <int CTRL>
__device__ __forceinline__ double dpp_f64(double v) {
  const int lo = __builtin_amdgcn_update_dpp(0, (int)f64_lo(v), CTRL, 0xF, 0xF, false);
  const int hi = __builtin_amdgcn_update_dpp(0, (int)f64_hi(v), CTRL, 0xF, 0xF, false);
  return f64_of((uint32_t)lo, (uint32_t)hi);
}

// The value of lane l (wave-uniform).
__device__ __forceinline__ double readlane_f64(double v, int l) {
  return f64_of((uint32_t)__builtin_amdgcn_readlane((int)f64_lo(v), l),
                (uint32_t)__builtin_amdgcn_readlane((int)f64_hi(v), l));
}

// a + b after lanes 32-63 of a trade places with lanes 0-31 of b: lane l < 32
// gets a_l + a_(l+32), lane l >= 32 gets b_(l-32) + b_l.
__device__ __forceinline__ double swap32_add(double a, double b) {
  const auto lo = __builtin_amdgcn_permlane32_swap(f64_lo(a), f64_lo(b), false, false);
  const auto hi = __builtin_amdgcn_permlane32_swap(f64_hi(a), f64_hi(b), false, false);
  return f64_of(lo[0], hi[0]) + f64_of(lo[1], hi[1]);
}

// The same one level down: lanes 16-31 and 48-63 of a trade places with lanes
// 0-15 and 32-47 of b; lane l gets a_l + a_(l+16) where bit 4 of l is 0 and
// b_(l-16) + b_l where it is 1.
__device__ __forceinline__ double swap16_add(double a, double b) {
  const auto lo = __builtin_amdgcn_permlane16_swap(f64_lo(a), f64_lo(b), false, false);
  const auto hi = __builtin_amdgcn_permlane16_swap(f64_hi(a), f64_hi(b), false, false);
  return f64_of(lo[0], hi[0]) + f64_of(lo[1], hi[1]);
}

// Sum over each group of 8 lanes (lanes 8 k ... 8 k + 7), the same bits in all
// 8: lane i with 7 - i, then i ^ 2, then i ^ 1 (each step adds the same two
// values in both lanes of a pair).
__device__ __forceinline__ double oct_sum_f64(double v) {
  v += dpp_f64<DPP_HALF_MIRROR>(v);
  v += dpp_f64<DPP_XOR2>(v);
  v += dpp_f64<DPP_XOR1>(v);
  return v;
}

__device__ __forceinline__ double wave_sum_f64(double v) {
  v = swap32_add(v, v);
  v = swap16_add(v, v);
  v += dpp_f64<DPP_ROR8>(v);
  return oct_sum_f64(v);
}

// Sum 8 values over the 64 lanes of a wave without LDS round trips: four
// 32-lane trades (v_permlane32_swap), two 16-lane trades (v_permlane16_swap),
// an 8-lane exchange (DPP row_ror:8), then a sum over each 8-lane group.  On
// return lane l holds the full sum of value index ((l>>5)&1)*4 + ((l>>4)&1)*2 +
// ((l>>3)&1).  Every lane of the wave must be active.
__device__ __forceinline__ double wave_sum8_f64(const double (&v)[8]) {
  const int lane = threadIdx.x & 63;
  double w[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) w[e] = swap32_add(v[e], v[e + 4]);
  double x[2];
#pragma unroll
  for (int e = 0; e < 2; ++e) x[e] = swap16_add(w[e], w[e + 2]);
  const bool b8 = lane & 8;
  const double y = (b8 ? x[1] : x[0]) + dpp_f64<DPP_ROR8>(b8 ? x[0] : x[1]);
  return oct_sum_f64(y);
}
