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

// Fused row norms and router partials for D <= 512 NW CPT (one read of X for
// both): workgroup (window, group of RT_RB rows) of NW waves covers every
// column, thread t columns 8 t + 512 NW c (c < CPT).  Rows go R at a time (the next R in
// flight): each thread's share of |x|^2 is summed over the workgroup in a
// fixed order (wave butterfly, then the NW waves in order, through a
// double-buffered LDS slot: one barrier per R rows); the row's outputs are those of the row-norm
// kernel (|x|^2 of the bf16 values, |x|, 1 / |x|, the feature-map scale, taken
// after the row loop from |x|^2 kept in LDS, and, for fp32 X, the bf16 copy); S and U are accumulated for the thread's columns
// and written as the group's partial vectors, added over the groups in order
// by k_route_su.
constexpr int RT_RB = 256;                     // rows per workgroup

template <int DT>
struct RtRaw;
template <> struct RtRaw<0> { uint4 v; };
template <> struct RtRaw<1> { float4 lo, hi; };

template <int DT>
__device__ __forceinline__ RtRaw<DT> rt_raw(const void* X, int64_t ldx, int64_t row, int col) {
  RtRaw<DT> r;
  if constexpr (DT == 0) {
    r.v = *(const uint4*)((const uint16_t*)X + row * ldx + col);
  } else {
    const float4* p = (const float4*)((const float*)X + row * ldx + col);
    r.lo = p[0];
    r.hi = p[1];
  }
  return r;
}

template <int DT>
__device__ __forceinline__ void rt_unpack(const RtRaw<DT>& r, float (&x)[8]) {
  if constexpr (DT == 0) {
    const uint32_t w[4] = {r.v.x, r.v.y, r.v.z, r.v.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      x[2 * e] = __uint_as_float(w[e] << 16);
      x[2 * e + 1] = __uint_as_float(w[e] & 0xFFFF0000u);
    }
  } else {
    x[0] = r.lo.x; x[1] = r.lo.y; x[2] = r.lo.z; x[3] = r.lo.w;
    x[4] = r.hi.x; x[5] = r.hi.y; x[6] = r.hi.z; x[7] = r.hi.w;
  }
}

template <int DT, int NW, int CPT>
__global__ __launch_bounds__(64 * NW) void k_route_norm(
    const void* __restrict__ X, int64_t ldx, int L, int D, double inv2sqrtD, double sqrt2m,
    int gauss, double* __restrict__ nrm2_fm, double* __restrict__ nrm_x,
    double* __restrict__ inv_x, float* __restrict__ rowscale, uint16_t* __restrict__ Xb,
    double* __restrict__ psu) {
  constexpr int R = 2;                         // rows per batch
  constexpr int NV = (DT == 0) ? 1 : 2;        // norms per row: bf16 |x|^2 (and fp32 |x|^2)
  const int win = blockIdx.x, g = blockIdx.y, G = gridDim.y, tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int rbeg = g * RT_RB, nrow = min(RT_RB, L - rbeg);
  const int64_t row0 = (int64_t)win * L + rbeg;
  int col[CPT];
  bool cin[CPT];
#pragma unroll
  for (int c = 0; c < CPT; ++c) {
    const int c8 = 8 * tid + 512 * NW * c;
    cin[c] = c8 < D;
    col[c] = min(c8, D - 8);
  }
  double S[CPT][8], U[CPT][8];
#pragma unroll
  for (int c = 0; c < CPT; ++c)
#pragma unroll
    for (int k = 0; k < 8; ++k) S[c][k] = U[c][k] = 0.0;
  __shared__ double red[2][NW][R * NV];
  __shared__ double sq_l[RT_RB];
  RtRaw<DT> rc[R][CPT], rn[R][CPT];
  auto load = [&](RtRaw<DT> (&dst)[R][CPT], int b) {
#pragma unroll
    for (int e = 0; e < R; ++e)
#pragma unroll
      for (int c = 0; c < CPT; ++c) dst[e][c] = rt_raw<DT>(X, ldx, row0 + min(b + e, nrow - 1), col[c]);
  };
  load(rc, 0);
  // a row's values are unpacked from the raw registers twice (for |x|^2, then
  // for S and U) rather than kept as floats; columns past D are masked to 0
  auto values = [&](const RtRaw<DT>& r, int c, float (&v)[8]) {
    rt_unpack<DT>(r, v);
#pragma unroll
    for (int k = 0; k < 8; ++k) v[k] = cin[c] ? v[k] : 0.0f;
  };
  int par = 0;
  for (int b = 0; b < nrow; b += R) {
    if (b + R < nrow) load(rn, b + R);
    double q[R * NV];
#pragma unroll
    for (int e = 0; e < R; ++e) {
      double sfm = 0.0, sx = 0.0;
#pragma unroll
      for (int c = 0; c < CPT; ++c) {
        float v[8];
        values(rc[e][c], c, v);
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          if constexpr (DT == 0) {
            sfm = fma((double)v[k], (double)v[k], sfm);
          } else {
            const double hv = (double)bf16_to_f32(f32_to_bf16_rne(v[k]));
            sfm = fma(hv, hv, sfm);
            sx = fma((double)v[k], (double)v[k], sx);
          }
        }
      }
      q[e * NV] = wave_sum_f64(sfm);
      if constexpr (NV == 2) q[e * NV + 1] = wave_sum_f64(sx);
    }
    if (lane == 0) {
#pragma unroll
      for (int v = 0; v < R * NV; ++v) red[par][wave][v] = q[v];
    }
    __syncthreads();
#pragma unroll
    for (int v = 0; v < R * NV; ++v) {
      double t = 0.0;
#pragma unroll
      for (int w8 = 0; w8 < NW; ++w8) t += red[par][w8][v];
      q[v] = t;
    }
    par ^= 1;
#pragma unroll
    for (int e = 0; e < R; ++e) {
      if (b + e < nrow) {
        const double sfm = q[e * NV], sx = (NV == 2) ? q[e * NV + 1] : sfm;
        const double nx = sqrt(sx);
        const double inv = nx > 0.0 ? 1.0 / nx : 0.0;
        const int64_t row = row0 + b + e;
#pragma unroll
        for (int c = 0; c < CPT; ++c) {
          float v[8];
          values(rc[e][c], c, v);
#pragma unroll
          for (int k = 0; k < 8; ++k) {
            S[c][k] += (double)v[k];
            U[c][k] = fma((double)v[k], inv, U[c][k]);
          }
          if constexpr (DT == 1) {
            if (cin[c]) {
              uint16_t hb[8];
#pragma unroll
              for (int k = 0; k < 8; ++k) hb[k] = f32_to_bf16_rne(v[k]);
              uint4 pk;
              pk.x = (uint32_t)hb[0] | ((uint32_t)hb[1] << 16);
              pk.y = (uint32_t)hb[2] | ((uint32_t)hb[3] << 16);
              pk.z = (uint32_t)hb[4] | ((uint32_t)hb[5] << 16);
              pk.w = (uint32_t)hb[6] | ((uint32_t)hb[7] << 16);
              *(uint4*)(Xb + row * (int64_t)D + col[c]) = pk;
            }
          }
        }
        if (tid == 0) {
          nrm2_fm[row] = sfm;
          nrm_x[row] = nx;
          inv_x[row] = inv;
          sq_l[b + e] = sfm;                       // feature-map scale after the loop
        }
      }
    }
#pragma unroll
    for (int e = 0; e < R; ++e)
#pragma unroll
      for (int c = 0; c < CPT; ++c) rc[e][c] = rn[e][c];
  }
  // feature-map scales of the group's rows (the exp kept out of the row loop)
  __syncthreads();
  for (int r = tid; r < nrow; r += 64 * NW) {
    const double sc = gauss ? 1.0 : exp(sq_l[r] * inv2sqrtD);
    rowscale[row0 + r] = (float)(sc * sqrt2m);
  }
  // partial vectors of the group: psu[((win G + g) 2 + {0: S, 1: U}) D + col]
  double* ps = psu + ((int64_t)win * G + g) * 2 * D;
#pragma unroll
  for (int c = 0; c < CPT; ++c) {
    if (cin[c]) {
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        ps[col[c] + k] = S[c][k];
        ps[D + col[c] + k] = U[c][k];
      }
    }
  }
}

// (window, slice of 64 columns), one lane per column: S and U summed over the
// row groups in order, then the slice's U.S and |S|^2 (wave butterfly)
__global__ __launch_bounds__(64) void k_route_su(const double* __restrict__ psu, int G, int D,
                                                 double* __restrict__ part) {
  const int win = blockIdx.x, cs = blockIdx.y, lane = threadIdx.x;
  const int col = cs * RT_COLS + lane;
  const int cc = min(col, D - 1);
  double St = 0.0, Ut = 0.0;
  for (int g = 0; g < G; ++g) {
    const double* ps = psu + ((int64_t)win * G + g) * 2 * D;
    St += ps[cc];
    Ut += ps[D + cc];
  }
  const bool in = col < D;
  double dot = in ? Ut * St : 0.0, ss = in ? St * St : 0.0;
  dot = wave_sum_f64(dot);
  ss = wave_sum_f64(ss);
  if (lane == 0) {
    part[((int64_t)win * gridDim.y + cs) * 2 + 0] = dot;
    part[((int64_t)win * gridDim.y + cs) * 2 + 1] = ss;
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

int route_norm_groups(int L, int D) { return D <= 4096 ? (L + RT_RB - 1) / RT_RB : 0; }

template <int NW, int CPT>
static void launch_route_norm(int dtype, dim3 grid, hipStream_t s, const void* X, int64_t ldx,
                              int L, int D, double inv2sqrtD, double sqrt2m, int gauss,
                              double* nrm2_fm, double* nrm_x, double* inv_x, float* rowscale,
                              uint16_t* Xb, double* psu) {
  if (dtype == 0)
    hipLaunchKernelGGL((k_route_norm<0, NW, CPT>), grid, dim3(64 * NW), 0, s, X, ldx, L, D, inv2sqrtD,
                       sqrt2m, gauss, nrm2_fm, nrm_x, inv_x, rowscale, Xb, psu);
  else
    hipLaunchKernelGGL((k_route_norm<1, NW, CPT>), grid, dim3(64 * NW), 0, s, X, ldx, L, D, inv2sqrtD,
                       sqrt2m, gauss, nrm2_fm, nrm_x, inv_x, rowscale, Xb, psu);
}

hipError_t launch_route_norm_scores(const void* X, int dtype, int64_t ldx, int n_win, int L,
                                    int D, int m, int gauss, double* nrm2_fm, double* nrm_x,
                                    double* inv_x, float* rowscale, uint16_t* Xb, double* psu,
                                    double* part, double* scores, hipStream_t s) {
  (void)hipGetLastError();
  if (n_win <= 0) return hipSuccess;
  const int G = route_norm_groups(L, D);
  if (G < 1 || D % 8 != 0 || D < 8) return hipErrorInvalidValue;
  const double inv2sqrtD = 1.0 / (2.0 * sqrt((double)D));
  const double sqrt2m = sqrt(2.0 / (double)m);
  const dim3 grid(n_win, G);
  // up to 2048 columns one chunk per thread on D / 512 waves; wider rows two
  // chunks on 4 waves (measured faster than one chunk on 8 waves at D = 4096)
  if (D <= 512) launch_route_norm<1, 1>(dtype, grid, s, X, ldx, L, D, inv2sqrtD, sqrt2m, gauss, nrm2_fm, nrm_x, inv_x, rowscale, Xb, psu);
  else if (D <= 1024) launch_route_norm<2, 1>(dtype, grid, s, X, ldx, L, D, inv2sqrtD, sqrt2m, gauss, nrm2_fm, nrm_x, inv_x, rowscale, Xb, psu);
  else if (D <= 2048) launch_route_norm<4, 1>(dtype, grid, s, X, ldx, L, D, inv2sqrtD, sqrt2m, gauss, nrm2_fm, nrm_x, inv_x, rowscale, Xb, psu);
  else launch_route_norm<4, 2>(dtype, grid, s, X, ldx, L, D, inv2sqrtD, sqrt2m, gauss, nrm2_fm, nrm_x, inv_x, rowscale, Xb, psu);
  const int ncs = route_slices(D);
  hipLaunchKernelGGL(k_route_su, dim3(n_win, ncs), dim3(64), 0, s, psu, G, D, part);
  hipLaunchKernelGGL(k_route_final, dim3(n_win), dim3(64), 0, s, part, ncs, L, scores);
  return hipGetLastError();
}

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
