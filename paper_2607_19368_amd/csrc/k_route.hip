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

// Fused row norms and router partials for fp32 X, D <= 512 NW CPT (one read of
// X for both): workgroup (window, group of RT_RB rows) of NW waves covers every
// column, thread t columns 8 t + 512 NW c (c < CPT).  Rows go two at a time
// (the next two in flight): each thread's share of the row's two norms (|x|^2
// of the bf16-rounded values, which the feature map sees, and of the fp32
// values) is summed over the workgroup in a fixed order (wave butterfly, then
// the NW waves in order, through a double-buffered LDS slot: one barrier per two
// rows); the row's outputs are those of the row-norm kernel (|x|^2 of the bf16
// values, |x|, 1 / |x|, the feature-map scale, taken after the row loop from
// |x|^2 kept in LDS, and the bf16 copy of the row); S and U are accumulated for
// the thread's columns and written as the group's partial vectors, added over
// the groups in order by k_route_su.
constexpr int RT_RB = 256;                     // rows per workgroup

struct RtRaw { float4 lo, hi; };

__device__ __forceinline__ RtRaw rt_raw(const float* X, int64_t ldx, int64_t row, int col) {
  const float4* p = (const float4*)(X + row * ldx + col);
  return RtRaw{p[0], p[1]};
}

__device__ __forceinline__ void rt_unpack(const RtRaw& r, float (&x)[8]) {
  x[0] = r.lo.x; x[1] = r.lo.y; x[2] = r.lo.z; x[3] = r.lo.w;
  x[4] = r.hi.x; x[5] = r.hi.y; x[6] = r.hi.z; x[7] = r.hi.w;
}

template <int NW, int CPT>
__global__ __launch_bounds__(64 * NW) void k_route_norm_f32(
    const float* __restrict__ X, int64_t ldx, int L, int D, double inv2sqrtD, double sqrt2m,
    int gauss, double* __restrict__ nrm2_fm, double* __restrict__ nrm_x,
    double* __restrict__ inv_x, float* __restrict__ rowscale, uint16_t* __restrict__ Xb,
    double* __restrict__ psu) {
  constexpr int R = 2;                         // rows per batch
  constexpr int NV = 2;                        // norms per row: bf16 |x|^2, fp32 |x|^2
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
  RtRaw rc[R][CPT], rn[R][CPT];
  auto load = [&](RtRaw (&dst)[R][CPT], int b) {
#pragma unroll
    for (int e = 0; e < R; ++e)
#pragma unroll
      for (int c = 0; c < CPT; ++c) dst[e][c] = rt_raw(X, ldx, row0 + min(b + e, nrow - 1), col[c]);
  };
  load(rc, 0);
  // a row's values are unpacked from the raw registers twice (for |x|^2, then
  // for S and U) rather than kept as floats; columns past D are masked to 0
  auto values = [&](const RtRaw& r, int c, float (&v)[8]) {
    rt_unpack(r, v);
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
          const double hv = (double)bf16_to_f32(f32_to_bf16_rne(v[k]));
          sfm = fma(hv, hv, sfm);
          sx = fma((double)v[k], (double)v[k], sx);
        }
      }
      q[e * NV] = wave_sum_f64(sfm);
      q[e * NV + 1] = wave_sum_f64(sx);
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
        const double sfm = q[e * NV], sx = q[e * NV + 1];
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

// The same outputs for bf16 X, with the rows streamed through LDS instead of
// registers so that more of them are in flight: each thread's 16-byte pieces of
// a batch of R rows go straight from memory into its own slots of a ring of
// NS batches (direct-to-LDS loads), NS - 1 batches ahead of the one being
// summed; a thread reads back only what its own loads wrote, so a wait on its
// own load counter is the only synchronisation the ring needs.  Workgroup
// (window, group g): rows RT_RB g ... RT_RB (g + 1) - 1 of the window.
//
// Per batch: the thread's values, converted to double once, give its share of
// each row's |x|^2; the two rows' shares are summed over the wave together
// (rs_pair_sum) and over the NW waves in order through a double-buffered LDS
// slot (one barrier per batch, at the top of the next iteration, which then
// adds the values into S and U with the 1 / |x| of both rows taken by one
// square root and one division on the two halves of the wave).  |x|, 1 / |x|
// and the feature-map scale of the group's rows are written after the row loop
// from |x|^2 kept in LDS.  FULL: D == 512 NW CPT, every column in range.
typedef __attribute__((address_space(1))) const void* rs_gptr;
typedef __attribute__((address_space(3))) void* rs_lptr;

template <int N>
__device__ __forceinline__ void rs_wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt field");
  asm volatile("s_waitcnt vmcnt(%0)" ::"i"(N) : "memory");
}

// This thread's LPB pieces of a ring stage, at byte offsets k STRIDE from p,
// read with one wait for all of them.  Written as one asm statement because
// the compiler, unable to tell these reads from the direct-to-LDS writes still
// in flight, would otherwise wait for every load before them.
typedef unsigned rs_u32x4 __attribute__((ext_vector_type(4)));
template <int LPB, int STRIDE>
__device__ __forceinline__ void rs_read(const uint16_t* p, rs_u32x4 (&w)[LPB]) {
  const uint32_t a = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) uint16_t*)p;
  static_assert(LPB == 2 || LPB == 4 || LPB == 8, "unsupported piece count");
  static_assert((LPB - 1) * STRIDE < 65536, "offset field");
  if constexpr (LPB == 2)
    asm volatile("ds_read_b128 %0, %2\n\tds_read_b128 %1, %2 offset:%3\n\ts_waitcnt lgkmcnt(0)"
                 : "=&v"(w[0]), "=&v"(w[1]) : "v"(a), "i"(STRIDE) : "memory");
  else if constexpr (LPB == 8)
    asm volatile("ds_read_b128 %0, %8\n\tds_read_b128 %1, %8 offset:%9\n\t"
                 "ds_read_b128 %2, %8 offset:%10\n\tds_read_b128 %3, %8 offset:%11\n\t"
                 "ds_read_b128 %4, %8 offset:%12\n\tds_read_b128 %5, %8 offset:%13\n\t"
                 "ds_read_b128 %6, %8 offset:%14\n\tds_read_b128 %7, %8 offset:%15\n\t"
                 "s_waitcnt lgkmcnt(0)"
                 : "=&v"(w[0]), "=&v"(w[1]), "=&v"(w[2]), "=&v"(w[3]), "=&v"(w[4]), "=&v"(w[5]),
                   "=&v"(w[6]), "=&v"(w[7])
                 : "v"(a), "i"(STRIDE), "i"(2 * STRIDE), "i"(3 * STRIDE), "i"(4 * STRIDE),
                   "i"(5 * STRIDE), "i"(6 * STRIDE), "i"(7 * STRIDE)
                 : "memory");
  else
    asm volatile("ds_read_b128 %0, %4\n\tds_read_b128 %1, %4 offset:%5\n\t"
                 "ds_read_b128 %2, %4 offset:%6\n\tds_read_b128 %3, %4 offset:%7\n\t"
                 "s_waitcnt lgkmcnt(0)"
                 : "=&v"(w[0]), "=&v"(w[1]), "=&v"(w[2]), "=&v"(w[3])
                 : "v"(a), "i"(STRIDE), "i"(2 * STRIDE), "i"(3 * STRIDE) : "memory");
}

// Wave sums of a and b in a fixed order, both returned in every lane: one
// 32-lane trade leaves a's pair sums in lanes 0-31 and b's in 32-63; sums over
// each row of 16 lanes (lane i with i ^ 1, i ^ 2, 7 - i, 15 - i: every lane of
// the row ends with the same bits), read out of lanes 0 and 16 (a) and 32 and
// 48 (b).
__device__ __forceinline__ double rs_row_sum(double v) {
  v += dpp_f64<DPP_XOR1>(v);
  v += dpp_f64<DPP_XOR2>(v);
  v += dpp_f64<DPP_HALF_MIRROR>(v);
  v += dpp_f64<DPP_MIRROR>(v);
  return v;
}

__device__ __forceinline__ void rs_pair_sum(double a, double b, double& sa, double& sb) {
  const double v = rs_row_sum(swap32_add(a, b));
  sa = readlane_f64(v, 0) + readlane_f64(v, 16);
  sb = readlane_f64(v, 32) + readlane_f64(v, 48);
}

// The same for four values, returned in a, b, c, d: after the 32-lane trades of
// (a, b) and (c, d), a 16-lane trade leaves a, c, b, d in rows 0, 1, 2, 3.
__device__ __forceinline__ void rs_quad_sum(double& a, double& b, double& c, double& d) {
  const double v = rs_row_sum(swap16_add(swap32_add(a, b), swap32_add(c, d)));
  a = readlane_f64(v, 0);
  c = readlane_f64(v, 16);
  b = readlane_f64(v, 32);
  d = readlane_f64(v, 48);
}

template <int NW, int CPT, int R, int NS, bool FULL>
__global__ __launch_bounds__(64 * NW) void k_route_norm_stream(
    const uint16_t* __restrict__ X, int64_t ldx, int L, int D, double inv2sqrtD, double sqrt2m,
    int gauss, double* __restrict__ nrm2_fm, double* __restrict__ nrm_x,
    double* __restrict__ inv_x, float* __restrict__ rowscale, double* __restrict__ psu) {
  static_assert(R == 2 || R == 4, "rows per batch");
  constexpr int LPB = R * CPT;                   // loads per thread per batch of R rows
  constexpr int SLOT = NW * 64 * 8;              // one load of the workgroup (bf16 values)
  constexpr int STAGE = LPB * SLOT;
  constexpr int AHEAD = (NS - 1) * LPB;          // loads younger than the awaited batch
  __shared__ __attribute__((aligned(16))) uint16_t ring[NS * STAGE];
  __shared__ double red[2][NW][R];
  __shared__ double sq_l[RT_RB];
  const int win = blockIdx.x, g = blockIdx.y, G = gridDim.y, tid = threadIdx.x;
  const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int rbeg = g * RT_RB, nrow = min(RT_RB, L - rbeg);
  const int nb = (nrow + R - 1) / R;
  const uint16_t* xg = X + ((int64_t)win * L + rbeg) * ldx;
  int col[CPT];
  bool cin[CPT];
#pragma unroll
  for (int c = 0; c < CPT; ++c) {
    const int c8 = 8 * tid + 512 * NW * c;
    cin[c] = FULL || c8 < D;
    col[c] = min(c8, D - 8);
  }
  // batch j into ring stage j % RS_NS: load (e, c) of the workgroup fills slot
  // e CPT + c, this wave's 64 lanes at 1 KiB offset wave (a row past the
  // group's last is clamped to it and never summed)
  auto issue = [&](int j) {
    uint16_t* st = ring + (j % NS) * STAGE;
#pragma unroll
    for (int e = 0; e < R; ++e) {
      const uint16_t* xr = xg + (int64_t)min(R * j + e, nrow - 1) * ldx;
#pragma unroll
      for (int c = 0; c < CPT; ++c)
        __builtin_amdgcn_global_load_lds((rs_gptr)(xr + col[c]),
                                         (rs_lptr)(st + (e * CPT + c) * SLOT + wave * 512), 16, 0, 0);
    }
  };
  double xv[R][CPT][8];                          // the batch's values of this thread
  // wait for batch j (issued up to batch j + RS_NS - 1 while that exists), take
  // this thread's values of it and put the wave's shares of both rows' |x|^2
  // into red[j & 1][wave]
  auto fetch = [&](int j) {
    if (j + NS - 1 < nb) rs_wait_vm<AHEAD>();
    else rs_wait_vm<0>();
    rs_u32x4 raw[LPB];
    rs_read<LPB, SLOT * 2>(ring + (j % NS) * STAGE + tid * 8, raw);
    double p[R];
#pragma unroll
    for (int e = 0; e < R; ++e) {
      p[e] = 0.0;
#pragma unroll
      for (int c = 0; c < CPT; ++c) {
        const rs_u32x4 w = raw[e * CPT + c];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          float lo = __uint_as_float(w[q] << 16), hi = __uint_as_float(w[q] & 0xFFFF0000u);
          if constexpr (!FULL) {
            lo = cin[c] ? lo : 0.0f;
            hi = cin[c] ? hi : 0.0f;
          }
          xv[e][c][2 * q] = (double)lo;
          xv[e][c][2 * q + 1] = (double)hi;
        }
#pragma unroll
        for (int k = 0; k < 8; ++k) p[e] = fma(xv[e][c][k], xv[e][c][k], p[e]);
      }
    }
    if constexpr (R == 2) rs_pair_sum(p[0], p[1], p[0], p[1]);
    else rs_quad_sum(p[0], p[1], p[2], p[3]);
    if (lane == 0) {
#pragma unroll
      for (int e = 0; e < R; ++e) red[j & 1][wave][e] = p[e];
    }
  };
  double S[CPT][8], U[CPT][8];
#pragma unroll
  for (int c = 0; c < CPT; ++c)
#pragma unroll
    for (int k = 0; k < 8; ++k) S[c][k] = U[c][k] = 0.0;
#pragma unroll
  for (int j = 0; j < NS; ++j)
    if (j < nb) issue(j);
  fetch(0);
  for (int j = 0; j < nb; ++j) {
    // the waves' shares of batch j are in red[j & 1]: a barrier on the LDS
    // writes only (__syncthreads() would also wait for the ring loads in
    // flight), then the rows' |x|^2 in wave order
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
    double q[R];
#pragma unroll
    for (int e = 0; e < R; ++e) {
      q[e] = 0.0;
#pragma unroll
      for (int w8 = 0; w8 < NW; ++w8) q[e] += red[j & 1][w8][e];
    }
    // 1 / |x| of row e in lanes 64 e / R ... 64 (e + 1) / R - 1 of the wave
    double qh = q[0];
#pragma unroll
    for (int e = 1; e < R; ++e) qh = lane >= 64 * e / R ? q[e] : qh;
    const double nh = sqrt(qh);
    const double ih = nh > 0.0 ? 1.0 / nh : 0.0;
#pragma unroll
    for (int e = 0; e < R; ++e) {
      if (R * j + e < nrow) {
        const double inv = readlane_f64(ih, 64 * e / R);
#pragma unroll
        for (int c = 0; c < CPT; ++c)
#pragma unroll
          for (int k = 0; k < 8; ++k) {
            S[c][k] += xv[e][c][k];
            U[c][k] = fma(xv[e][c][k], inv, U[c][k]);
          }
        if (tid == 0) sq_l[R * j + e] = q[e];
      }
    }
    if (j + 1 < nb) {
      // batch j's stage is free (its values are in registers): refill it with
      // batch j + NS, then take batch j + 1
      if (j + NS < nb) issue(j + NS);
      fetch(j + 1);
    }
  }
  __syncthreads();
  for (int r = tid; r < nrow; r += 64 * NW) {
    const int64_t row = (int64_t)win * L + rbeg + r;
    const double sfm = sq_l[r];
    const double nx = sqrt(sfm);
    nrm2_fm[row] = sfm;
    nrm_x[row] = nx;
    inv_x[row] = nx > 0.0 ? 1.0 / nx : 0.0;
    const double sc = gauss ? 1.0 : exp(sfm * inv2sqrtD);
    rowscale[row] = (float)(sc * sqrt2m);
  }
  // the group's partial vectors, psu[((win G + g) 2 + {0: S, 1: U}) D + col],
  // turned around in the (now idle) ring so that each wave stores 1 KiB runs:
  // the wave's 512 consecutive values of a vector go to LDS as 8 per lane and
  // come back as 2 per lane from 4 consecutive 1 KiB quarters
  double* ps = psu + ((int64_t)win * G + g) * 2 * D;
  double* tw = (double*)ring + wave * 512;       // this wave's 4 KiB (ring >= 4 NW KiB)
  static_assert(NS * STAGE * 2 >= NW * 4096, "transpose space");
#pragma unroll
  for (int c = 0; c < CPT; ++c)
#pragma unroll
    for (int v = 0; v < 2; ++v) {
#pragma unroll
      for (int k = 0; k < 8; k += 2)
        *(double2*)(tw + 8 * lane + k) = v == 0 ? make_double2(S[c][k], S[c][k + 1])
                                                : make_double2(U[c][k], U[c][k + 1]);
      __builtin_amdgcn_wave_barrier();
      // the wave's columns: 8 (64 wave + lane') + 512 NW c, lane' < 64
      const int wcol = 512 * wave + 512 * NW * c;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int o = 128 * q + 2 * lane;          // value index within the wave's 512
        if (wcol + o < D) *(double2*)(ps + (int64_t)v * D + wcol + o) = *(const double2*)(tw + o);
      }
      __builtin_amdgcn_wave_barrier();
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
  if (dtype == 1)
    hipLaunchKernelGGL((k_route_norm_f32<NW, CPT>), grid, dim3(64 * NW), 0, s, (const float*)X, ldx,
                       L, D, inv2sqrtD, sqrt2m, gauss, nrm2_fm, nrm_x, inv_x, rowscale, Xb, psu);
  else if (D == 512 * NW * CPT)
    hipLaunchKernelGGL((k_route_norm_stream<NW, CPT, 2, 4, true>), grid, dim3(64 * NW), 0, s,
                       (const uint16_t*)X, ldx, L, D, inv2sqrtD, sqrt2m, gauss, nrm2_fm, nrm_x,
                       inv_x, rowscale, psu);
  else
    hipLaunchKernelGGL((k_route_norm_stream<NW, CPT, 2, 4, false>), grid, dim3(64 * NW), 0, s,
                       (const uint16_t*)X, ldx, L, D, inv2sqrtD, sqrt2m, gauss, nrm2_fm, nrm_x,
                       inv_x, rowscale, psu);
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
