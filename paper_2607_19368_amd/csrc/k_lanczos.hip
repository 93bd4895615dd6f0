// Implicit Lanczos with full re-orthogonalization (Algorithm 2; operator of
// Eq. 4, A v = Phi (Phi^T v), never forming the N x N kernel).
//
// Each window runs its own recurrence; all windows advance in lockstep (grid
// dimension y = window).  Vectors and every reduction are fp64; Phi is fp32.
//
// Step j keeps q_j (Q[j], length L) and t_j = Phi^T q_j (T[j], length m) and
// runs four kernels:
//   phit    partials of Phi^T v, v = q_0 (j = 0) or z1 of step j-1 (the vector
//           after the first Gram-Schmidt pass), over (row group, 256-column
//           slice) blocks; the first blocks of the launch reduce the partials
//           of h2 = Q^T z1 and |z1|^2 of step j-1.
//   finish  beta_{j-1} = |z1 - Q h2| = sqrt(|z1|^2 - |h2|^2) (Q orthonormal),
//           the breakdown test, and t_j = (Phi^T z1 - sum_k h2_k t_k) / beta
//           (the second Gram-Schmidt pass applied in feature space; its
//           coefficients h2 are at rounding level).
//   phiu    u = Phi t_j (= A q_j) over row blocks; the first blocks of the
//           launch form h1 = Q_j^T u as t_k^T t_j (k <= j), the same inner
//           products taken in feature space, so no pass over Q is needed.
//   orth    per 32 rows: q_j = (z1 - Q_{j-1} h2) / beta (second pass in row
//           space, stored as Q[j]); alpha_j = h1_j = q_j^T A q_j;
//           z1 = u - Q_j h1 (first classical Gram-Schmidt pass of step j);
//           partials of h2 = Q_j^T z1 and |z1|^2.  One read of Q_j feeds both
//           the q_j update and z1.
// Phi is streamed twice per step: Phi^T z1 is always streamed.  (Forming
// Phi^T q_{j+1} from Phi^T u through the whole three-term recurrence would save
// a pass but multiplies rounding errors by alpha_j / beta_j every step.)  All
// partial sums are combined in a fixed order, so results are bitwise
// reproducible.  alpha_j and beta_j are those of Algorithm 2: alpha_j before any
// subtraction, beta_j the norm after re-orthogonalization.
#include "slh_device.h"
#include "slh_internal.h"

#include <hip/hip_ext.h>

#include <algorithm>

namespace slh {

// Sum 8 values over the 64 lanes of a wave with 10 shuffles.  On return lane l
// holds the full sum of value index ((l>>5)&1)*4 + ((l>>4)&1)*2 + ((l>>3)&1).
__device__ __forceinline__ double wave_sum8_f64(const double (&v)[8]) {
  const int lane = threadIdx.x & 63;
  double w[4];
  const bool b32 = lane & 32;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    double keep = b32 ? v[e + 4] : v[e];
    double send = b32 ? v[e] : v[e + 4];
    w[e] = keep + __shfl_xor(send, 32, 64);
  }
  double x[2];
  const bool b16 = lane & 16;
#pragma unroll
  for (int e = 0; e < 2; ++e) {
    double keep = b16 ? w[e + 2] : w[e];
    double send = b16 ? w[e] : w[e + 2];
    x[e] = keep + __shfl_xor(send, 16, 64);
  }
  const bool b8 = lane & 8;
  double y = (b8 ? x[1] : x[0]) + __shfl_xor(b8 ? x[0] : x[1], 8, 64);
  y += __shfl_xor(y, 4, 64);
  y += __shfl_xor(y, 2, 64);
  y += __shfl_xor(y, 1, 64);
  return y;
}

// The same over each half wave (lanes 0-31 and 32-63 separately): lane l holds
// the half-wave sum of value index ((l>>4)&1)*4 + ((l>>3)&1)*2 + ((l>>2)&1).
__device__ __forceinline__ double half_sum8_f64(const double (&v)[8]) {
  const int lane = threadIdx.x & 63;
  double w[4];
  const bool b16 = lane & 16;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    double keep = b16 ? v[e + 4] : v[e];
    double send = b16 ? v[e] : v[e + 4];
    w[e] = keep + __shfl_xor(send, 16, 64);
  }
  double x[2];
  const bool b8 = lane & 8;
#pragma unroll
  for (int e = 0; e < 2; ++e) {
    double keep = b8 ? w[e + 2] : w[e];
    double send = b8 ? w[e] : w[e + 2];
    x[e] = keep + __shfl_xor(send, 8, 64);
  }
  const bool b4 = lane & 4;
  double y = (b4 ? x[1] : x[0]) + __shfl_xor(b4 ? x[0] : x[1], 4, 64);
  y += __shfl_xor(y, 2, 64);
  y += __shfl_xor(y, 1, 64);
  return y;
}

// Sum of src[g * ld] over g < G with 8 loads in flight (fixed order).
__device__ __forceinline__ double sum_strided(const double* __restrict__ src, int64_t ld, int G) {
  double acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  int g = 0;
  for (; g + 8 <= G; g += 8) {
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] += src[(int64_t)(g + e) * ld];
  }
#pragma unroll
  for (int e = 0; e < 7; ++e)
    if (g + e < G) acc[e] += src[(int64_t)(g + e) * ld];
  return ((acc[0] + acc[1]) + (acc[2] + acc[3])) + ((acc[4] + acc[5]) + (acc[6] + acc[7]));
}

// Column reduction by one block of NT threads: returns, in the threads with
// threadIdx.x < CPB, sum_{g<G} src[g*ld + c0 + threadIdx.x] (0 past ncol);
// CPB columns x (NT / CPB) partial lanes, fixed order.  All threads must call it.
template <int CPB, int NT>
__device__ __forceinline__ double block_colsum(const double* __restrict__ src, int64_t ld, int G,
                                               int c0, int ncol) {
  constexpr int PL = NT / CPB;
  __shared__ double red[PL][CPB + 1];
  const int tid = threadIdx.x, cl = tid % CPB, pl = tid / CPB;
  const int col = c0 + cl;
  double acc = 0.0;
  if (col < ncol) {
    const int cnt = (G - pl + PL - 1) / PL;
    acc = sum_strided(src + (int64_t)pl * ld + col, (int64_t)PL * ld, cnt > 0 ? cnt : 0);
  }
  red[pl][cl] = acc;
  __syncthreads();
  double t = 0.0;
  if (tid < CPB && col < ncol) {
    for (int p = 0; p < PL; ++p) t += red[p][cl];
  }
  __syncthreads();
  return t;
}

// ---------------------------------------------------------------------------
// phit: blocks [0, nx) reduce h2 (k < j) and |z1|^2 of step j-1 over the orth
// blocks; the rest own (row group rg, 256-column slice sl): each of the 8
// waves streams rows r0 + wave + 8 q (q < RWA) of the slice, lane = 4 columns
// (one float4), 8 rows in flight plus the next 8.  Loads are unconditional
// (row clamped into the group); rows past the group carry weight 0.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(512) void k_lz_phit(LanczosWS w, int j) {
  const int a = blockIdx.y;
  if (w.stop[a]) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int L = w.L, m = w.m, hs = w.ldq + 1;
  const int nx = (j > 0) ? (j + 15) / 16 + 1 : 0;
  int g = blockIdx.x;
  if (g < nx) {
    const double* hp = w.H2part + (int64_t)a * w.G3 * hs;
    double* dst = w.H2 + (int64_t)a * hs;
    if (g == nx - 1) {                         // |z1|^2 (slot ldq)
      const double v = block_colsum<1, 512>(hp + w.ldq, hs, w.G3, 0, 1);
      if (tid == 0) dst[w.ldq] = v;
    } else {
      const int c0 = g * 16;
      const double v = block_colsum<16, 512>(hp, hs, w.G3, c0, j);
      if (tid < 16 && c0 + tid < j) dst[c0 + tid] = v;
    }
    return;
  }
  g -= nx;
  const int ns = m >> 8;
  const int sl = g % ns, rg = g / ns;
  const int r0 = rg * w.RBA;
  const int r1 = min(L, r0 + w.RBA);
  const float* base = w.Phi + (int64_t)a * L * m + sl * 256 + 4 * lane;
  const double* vsrc = (j == 0) ? (w.Q + (int64_t)a * w.ldq * L) : (w.Z1 + (int64_t)a * L);
  double s0 = 0.0, s1 = 0.0, s2 = 0.0, s3 = 0.0;
  float4 vc[8], vn[8];
  auto load8 = [&](float4 (&dst)[8], int b) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int i = min(r0 + wave + 8 * (8 * b + e), r1 - 1);
      dst[e] = *(const float4*)(base + (int64_t)i * m);
    }
  };
  const int nb = w.RWA / 8;
  load8(vc, 0);
  for (int b = 0; b < nb; ++b) {
    if (b + 1 < nb) load8(vn, b + 1);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int i = r0 + wave + 8 * (8 * b + e);
      const double vi = vsrc[min(i, r1 - 1)];
      const double qi = (i < r1) ? vi : 0.0;
      s0 = fma((double)vc[e].x, qi, s0);
      s1 = fma((double)vc[e].y, qi, s1);
      s2 = fma((double)vc[e].z, qi, s2);
      s3 = fma((double)vc[e].w, qi, s3);
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) vc[e] = vn[e];
  }
  __shared__ double cred[8][257];
  cred[wave][4 * lane + 0] = s0;
  cred[wave][4 * lane + 1] = s1;
  cred[wave][4 * lane + 2] = s2;
  cred[wave][4 * lane + 3] = s3;
  __syncthreads();
  if (tid < 256) {
    double t = 0.0;
#pragma unroll
    for (int q = 0; q < 8; ++q) t += cred[q][tid];
    w.Spart[((int64_t)a * w.GA + rg) * m + sl * 256 + tid] = t;
  }
}

// ---------------------------------------------------------------------------
// finish: beta_{j-1}, breakdown, and t_j on 16 columns per block (256 threads:
// 16 columns x 16 partial lanes).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_lz_finish(LanczosWS w, int j) {
  const int a = blockIdx.y, g = blockIdx.x, tid = threadIdx.x;
  if (w.stop[a]) return;
  const int m = w.m, hs = w.ldq + 1;
  __shared__ double h2[264];
  __shared__ double sh;
  __shared__ double red[4];
  double inv = 1.0;
  if (j > 0) {
    const double* H2 = w.H2 + (int64_t)a * hs;
    double hh = 0.0;
    for (int k = tid; k < j; k += 256) {
      const double v = H2[k];
      h2[k] = v;
      hh = fma(v, v, hh);
    }
    hh = block_sum_f64(hh, red);
    if (tid == 0) {
      const double b2 = H2[w.ldq] - hh;       // |z1 - Q h2|^2 for orthonormal Q
      const double beta = b2 > 0.0 ? sqrt(b2) : 0.0;
      const bool brk = !(beta > w.tol * w.amax[a]);
      sh = brk ? 0.0 : beta;
      if (g == 0) {
        w.beta[(int64_t)a * w.n_it + j - 1] = beta;
        if (brk) w.stop[a] = 1;                // n_eff stays j
      }
    }
    __syncthreads();
    if (sh == 0.0) return;
    inv = 1.0 / sh;
  }
  const int cl = tid & 15, pl = tid >> 4;
  const int c = g * 16 + cl;
  const int cc = min(c, m - 1);
  const double* Sp = w.Spart + (int64_t)a * w.GA * m + cc;
  const int cnt = (w.GA - pl + 15) / 16;
  const double s = sum_strided(Sp + (int64_t)pl * m, (int64_t)16 * m, cnt > 0 ? cnt : 0);
  double corr = 0.0;
  if (j > 0) {
    const double* Ta = w.T + (int64_t)a * w.ldq * m + cc;
    double acc[4] = {0, 0, 0, 0};
    int k = pl;
    for (; k + 48 < j; k += 64) {
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[e] = fma(Ta[(int64_t)(k + 16 * e) * m], h2[k + 16 * e], acc[e]);
    }
    for (; k < j; k += 16) acc[0] = fma(Ta[(int64_t)k * m], h2[k], acc[0]);
    corr = (acc[0] + acc[1]) + (acc[2] + acc[3]);
  }
  __shared__ double rs[16][17], rc[16][17];
  rs[pl][cl] = s;
  rc[pl][cl] = corr;
  __syncthreads();
  if (tid < 16 && c < m) {
    double S = 0.0, C = 0.0;
    for (int p = 0; p < 16; ++p) {
      S += rs[p][cl];
      C += rc[p][cl];
    }
    w.T[((int64_t)a * w.ldq + j) * m + c] = (j > 0) ? (S - C) * inv : S;
  }
}

// ---------------------------------------------------------------------------
// phiu: blocks [0, nx) form h1_k = t_k^T t_j, k <= j (one wave per k); the
// rest compute u = Phi t_j on RBB = RP * RPT rows each.  A row is covered by M4
// threads (4 columns each); every thread keeps its partial dot of each row it
// streams and one block-level reduction at the end gives u.
// ---------------------------------------------------------------------------
template <int M4>
__global__ __launch_bounds__(512) void k_lz_phiu(LanczosWS w, int j) {
  constexpr int RP = 512 / M4;
  constexpr int WPR = M4 >= 64 ? M4 / 64 : 1;     // waves per row group
  constexpr int MAXR = 32;                        // rows per thread kept (RPT <= 32)
  const int a = blockIdx.y;
  if (w.stop[a]) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int L = w.L, m = w.m;
  const double* Ta = w.T + (int64_t)a * w.ldq * m;
  const double* tj = Ta + (int64_t)j * m;
  const int nx = (j + 8) / 8;
  int g = blockIdx.x;
  if (g < nx) {
    const int k = g * 8 + wave;
    if (k > j) return;
    const double* tk = Ta + (int64_t)k * m;
    double acc[4] = {0, 0, 0, 0};
    for (int c0 = 0; c0 < m; c0 += 256) {      // m is a multiple of 256
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[e] = fma(tk[c0 + 64 * e + lane], tj[c0 + 64 * e + lane], acc[e]);
    }
    double v = (acc[0] + acc[1]) + (acc[2] + acc[3]);
    v = wave_sum_f64(v);
    if (lane == 0) w.H1[(int64_t)a * (w.ldq + 1) + k] = v;
    return;
  }
  g -= nx;
  const int r0 = g * w.RBB;
  const int r1 = min(L, r0 + w.RBB);
  const float* Phi = w.Phi + (int64_t)a * L * m;
  __shared__ double ured[8][MAXR];
  const int c4 = tid % M4, rs = tid / M4;
  const bool cin = 4 * c4 < m;
  const int cc = min(c4, m / 4 - 1);
  double t0 = tj[4 * cc + 0], t1 = tj[4 * cc + 1], t2 = tj[4 * cc + 2], t3 = tj[4 * cc + 3];
  if (!cin) t0 = t1 = t2 = t3 = 0.0;
  const float* base = Phi + 4 * cc;
  float4 vc[8], vn[8];
  auto load8 = [&](float4 (&dst)[8], int b) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int i = min(r0 + rs + RP * (8 * b + e), r1 - 1);
      dst[e] = *(const float4*)(base + (int64_t)i * m);
    }
  };
  double p[MAXR];
  const int nb = w.RPT / 8;
  load8(vc, 0);
#pragma unroll
  for (int b = 0; b < MAXR / 8; ++b) {
    if (b < nb) {
      if (b + 1 < nb) load8(vn, b + 1);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        double d = (double)vc[e].x * t0;
        d = fma((double)vc[e].y, t1, d);
        d = fma((double)vc[e].z, t2, d);
        p[8 * b + e] = fma((double)vc[e].w, t3, d);
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) vc[e] = vn[e];
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) p[8 * b + e] = 0.0;
    }
  }
  // reduce p[q] over the wave (8 rows per butterfly), then over the WPR waves of a row group
#pragma unroll
  for (int q0 = 0; q0 < MAXR; q0 += 8) {
    if (q0 < w.RPT) {
      double v8[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) v8[e] = p[q0 + e];
      const double tot = wave_sum8_f64(v8);
      const int idx = ((lane >> 5) & 1) * 4 + ((lane >> 4) & 1) * 2 + ((lane >> 3) & 1);
      if ((lane & 7) == 0) ured[wave][q0 + idx] = tot;
    }
  }
  __syncthreads();
  for (int x = tid; x < RP * w.RPT; x += 512) {
    const int rsx = x / w.RPT, q = x % w.RPT;
    double u = 0.0;
    for (int ww = 0; ww < WPR; ++ww) u += ured[rsx * WPR + ww][q];
    const int i = r0 + rsx + RP * q;
    if (i < r1) w.U[(int64_t)a * L + i] = u;
  }
}

// ---------------------------------------------------------------------------
// orth on 32 rows per block (256 threads = 32 rows x 8 k-groups).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_lz_orth(LanczosWS w, int j) {
  const int a = blockIdx.y, g = blockIdx.x;
  if (w.stop[a]) return;
  const int tid = threadIdx.x, lane = tid & 63;
  const int L = w.L, hs = w.ldq + 1;
  const int rl = tid & 31, kg = tid >> 5;
  const int r0 = g * 32;
  const int i = r0 + rl;
  const int ic = min(i, L - 1);
  const double* Qa = w.Q + (int64_t)a * w.ldq * L;
  __shared__ double h1[264], h2[264];
  __shared__ double rq[8][33], rz[8][33];
  __shared__ double sz[32], sq[32];
  for (int k = tid; k <= j; k += 256) h1[k] = w.H1[(int64_t)a * hs + k];
  for (int k = tid; k < j; k += 256) h2[k] = w.H2[(int64_t)a * hs + k];
  __syncthreads();
  if (g == 0 && tid == 0) {
    w.alpha[(int64_t)a * w.n_it + j] = h1[j];
    w.amax[a] = fmax(j ? w.amax[a] : 0.0, fabs(h1[j]));
    w.neff[a] = j + 1;
  }
  // one pass over Q_{j-1} on this block's rows: Q h2 (q_j update) and Q h1 (z1)
  {
    double aq[4] = {0, 0, 0, 0}, az[4] = {0, 0, 0, 0};
    int k = kg;
    for (; k + 24 < j; k += 32) {
      double qv[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) qv[e] = Qa[(int64_t)(k + 8 * e) * L + ic];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        aq[e] = fma(qv[e], h2[k + 8 * e], aq[e]);
        az[e] = fma(qv[e], h1[k + 8 * e], az[e]);
      }
    }
    for (; k < j; k += 8) {
      const double qv = Qa[(int64_t)k * L + ic];
      aq[0] = fma(qv, h2[k], aq[0]);
      az[0] = fma(qv, h1[k], az[0]);
    }
    rq[kg][rl] = (aq[0] + aq[1]) + (aq[2] + aq[3]);
    rz[kg][rl] = (az[0] + az[1]) + (az[2] + az[3]);
  }
  __syncthreads();
  if (tid < 32) {
    double z = 0.0, q = 0.0;
    if (i < L) {
      if (j > 0) {
        double sub = 0.0;
        for (int p = 0; p < 8; ++p) sub += rq[p][rl];
        q = (w.Z1[(int64_t)a * L + i] - sub) / w.beta[(int64_t)a * w.n_it + j - 1];
        w.Q[((int64_t)a * w.ldq + j) * L + i] = q;
      } else {
        q = Qa[i];
      }
      double zs = 0.0;
      for (int p = 0; p < 8; ++p) zs += rz[p][rl];
      z = w.U[(int64_t)a * L + i] - fma(q, h1[j], zs);
      w.Z1[(int64_t)a * L + i] = z;
    }
    sz[rl] = z;
    sq[rl] = q;
  }
  __syncthreads();
  // partials of h2_k = sum over these rows of Q[k] z1, k <= j: thread (row, k-group),
  // k = kb + 8 kg + e; 8 products per thread, summed over the 32 rows of each half wave
  double* hp = w.H2part + ((int64_t)a * w.G3 + g) * hs;
  const double zl = sz[rl];
  for (int kb = 0; kb <= j; kb += 64) {
    double v8[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int k = kb + 8 * kg + e;
      const double qv = (k < j) ? Qa[(int64_t)max(0, min(k, j - 1)) * L + ic] : sq[rl];
      v8[e] = (k <= j) ? qv * zl : 0.0;
    }
    const double tot = half_sum8_f64(v8);
    const int k = kb + 8 * kg + ((lane >> 4) & 1) * 4 + ((lane >> 3) & 1) * 2 + ((lane >> 2) & 1);
    if ((lane & 3) == 0 && k <= j) hp[k] = tot;
  }
  if (tid == 0) {
    double nz = 0.0;
    for (int p = 0; p < 32; ++p) nz = fma(sz[p], sz[p], nz);
    hp[w.ldq] = nz;
  }
}

// beta of the last step (reported; T does not use it): one block per window
// reduces h2 and |z1|^2 of the last orthogonalisation.
__global__ __launch_bounds__(256) void k_lz_last_beta(LanczosWS w) {
  const int a = blockIdx.x, tid = threadIdx.x;
  if (w.stop[a]) return;
  const int j = w.n_it, hs = w.ldq + 1;
  const double* hp = w.H2part + (int64_t)a * w.G3 * hs;
  __shared__ double red[4];
  double hh = 0.0;
  for (int c0 = 0; c0 < j; c0 += 16) {
    const double v = block_colsum<16, 256>(hp, hs, w.G3, c0, j);
    if (tid < 16) hh = fma(v, v, hh);
  }
  const double nz = block_colsum<1, 256>(hp + w.ldq, hs, w.G3, 0, 1);
  hh = block_sum_f64(hh, red);
  if (tid == 0) {
    const double b2 = nz - hh;
    w.beta[(int64_t)a * w.n_it + j - 1] = b2 > 0.0 ? sqrt(b2) : 0.0;
  }
}

// q_0 of every active window into Q[a][0]; clear the per-window state.
__global__ void k_lz_start(LanczosWS w, const double* __restrict__ q1) {
  const int a = blockIdx.y;
  for (int i = blockIdx.x * 256 + threadIdx.x; i < w.L; i += gridDim.x * 256)
    w.Q[(int64_t)a * w.ldq * w.L + i] = q1[(int64_t)a * w.L + i];
  if (blockIdx.x == 0 && threadIdx.x < w.n_it) {
    w.alpha[(int64_t)a * w.n_it + threadIdx.x] = 0.0;
    w.beta[(int64_t)a * w.n_it + threadIdx.x] = 0.0;
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    w.stop[a] = 0;
    w.neff[a] = 0;
    w.amax[a] = 0.0;
  }
}


// Launch, with the kernel's own start / end timestamps in (e0, e1) when given.
template <typename K>
static void launch_timed(K kernel, dim3 grid, dim3 block, hipStream_t s, hipEvent_t e0,
                         hipEvent_t e1, const LanczosWS& w, int j) {
  if (e0) hipExtLaunchKernelGGL(kernel, grid, block, 0, s, e0, e1, 0, w, j);
  else hipLaunchKernelGGL(kernel, grid, block, 0, s, w, j);
}

static void phiu_launch(const LanczosWS& w, int j, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  const dim3 grid((j + 8) / 8 + w.GB, w.n_act);
  const int m4 = w.m / 4;
  if (m4 <= 64) launch_timed(k_lz_phiu<64>, grid, dim3(512), s, e0, e1, w, j);
  else if (m4 <= 128) launch_timed(k_lz_phiu<128>, grid, dim3(512), s, e0, e1, w, j);
  else if (m4 <= 256) launch_timed(k_lz_phiu<256>, grid, dim3(512), s, e0, e1, w, j);
  else launch_timed(k_lz_phiu<512>, grid, dim3(512), s, e0, e1, w, j);
}

int lanczos_m4(int m) {
  const int m4 = m / 4;
  return m4 <= 64 ? 64 : m4 <= 128 ? 128 : m4 <= 256 ? 256 : 512;
}

hipError_t launch_lanczos(const LanczosWS& w, const double* q1_act, hipStream_t s,
                          const hipEvent_t* ev_before, const hipEvent_t* ev_after) {
  (void)hipGetLastError();
  hipLaunchKernelGGL(k_lz_start, dim3((w.L + 255) / 256, w.n_act), dim3(256), 0, s, w, q1_act);
  const int ns = w.m / 256;
  for (int j = 0; j < w.n_it; ++j) {
    const int nx = (j > 0) ? (j + 15) / 16 + 1 : 0;
    launch_timed(k_lz_phit, dim3(nx + ns * w.GA, w.n_act), dim3(512), s,
                 ev_before ? ev_before[2 * j] : nullptr, ev_after ? ev_after[2 * j] : nullptr, w, j);
    hipLaunchKernelGGL(k_lz_finish, dim3(w.m / 16, w.n_act), dim3(256), 0, s, w, j);
    phiu_launch(w, j, s, ev_before ? ev_before[2 * j + 1] : nullptr,
                ev_after ? ev_after[2 * j + 1] : nullptr);
    hipLaunchKernelGGL(k_lz_orth, dim3(w.G3, w.n_act), dim3(256), 0, s, w, j);
  }
  hipLaunchKernelGGL(k_lz_last_beta, dim3(w.n_act), dim3(256), 0, s, w);
  return hipGetLastError();
}

}  // namespace slh
