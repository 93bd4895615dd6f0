// Implicit Lanczos with full re-orthogonalization (Algorithm 2; operator of
// Eq. 4, A v = Phi (Phi^T v), never forming the N x N kernel).
//
// Each window runs its own recurrence; all windows advance in lockstep (grid
// dimension y = window).  Vectors and every reduction are fp64; Phi is fp32.
//
// Step j (q_j = Q[j], t_j = Phi^T q_j = T[j]) is five kernels:
//   phit    partials of Phi^T v over row blocks, v = q_0 (j = 0) or z1 of step
//           j-1 (the vector after the first Gram-Schmidt pass); extra blocks of
//           the same launch reduce the partials of h2 and |z1|^2 of step j-1.
//   finish  beta_{j-1} = |z1 - Q h2| = sqrt(|z1|^2 - |h2|^2) (Q orthonormal) and
//           the breakdown test; then t_j = (Phi^T z1 - sum_k h2_k t_k) / beta
//           (m-space blocks) and q_j = (z1 - Q h2) / beta (row blocks): the
//           second Gram-Schmidt pass.  Its coefficients h2 are at rounding level,
//           so folding them into t by linearity is harmless, while Phi^T z1 itself
//           is always streamed.
//   phiu    u = Phi t_j (= A q_j) and partials of h1 = Q_j^T u.
//   colsum  h1.
//   orth    alpha_j = h1_j = q_j^T A q_j; z1 = u - Q_j h1 (first classical
//           Gram-Schmidt pass); partials of h2 = Q_j^T z1 and |z1|^2.
// Phi is streamed twice per step.  (Forming Phi^T q_{j+1} from Phi^T u by the
// whole three-term recurrence would save a pass but is unstable: it multiplies
// rounding errors by alpha_j / beta_j every step.)  All partial sums are
// combined in a fixed order, so results are bitwise reproducible.  The
// Lanczos quantities are those of Algorithm 2: alpha_j = q_j^T A q_j before
// any subtraction, beta_j the norm after re-orthogonalization; the
// corrections are not folded into T.
#include "slh_device.h"
#include "slh_internal.h"

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
__device__ __forceinline__ int sum8_index(int lane) {
  return ((lane >> 5) & 1) * 4 + ((lane >> 4) & 1) * 2 + ((lane >> 3) & 1);
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

// Thread layout of the two passes over Phi (512 threads): a row is covered by
// M4 = m/4 threads, each owning 4 consecutive columns (one float4); RP = 512/M4
// rows are covered at once; a block owns RB1 = RP * RPT rows (RPT a multiple of
// 8); each thread streams its RPT rows in batches of 8 with the next batch's
// loads in flight.  Loads are unconditional (row index clamped into the block):
// rows past the block contribute nothing through their zero weight.

// ---------------------------------------------------------------------------
// phit: partials of Phi^T v over the block's rows (v = q_0 or z1); blocks
// G1.. of the launch reduce the h2 / |z1|^2 partials of the previous step.
// ---------------------------------------------------------------------------
template <int M4>
__global__ __launch_bounds__(512) void k_lz_phit(LanczosWS w, int j) {
  constexpr int RP = 512 / M4;
  const int a = blockIdx.y, g = blockIdx.x;
  if (w.stop[a]) return;
  const int tid = threadIdx.x;
  const int L = w.L, m = w.m, hs = w.ldq + 1;
  if (g >= w.G1) {
    // reduce h2 (k < j) and |z1|^2 (slot ldq) of step j-1 over the orth blocks
    const int c0 = (g - w.G1) * 16;
    const double* hp = w.H2part + (int64_t)a * w.G3 * hs;
    double* dst = w.H2 + (int64_t)a * hs;
    const double v = block_colsum<16, 512>(hp, hs, w.G3, c0, j);
    if (tid < 16 && c0 + tid < j) dst[c0 + tid] = v;
    if (g == w.G1 && tid == 511) dst[w.ldq] = sum_strided(hp + w.ldq, hs, w.G3);
    return;
  }
  const int r0 = g * w.RB1;
  const int r1 = min(L, r0 + w.RB1);
  const float* Phi = w.Phi + (int64_t)a * L * m;
  const double* vsrc = (j == 0) ? (w.Q + (int64_t)a * w.ldq * L) : (w.Z1 + (int64_t)a * L);
  const int c4 = tid % M4, rs = tid / M4;
  const bool cin = 4 * c4 < m;
  const float* base = Phi + 4 * min(c4, m / 4 - 1);
  double s0 = 0.0, s1 = 0.0, s2 = 0.0, s3 = 0.0;
  float4 vc[8], vn[8];
  auto load8 = [&](float4 (&dst)[8], int b) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int i = min(r0 + rs + RP * (8 * b + e), r1 - 1);
      dst[e] = *(const float4*)(base + (int64_t)i * m);
    }
  };
  const int nb = w.RPT / 8;
  load8(vc, 0);
  for (int b = 0; b < nb; ++b) {
    if (b + 1 < nb) load8(vn, b + 1);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int i = r0 + rs + RP * (8 * b + e);
      const double vi = vsrc[min(i, r1 - 1)];
      const double qi = (cin && i < r1) ? vi : 0.0;
      s0 = fma((double)vc[e].x, qi, s0);
      s1 = fma((double)vc[e].y, qi, s1);
      s2 = fma((double)vc[e].z, qi, s2);
      s3 = fma((double)vc[e].w, qi, s3);
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) vc[e] = vn[e];
  }
  double* sp = w.Spart + ((int64_t)a * w.G1 + g) * m;
  if (RP == 1) {
    if (cin) {
      sp[4 * c4 + 0] = s0;
      sp[4 * c4 + 1] = s1;
      sp[4 * c4 + 2] = s2;
      sp[4 * c4 + 3] = s3;
    }
  } else {
    __shared__ double cred[RP > 1 ? RP : 1][RP > 1 ? 4 * M4 : 1];
    if (cin) {
      cred[rs][4 * c4 + 0] = s0;
      cred[rs][4 * c4 + 1] = s1;
      cred[rs][4 * c4 + 2] = s2;
      cred[rs][4 * c4 + 3] = s3;
    }
    __syncthreads();
    for (int c = tid; c < m; c += 512) {
      double t = 0.0;
      for (int q = 0; q < RP; ++q) t += cred[q][c];
      sp[c] = t;
    }
  }
}

// ---------------------------------------------------------------------------
// finish: beta_{j-1}, breakdown, t_j (blocks [0, NT), 16 columns each) and
// q_j (blocks [NT, NT + NQ), 32 rows each).  256 threads.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_lz_finish(LanczosWS w, int j) {
  const int a = blockIdx.y, g = blockIdx.x, tid = threadIdx.x;
  if (w.stop[a]) return;
  const int L = w.L, m = w.m, hs = w.ldq + 1;
  const int NT = (m + 15) / 16;
  __shared__ double h2[264];
  __shared__ double sh[2];
  double inv = 1.0;
  if (j > 0) {
    const double* H2 = w.H2 + (int64_t)a * hs;
    double hh = 0.0;
    for (int k = tid; k < j; k += 256) {
      const double v = H2[k];
      h2[k] = v;
      hh = fma(v, v, hh);
    }
    __shared__ double red[4];
    hh = block_sum_f64(hh, red);
    if (tid == 0) {
      const double b2 = H2[w.ldq] - hh;       // |z1 - Q h2|^2 for orthonormal Q
      const double beta = b2 > 0.0 ? sqrt(b2) : 0.0;
      const bool brk = !(beta > w.tol * w.amax[a]);
      sh[0] = brk ? 0.0 : beta;
      if (g == 0) {
        w.beta[(int64_t)a * w.n_it + j - 1] = beta;
        if (brk) w.stop[a] = 1;                // n_eff stays j
      }
    }
    __syncthreads();
    if (sh[0] == 0.0) return;
    inv = 1.0 / sh[0];
  }
  if (g < NT) {
    // t_j = (sum_g Spart[g] - sum_{k<j} h2_k t_k) / beta on 16 columns
    const int c0 = g * 16;
    double v = block_colsum<16, 256>(w.Spart + (int64_t)a * w.G1 * m, m, w.G1, c0, m);
    if (tid < 16 && c0 + tid < m) {
      const int c = c0 + tid;
      if (j > 0) {
        const double* Ta = w.T + (int64_t)a * w.ldq * m + c;
        double acc[4] = {0, 0, 0, 0};
        int k = 0;
        for (; k + 4 <= j; k += 4) {
#pragma unroll
          for (int e = 0; e < 4; ++e) acc[e] = fma(Ta[(int64_t)(k + e) * m], h2[k + e], acc[e]);
        }
        for (; k < j; ++k) acc[0] = fma(Ta[(int64_t)k * m], h2[k], acc[0]);
        v = (v - ((acc[0] + acc[1]) + (acc[2] + acc[3]))) * inv;
      }
      w.T[((int64_t)a * w.ldq + j) * m + c] = v;
    }
    return;
  }
  if (j == 0) return;
  // q_j = (z1 - Q_{j-1} h2) / beta on 32 rows: thread = (row, k-group of 8)
  __shared__ double qred[8][33];
  const int r0 = (g - NT) * 32;
  const int rl = tid & 31, kg = tid >> 5;
  const int i = r0 + rl;
  const int ic = min(i, L - 1);
  const double* Qa = w.Q + (int64_t)a * w.ldq * L;
  double acc[4] = {0, 0, 0, 0};
  {
    int k = kg;
    for (; k + 24 < j; k += 32) {
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[e] = fma(Qa[(int64_t)(k + 8 * e) * L + ic], h2[k + 8 * e], acc[e]);
    }
    for (; k < j; k += 8) acc[0] = fma(Qa[(int64_t)k * L + ic], h2[k], acc[0]);
  }
  qred[kg][rl] = (acc[0] + acc[1]) + (acc[2] + acc[3]);
  __syncthreads();
  if (tid < 32 && i < L) {
    double sub = 0.0;
    for (int q = 0; q < 8; ++q) sub += qred[q][rl];
    w.Q[((int64_t)a * w.ldq + j) * L + i] = (w.Z1[(int64_t)a * L + i] - sub) * inv;
  }
}

// ---------------------------------------------------------------------------
// phiu: u = Phi t_j on the block's rows and the partial h1 = Q_j^T u.
// Each thread keeps its partial dot of every row it streams; one block-level
// reduction at the end gives the u values.
// ---------------------------------------------------------------------------
template <int M4>
__global__ __launch_bounds__(512) void k_lz_phiu(LanczosWS w, int j) {
  constexpr int RP = 512 / M4;
  constexpr int WPR = M4 >= 64 ? M4 / 64 : 1;     // waves per row group
  constexpr int MAXR = 32;                        // rows per thread kept (RPT <= 32)
  const int a = blockIdx.y, g = blockIdx.x;
  if (w.stop[a]) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int L = w.L, m = w.m;
  const int r0 = g * w.RB1;
  const int r1 = min(L, r0 + w.RB1);
  const float* Phi = w.Phi + (int64_t)a * L * m;
  const double* Qa = w.Q + (int64_t)a * w.ldq * L;
  __shared__ double su[256];
  __shared__ double ured[8][MAXR];
  const int c4 = tid % M4, rs = tid / M4;
  const bool cin = 4 * c4 < m;
  const double* tj = w.T + ((int64_t)a * w.ldq + j) * m;
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
      if ((lane & 7) == 0) ured[wave][q0 + sum8_index(lane)] = tot;
    }
  }
  __syncthreads();
  for (int x = tid; x < RP * w.RPT; x += 512) {
    const int rsx = x / w.RPT, q = x % w.RPT;
    double u = 0.0;
    for (int ww = 0; ww < WPR; ++ww) u += ured[rsx * WPR + ww][q];
    const int i = r0 + rsx + RP * q;
    if (i < r1) {
      w.U[(int64_t)a * L + i] = u;
      su[i - r0] = u;
    }
  }
  __syncthreads();
  // partial h1_k = sum_{i in block} Q[k][i] u_i, k <= j: wave handles k = wave*8 + 64*q + e,
  // lane = row within 64-row chunks; 8 independent loads per lane per chunk
  const int nr = r1 - r0;
  double* hp = w.H1part + ((int64_t)a * w.G1 + g) * (w.ldq + 1);
  for (int k0 = wave * 8; k0 <= j; k0 += 64) {
    double v8[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    for (int i0 = 0; i0 < nr; i0 += 64) {
      const int il = i0 + lane;
      const int ic = min(il, nr - 1);
      const double uu = (il < nr) ? su[ic] : 0.0;
      double qv[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) qv[e] = Qa[(int64_t)min(k0 + e, j) * L + r0 + ic];
#pragma unroll
      for (int e = 0; e < 8; ++e) v8[e] = fma(qv[e], uu, v8[e]);
    }
    const double tot = wave_sum8_f64(v8);
    const int k = k0 + sum8_index(lane);
    if ((lane & 7) == 0 && k <= j) hp[k] = tot;
  }
}

// h1 = sum over the phiu blocks (4 columns per block, 64 partial lanes).
__global__ __launch_bounds__(256) void k_lz_h1sum(LanczosWS w, int j) {
  const int a = blockIdx.y;
  if (w.stop[a]) return;
  const int hs = w.ldq + 1, c0 = blockIdx.x * 4, tid = threadIdx.x;
  const double v = block_colsum<4, 256>(w.H1part + (int64_t)a * w.G1 * hs, hs, w.G1, c0, j + 1);
  if (tid < 4 && c0 + tid <= j) w.H1[(int64_t)a * hs + c0 + tid] = v;
}

// ---------------------------------------------------------------------------
// orth: z1 = u - Q_j h1 on this block's rows; partials of h2 = Q_j^T z1, |z1|^2.
// alpha_j = h1_j = q_j^T A q_j (taken before any subtraction).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_lz_orth(LanczosWS w, int j) {
  const int a = blockIdx.y, g = blockIdx.x;
  if (w.stop[a]) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int L = w.L, nh = j + 1;
  const int r0 = g * w.RB3, r1 = min(L, r0 + w.RB3);
  const double* Qa = w.Q + (int64_t)a * w.ldq * L;
  __shared__ double h1[257];
  __shared__ double sz[64];
  __shared__ double zred[4][64];
  __shared__ double hred[4][264];
  for (int k = tid; k < nh; k += 256) h1[k] = w.H1[(int64_t)a * (w.ldq + 1) + k];
  for (int k = tid; k < 4 * 264; k += 256) (&hred[0][0])[k] = 0.0;
  __syncthreads();
  if (g == 0 && tid == 0) {
    w.alpha[(int64_t)a * w.n_it + j] = h1[j];
    w.amax[a] = fmax(j ? w.amax[a] : 0.0, fabs(h1[j]));
    w.neff[a] = j + 1;
  }
  double nz = 0.0;
  for (int b0 = r0; b0 < r1; b0 += 64) {
    const int nb = min(64, r1 - b0);
    // z1 = u - Q h1 on 64 rows: lane = row, wave = k-group (k = wave mod 4)
    {
      const int i = b0 + min(lane, nb - 1);
      double acc[4] = {0, 0, 0, 0};
      {
        int k = wave;
        for (; k + 12 < nh; k += 16) {
#pragma unroll
          for (int e = 0; e < 4; ++e) acc[e] = fma(Qa[(int64_t)(k + 4 * e) * L + i], h1[k + 4 * e], acc[e]);
        }
        for (; k < nh; k += 4) acc[0] = fma(Qa[(int64_t)k * L + i], h1[k], acc[0]);
      }
      zred[wave][lane] = (acc[0] + acc[1]) + (acc[2] + acc[3]);
    }
    __syncthreads();
    if (tid < 64) {
      double z = 0.0;
      if (tid < nb) {
        z = w.U[(int64_t)a * L + b0 + tid] - ((zred[0][tid] + zred[1][tid]) + (zred[2][tid] + zred[3][tid]));
        w.Z1[(int64_t)a * L + b0 + tid] = z;
        nz = fma(z, z, nz);
      }
      sz[tid] = z;
    }
    __syncthreads();
    // partial h2_k over these rows: wave handles k = wave*8 + 32*q + e, lane = row
    const double zl = sz[lane];
    for (int k0 = wave * 8; k0 < nh; k0 += 32) {
      double v8[8];
      const int lc = min(lane, nb - 1);
#pragma unroll
      for (int e = 0; e < 8; ++e) v8[e] = Qa[(int64_t)min(k0 + e, nh - 1) * L + b0 + lc];
#pragma unroll
      for (int e = 0; e < 8; ++e) v8[e] = (k0 + e < nh) ? v8[e] * zl : 0.0;
      const double tot = wave_sum8_f64(v8);
      const int k = k0 + sum8_index(lane);
      if ((lane & 7) == 0 && k < nh) hred[wave][k] += tot;
    }
    __syncthreads();
  }
  __shared__ double nred[4];
  const double nzw = wave_sum_f64(nz);
  if (lane == 0) nred[wave] = nzw;
  __syncthreads();
  double* hp = w.H2part + ((int64_t)a * w.G3 + g) * (w.ldq + 1);
  for (int k = tid; k < nh; k += 256) hp[k] = hred[0][k] + hred[1][k] + hred[2][k] + hred[3][k];
  if (tid == 0) hp[w.ldq] = (nred[0] + nred[1]) + (nred[2] + nred[3]);
}

// beta of the last step (reported; T does not use it).
__global__ __launch_bounds__(256) void k_lz_last_beta(LanczosWS w) {
  const int a = blockIdx.x, tid = threadIdx.x;
  if (w.stop[a]) return;
  const int j = w.n_it, hs = w.ldq + 1;
  const double* hp = w.H2part + (int64_t)a * w.G3 * hs;
  __shared__ double red[4];
  __shared__ double snz;
  double hh = 0.0;
  for (int k = tid; k < j; k += 256) {
    const double acc = sum_strided(hp + k, hs, w.G3);
    hh = fma(acc, acc, hh);
  }
  if (tid == 255) snz = sum_strided(hp + w.ldq, hs, w.G3);
  hh = block_sum_f64(hh, red);
  if (tid == 0) {
    const double b2 = snz - hh;
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


template <int M4>
static void launch_pass(const LanczosWS& w, int j, bool passA, hipStream_t s) {
  if (passA) {
    // extra blocks reduce the h2 partials of the previous step
    const int extra = (j > 0) ? (j + 15) / 16 : 0;
    hipLaunchKernelGGL((k_lz_phit<M4>), dim3(w.G1 + extra, w.n_act), dim3(512), 0, s, w, j);
  } else {
    hipLaunchKernelGGL((k_lz_phiu<M4>), dim3(w.G1, w.n_act), dim3(512), 0, s, w, j);
  }
}

static void phi_pass(const LanczosWS& w, int j, bool passA, hipStream_t s) {
  const int m4 = w.m / 4;
  if (m4 <= 64) launch_pass<64>(w, j, passA, s);
  else if (m4 <= 128) launch_pass<128>(w, j, passA, s);
  else if (m4 <= 256) launch_pass<256>(w, j, passA, s);
  else launch_pass<512>(w, j, passA, s);
}

int lanczos_m4(int m) {
  const int m4 = m / 4;
  return m4 <= 64 ? 64 : m4 <= 128 ? 128 : m4 <= 256 ? 256 : 512;
}

hipError_t launch_lanczos(const LanczosWS& w, const double* q1_act, hipStream_t s,
                          const hipEvent_t* ev_before, const hipEvent_t* ev_after) {
  (void)hipGetLastError();
  hipLaunchKernelGGL(k_lz_start, dim3((w.L + 255) / 256, w.n_act), dim3(256), 0, s, w, q1_act);
  const int NT = (w.m + 15) / 16, NQ = (w.L + 31) / 32;
  for (int j = 0; j < w.n_it; ++j) {
    if (ev_before) (void)hipEventRecord(ev_before[2 * j], s);
    phi_pass(w, j, true, s);                                     // Phi^T (q_0 or z1)
    if (ev_after) (void)hipEventRecord(ev_after[2 * j], s);
    hipLaunchKernelGGL(k_lz_finish, dim3(NT + (j > 0 ? NQ : 0), w.n_act), dim3(256), 0, s, w, j);
    if (ev_before) (void)hipEventRecord(ev_before[2 * j + 1], s);
    phi_pass(w, j, false, s);                                    // u = Phi t_j, h1 partials
    if (ev_after) (void)hipEventRecord(ev_after[2 * j + 1], s);
    hipLaunchKernelGGL(k_lz_h1sum, dim3((j + 1 + 3) / 4, w.n_act), dim3(256), 0, s, w, j);
    hipLaunchKernelGGL(k_lz_orth, dim3(w.G3, w.n_act), dim3(256), 0, s, w, j);
  }
  hipLaunchKernelGGL(k_lz_last_beta, dim3(w.n_act), dim3(256), 0, s, w);
  return hipGetLastError();
}

}  // namespace slh
