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
//   phiu    u = Phi t_j (= A q_j): the same (row group, column slice) blocks
//           write per-slice partial row dots; the first blocks of the launch
//           form h1 = Q_j^T u as t_k^T t_j (k <= j), the same inner products
//           taken in feature space, so no pass over Q is needed.
//   orth    per 32 rows: u from its slice partials; q_j = (z1 - Q_{j-1} h2) /
//           beta (second pass in row space, stored as Q[j]); alpha_j = h1_j;
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

// Value of v in lane l (l uniform), through the scalar unit.
__device__ __forceinline__ double readlane_f64(double v, int l) {
  const unsigned long long x = (unsigned long long)__double_as_longlong(v);
  const unsigned lo = (unsigned)__builtin_amdgcn_readlane((int)(unsigned)x, l);
  const unsigned hi = (unsigned)__builtin_amdgcn_readlane((int)(unsigned)(x >> 32), l);
  return __longlong_as_double((long long)(((unsigned long long)hi << 32) | lo));
}

// Sum of src[g * ld] over g < G with 8 loads in flight (fixed order).
// Every batch issues its 8 loads unconditionally (index clamped to G - 1, the
// surplus values masked to zero afterwards), so a ragged tail costs one round
// trip rather than one per element.
__device__ __forceinline__ double sum_strided(const double* __restrict__ src, int64_t ld, int G) {
  double acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  for (int g = 0; g < G; g += 8) {
    double v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = src[(int64_t)min(g + e, G - 1) * ld];
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] += (g + e < G) ? v[e] : 0.0;
  }
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

// Block g of nx = ceil(j / 16) + 1 (512 threads): H2[k] = sum over the orth
// blocks of the h2 partials for k in [16 g, 16 g + 16) (k < j), or, for the
// last block, |z1|^2 (slot ldq).
__device__ __forceinline__ void h2_reduce_block(const LanczosWS& w, int a, int j, int g, int nx) {
  const int hs = w.ldq + 1;
  const double* hp = w.H2part + (int64_t)a * w.G3 * hs;
  double* dst = w.H2 + (int64_t)a * hs;
  if (g == nx - 1) {
    const double v = block_colsum<1, 512>(hp + w.ldq, hs, w.G3, 0, 1);
    if (threadIdx.x == 0) dst[w.ldq] = v;
  } else {
    const int c0 = g * 16;
    const double v = block_colsum<16, 512>(hp, hs, w.G3, c0, j);
    if (threadIdx.x < 16 && c0 + threadIdx.x < j) dst[c0 + threadIdx.x] = v;
  }
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
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int L = w.L, m = w.m, hs = w.ldq + 1;
  const int nx = (j > 0) ? (j + 15) / 16 + 1 : 0;
  int g = blockIdx.x;
  if (g < nx) {
    if (w.stop[a]) return;
    h2_reduce_block(w, a, j, g, nx);
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
  double wc, wn;
  // rows r0 + wave + 8 (8 b + e), e < 8, of batch b; lane e (mod 8) also loads the
  // weight of row e (0 past the group), broadcast when the batch is consumed
  auto load8 = [&](float4 (&dst)[8], double& wd, int b) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int i = min(r0 + wave + 8 * (8 * b + e), r1 - 1);
      dst[e] = *(const float4*)(base + (int64_t)i * m);
    }
    const int iw = r0 + wave + 8 * (8 * b + (lane & 7));
    const double v = vsrc[min(iw, r1 - 1)];
    wd = (iw < r1) ? v : 0.0;
  };
  const int nb = w.RWA / 8;
  load8(vc, wc, 0);                 // in flight while the stop flag is read
  if (w.stop[a]) return;
  for (int b = 0; b < nb; ++b) {
    if (b + 1 < nb) load8(vn, wn, b + 1);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const double q = readlane_f64(wc, e);
      s0 = fma((double)vc[e].x, q, s0);
      s1 = fma((double)vc[e].y, q, s1);
      s2 = fma((double)vc[e].z, q, s2);
      s3 = fma((double)vc[e].w, q, s3);
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) vc[e] = vn[e];
    wc = wn;
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
// 16 columns x 16 partial lanes).  Every load is issued before the first
// reduction.
// ---------------------------------------------------------------------------
// KT = 16-step slots of k per thread: 16 KT >= n_it (fewer registers for short runs)
template <int KT>
__global__ __launch_bounds__(256) void k_lz_finish(LanczosWS w, int j) {
  const int a = blockIdx.y, g = blockIdx.x, tid = threadIdx.x;
  const int m = w.m, hs = w.ldq + 1;
  const int cl = tid & 15, pl = tid >> 4;
  const int c = g * 16 + cl;                   // m is a multiple of 16
  const double* H2 = w.H2 + (int64_t)a * hs;
  // The loads of t_k and h2_k (k = pl + 16 e < j <= 16 KT), of the |h2|^2 terms
  // (k = tid, tid + 256 < j), of |z1|^2 and of the step state are all issued
  // before the first use, with clamped indices (surplus values are masked), so
  // the kernel waits on memory once.
  const int jm = max(j - 1, 0);
  const double* Ta = w.T + (int64_t)a * w.ldq * m + c;
  double tv[KT], hv[KT];
#pragma unroll
  for (int e = 0; e < KT; ++e) {
    const int k = min(pl + 16 * e, jm);
    tv[e] = Ta[(int64_t)k * m];
    hv[e] = H2[k];
  }
  const double hq0 = H2[min(tid, jm)], hq1 = H2[min(tid + 256, jm)];
  const double z2 = H2[w.ldq];
  const int stopped = w.stop[a];
  const double amax = w.amax[a];
  // partial of Phi^T z1 over row groups pl, pl + 16, ...
  const double* Sp = w.Spart + (int64_t)a * w.GA * m + c;
  const int cnt = (w.GA - pl + 15) / 16;
  const double s = sum_strided(Sp + (int64_t)pl * m, (int64_t)16 * m, cnt > 0 ? cnt : 0);
  // partial of sum_k h2_k t_k over k = pl, pl + 16, ... < j
  double corr;
  {
    double acc[4] = {0, 0, 0, 0};
#pragma unroll
    for (int e = 0; e < KT; ++e)
      if (pl + 16 * e < j) acc[e & 3] = fma(tv[e], hv[e], acc[e & 3]);
    corr = (acc[0] + acc[1]) + (acc[2] + acc[3]);
  }
  // |h2|^2 partial
  double hh = 0.0;
  if (tid < j) hh = fma(hq0, hq0, hh);
  if (tid + 256 < j) hh = fma(hq1, hq1, hh);
  if (stopped) return;
  __shared__ double red[4];
  __shared__ double sh;
  __shared__ double rs[16][17], rc[16][17];
  rs[pl][cl] = s;
  rc[pl][cl] = corr;
  double inv = 1.0;
  if (j > 0) {
    hh = block_sum_f64(hh, red);               // (its barriers also publish rs / rc)
    if (tid == 0) {
      const double b2 = z2 - hh;               // |z1 - Q h2|^2 for orthonormal Q
      const double beta = b2 > 0.0 ? sqrt(b2) : 0.0;
      const bool brk = !(beta > w.tol * amax);
      sh = brk ? 0.0 : beta;
      if (g == 0) {
        w.beta[(int64_t)a * w.n_it + j - 1] = beta;
        if (brk) w.stop[a] = 1;                // n_eff stays j
      }
    }
    __syncthreads();
    if (sh == 0.0) return;
    inv = 1.0 / sh;
  } else {
    __syncthreads();
  }
  if (tid < 16) {
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
// rest own (row group, 256-column slice) exactly as in phit and write the
// slice's partial of u = Phi t_j for each row (Upart[slice][row]): lane = 4
// columns, the 8 rows of a batch are summed over the wave in one butterfly.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(512) void k_lz_phiu(LanczosWS w, int j) {
  const int a = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int L = w.L, m = w.m;
  const double* Ta = w.T + (int64_t)a * w.ldq * m;
  const double* tj = Ta + (int64_t)j * m;
  const int nx = (j + 8) / 8;
  int g = blockIdx.x;
  if (g < nx) {
    if (w.stop[a]) return;
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
  const int ns = m >> 8;
  const int sl = g % ns, rg = g / ns;
  const int r0 = rg * w.RBA;
  const int r1 = min(L, r0 + w.RBA);
  const float* base = w.Phi + (int64_t)a * L * m + sl * 256 + 4 * lane;
  float4 vc[8], vn[8];
  auto load8 = [&](float4 (&dst)[8], int b) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int i = min(r0 + wave + 8 * (8 * b + e), r1 - 1);
      dst[e] = *(const float4*)(base + (int64_t)i * m);
    }
  };
  const int nb = w.RWA / 8;
  load8(vc, 0);                     // in flight while t_j and the stop flag are read
  const double* tc = tj + sl * 256 + 4 * lane;
  const double t0 = tc[0], t1 = tc[1], t2 = tc[2], t3 = tc[3];
  if (w.stop[a]) return;
  double* up = w.Upart + ((int64_t)a * ns + sl) * L;
  const int idx = ((lane >> 5) & 1) * 4 + ((lane >> 4) & 1) * 2 + ((lane >> 3) & 1);
  for (int b = 0; b < nb; ++b) {
    if (b + 1 < nb) load8(vn, b + 1);
    double p[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      double d = (double)vc[e].x * t0;
      d = fma((double)vc[e].y, t1, d);
      d = fma((double)vc[e].z, t2, d);
      p[e] = fma((double)vc[e].w, t3, d);
    }
    const double tot = wave_sum8_f64(p);
    const int i = r0 + wave + 8 * (8 * b + idx);
    if ((lane & 7) == 0 && i < r1) up[i] = tot;
#pragma unroll
    for (int e = 0; e < 8; ++e) vc[e] = vn[e];
  }
}

// ---------------------------------------------------------------------------
// orth on 32 rows per block (256 threads = 32 rows x 8 k-groups).  Thread
// (row, kg) loads Q[k][row] for k = kg + 8 t (k < j) once, into registers, and
// uses them for the q_j update, for z1 = u - Q h1 and for the h2 partials.
// ---------------------------------------------------------------------------
// MAXT = 8-step slots of k per thread: 8 MAXT >= n_it, MAXT a multiple of 8
// (fewer registers for short runs)
template <int MAXT>
__global__ __launch_bounds__(256) void k_lz_orth(LanczosWS w, int j) {
  static_assert(MAXT % 8 == 0, "slots are reduced 8 at a time");
  const int a = blockIdx.y, g = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63;
  const int L = w.L, hs = w.ldq + 1;
  const int rl = tid & 31, kg = tid >> 5;
  const int r0 = g * 32;
  const int i = r0 + rl;
  const int ic = min(i, L - 1);
  const double* Qa = w.Q + (int64_t)a * w.ldq * L;
  const int nt = (j - kg + 7) / 8;             // k = kg + 8 t < j
  // every global load of the kernel is issued here, before the first use
  // (indices clamped; values that are not needed are never used)
  const int jm = max(j - 1, 0);
  double qv[MAXT];
#pragma unroll
  for (int t = 0; t < MAXT; ++t)
    if (8 * t < j) qv[t] = Qa[(int64_t)min(kg + 8 * t, jm) * L + ic];
  const double* H1a = w.H1 + (int64_t)a * hs;
  const double* H2a = w.H2 + (int64_t)a * hs;
  const double h1v0 = H1a[min(tid, j)], h1v1 = H1a[min(tid + 256, j)];
  const double h2v0 = H2a[min(tid, jm)], h2v1 = H2a[min(tid + 256, jm)];
  const int ns = w.m >> 8;                     // <= 8 column slices
  const double* up = w.Upart + (int64_t)a * ns * L + ic;
  double us[8];
#pragma unroll
  for (int sl = 0; sl < 8; ++sl) us[sl] = up[(int64_t)min(sl, ns - 1) * L];
  const double zi = w.Z1[(int64_t)a * L + ic];
  const double bet = w.beta[(int64_t)a * w.n_it + jm];
  const double q0 = Qa[ic];
  const int stopped = w.stop[a];
  const double amax0 = (j > 0) ? w.amax[a] : 0.0;
  __shared__ double h1[264], h2[264];
  __shared__ double rq[8][33], rz[8][33];
  __shared__ double sz[32], sq[32];
  double ui = 0.0;
#pragma unroll
  for (int sl = 0; sl < 8; ++sl)
    if (sl < ns) ui += us[sl];
  if (tid <= j) h1[tid] = h1v0;
  if (tid + 256 <= j) h1[tid + 256] = h1v1;
  if (tid < j) h2[tid] = h2v0;
  if (tid + 256 < j) h2[tid + 256] = h2v1;
  if (stopped) return;
  __syncthreads();
  if (g == 0 && tid == 0) {
    w.alpha[(int64_t)a * w.n_it + j] = h1[j];
    w.amax[a] = fmax(amax0, fabs(h1[j]));
    w.neff[a] = j + 1;
  }
  // Q_{j-1} h2 (q_j update) and Q_{j-1} h1 (z1) over this thread's k
  {
    double aq[2] = {0, 0}, az[2] = {0, 0};
#pragma unroll
    for (int t = 0; t < MAXT; ++t) {
      if (t < nt) {
        const int k = kg + 8 * t;
        aq[t & 1] = fma(qv[t], h2[k], aq[t & 1]);
        az[t & 1] = fma(qv[t], h1[k], az[t & 1]);
      }
    }
    rq[kg][rl] = aq[0] + aq[1];
    rz[kg][rl] = az[0] + az[1];
  }
  __syncthreads();
  if (tid < 32) {
    double z = 0.0, q = 0.0;
    if (i < L) {
      if (j > 0) {
        double sub = 0.0;
        for (int p = 0; p < 8; ++p) sub += rq[p][rl];
        q = (zi - sub) / bet;
        w.Q[((int64_t)a * w.ldq + j) * L + i] = q;
      } else {
        q = q0;
      }
      double zs = 0.0;
      for (int p = 0; p < 8; ++p) zs += rz[p][rl];
      z = ui - fma(q, h1[j], zs);
      w.Z1[(int64_t)a * L + i] = z;
    }
    sz[rl] = z;
    sq[rl] = q;
  }
  __syncthreads();
  // partials of h2_k = sum over these rows of Q[k] z1 for k < j (from the registers,
  // summed over the 32 rows of each half wave, 8 values per butterfly) and k = j
  double* hp = w.H2part + ((int64_t)a * w.G3 + g) * hs;
  const double zl = sz[rl];
  const int idx = ((lane >> 4) & 1) * 4 + ((lane >> 3) & 1) * 2 + ((lane >> 2) & 1);
#pragma unroll
  for (int t0 = 0; t0 < MAXT; t0 += 8) {
    if (8 * t0 < j) {                          // block-uniform
      double v8[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) v8[e] = (t0 + e < nt) ? qv[t0 + e] * zl : 0.0;
      const double tot = half_sum8_f64(v8);
      const int k = kg + 8 * (t0 + idx);
      if ((lane & 3) == 0 && k < j) hp[k] = tot;
    }
  }
  if (tid < 64) {
    // k = j and |z1|^2 over the 32 rows: lanes 0-31 and 32-63 of wave 0
    const double v = (tid < 32) ? sq[rl] * sz[rl] : sz[rl] * sz[rl];
    double t = v;
#pragma unroll
    for (int o = 16; o >= 1; o >>= 1) t += __shfl_xor(t, o, 64);
    if (tid == 0) hp[j] = t;
    if (tid == 32) hp[w.ldq] = t;
  }
}

// beta of the last step (reported; T does not use it): h2 and |z1|^2 of the last
// orthogonalisation are reduced as at the start of a step, then
// beta = sqrt(|z1|^2 - |h2|^2).
__global__ __launch_bounds__(512) void k_lz_h2sum(LanczosWS w) {
  const int a = blockIdx.y;
  if (w.stop[a]) return;
  const int j = w.n_it, nx = (j + 15) / 16 + 1;
  h2_reduce_block(w, a, j, blockIdx.x, nx);
}

__global__ __launch_bounds__(256) void k_lz_last_beta(LanczosWS w) {
  const int a = blockIdx.x, tid = threadIdx.x;
  if (w.stop[a]) return;
  const int j = w.n_it, hs = w.ldq + 1;
  const double* H2 = w.H2 + (int64_t)a * hs;
  __shared__ double red[4];
  double hh = 0.0;
  for (int k = tid; k < j; k += 256) hh = fma(H2[k], H2[k], hh);
  hh = block_sum_f64(hh, red);
  if (tid == 0) {
    const double b2 = H2[w.ldq] - hh;
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

// the smallest slot counts that cover n_it (finish: 16 KT >= n_it; orth: 8 MAXT >= n_it,
// MAXT a multiple of 8)
static void launch_finish(const LanczosWS& w, int j, hipStream_t s) {
  const dim3 g(w.m / 16, w.n_act), b(256);
  const int kt = (w.n_it + 15) / 16;
  if (kt <= 2) hipLaunchKernelGGL(k_lz_finish<2>, g, b, 0, s, w, j);
  else if (kt <= 4) hipLaunchKernelGGL(k_lz_finish<4>, g, b, 0, s, w, j);
  else if (kt <= 6) hipLaunchKernelGGL(k_lz_finish<6>, g, b, 0, s, w, j);
  else if (kt <= 8) hipLaunchKernelGGL(k_lz_finish<8>, g, b, 0, s, w, j);
  else if (kt <= 12) hipLaunchKernelGGL(k_lz_finish<12>, g, b, 0, s, w, j);
  else hipLaunchKernelGGL(k_lz_finish<16>, g, b, 0, s, w, j);
}

static void launch_orth(const LanczosWS& w, int j, hipStream_t s) {
  const dim3 g(w.G3, w.n_act), b(256);
  const int mt = (w.n_it + 7) / 8;                 // MAXT: a multiple of 8 (h2 butterflies)
  if (mt <= 8) hipLaunchKernelGGL(k_lz_orth<8>, g, b, 0, s, w, j);
  else if (mt <= 16) hipLaunchKernelGGL(k_lz_orth<16>, g, b, 0, s, w, j);
  else if (mt <= 24) hipLaunchKernelGGL(k_lz_orth<24>, g, b, 0, s, w, j);
  else hipLaunchKernelGGL(k_lz_orth<32>, g, b, 0, s, w, j);
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
    launch_finish(w, j, s);
    launch_timed(k_lz_phiu, dim3((j + 8) / 8 + ns * w.GA, w.n_act), dim3(512), s,
                 ev_before ? ev_before[2 * j + 1] : nullptr,
                 ev_after ? ev_after[2 * j + 1] : nullptr, w, j);
    launch_orth(w, j, s);
  }
  hipLaunchKernelGGL(k_lz_h2sum, dim3((w.n_it + 15) / 16 + 1, w.n_act), dim3(512), 0, s, w);
  hipLaunchKernelGGL(k_lz_last_beta, dim3(w.n_act), dim3(256), 0, s, w);
  return hipGetLastError();
}

// reps x (Phi^T v, Phi t) of step j, launched exactly as in launch_lanczos
hipError_t launch_lanczos_passes(const LanczosWS& w, int j, int reps, hipStream_t s) {
  (void)hipGetLastError();
  const int ns = w.m / 256;
  const int nx = (j > 0) ? (j + 15) / 16 + 1 : 0;
  for (int q = 0; q < reps; ++q) {
    hipLaunchKernelGGL(k_lz_phit, dim3(nx + ns * w.GA, w.n_act), dim3(512), 0, s, w, j);
    hipLaunchKernelGGL(k_lz_phiu, dim3((j + 8) / 8 + ns * w.GA, w.n_act), dim3(512), 0, s, w, j);
  }
  return hipGetLastError();
}

}  // namespace slh
