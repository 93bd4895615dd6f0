// Eigh(T) for the Lanczos tridiagonal and the top-r Ritz coordinates
// (Algorithm 1: lambda, V = Eigh(T); Z = Q V[:, n-k:n]).
//
// One 256-thread workgroup per kept eigenpair.  The eigenvalue is isolated by
// Sturm-count multisection (256 probe points per round, one per thread; the
// count of negative pivots of T - x I is the number of eigenvalues below x)
// until the bracket is a few ulps wide; the eigenvector by inverse iteration with a
// partially pivoted LU of T - theta I (two solves from a fixed pseudo-random
// start).  The vector is normalised and its sign chosen so that its first
// nonzero entry is positive.  Everything is fp64.
#include "slh_device.h"
#include "slh_internal.h"

#include <float.h>

namespace slh {

#define EIG_NMAX 256

// 1/d from the hardware reciprocal refined by one Newton step (d a normal number)
__device__ __forceinline__ double rcp_nr(double d) {
  const double r = __builtin_amdgcn_rcp(d);
  return fma(r, fma(-d, r, 1.0), r);
}

// Number of eigenvalues of T below x: negative pivots of the LDL^T factorisation
// of T - x I (Sturm count), pivots below pivmin in magnitude replaced by -pivmin.
__device__ __forceinline__ int sturm_count(const double* al, const double* b2, int n, double x,
                                           double pivmin) {
  double d = al[0] - x;
  if (fabs(d) < pivmin) d = -pivmin;
  int cnt = d < 0.0;
#pragma unroll 4
  for (int i = 1; i < n; ++i) {
    d = (al[i] - x) - b2[i - 1] * rcp_nr(d);
    if (fabs(d) < pivmin) d = -pivmin;
    cnt += d < 0.0;
  }
  return cnt;
}

#define EIG_T 256                // threads per eigenpair: one multisection probe each

// theta: [n_act][r]; Seig: [n_act][n_it][r] (row k, kept column c)
__global__ __launch_bounds__(EIG_T) void k_tridiag_eig(const double* __restrict__ alpha,
                                                       const double* __restrict__ beta,
                                                       const int* __restrict__ neff, int n_it,
                                                       int r, double* __restrict__ theta,
                                                       double* __restrict__ Seig) {
  const int c = blockIdx.x, a = blockIdx.y, tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int n = neff[a];
  const int r_eff = min(r, n);
  double* Sa = Seig + (int64_t)a * n_it * r;
  if (c < r - r_eff) {
    for (int k = tid; k < n_it; k += EIG_T) Sa[(int64_t)k * r + c] = 0.0;
    if (tid == 0) theta[(int64_t)a * r + c] = 0.0;
    return;
  }
  const int kidx = n - r + c;   // ascending index of the wanted eigenvalue
  __shared__ double al[EIG_NMAX], b1[EIG_NMAX], b2[EIG_NMAX];
  __shared__ double y[EIG_NMAX], w[EIG_NMAX];
  __shared__ double fu1[EIG_NMAX], fu2[EIG_NMAX], fd[EIG_NMAX], fl[EIG_NMAX];
  __shared__ int piv[EIG_NMAX];
  __shared__ unsigned long long smask[EIG_T / 64];
  const double* alp = alpha + (int64_t)a * n_it;
  const double* bet = beta + (int64_t)a * n_it;
  for (int k = tid; k < n; k += EIG_T) {
    al[k] = alp[k];
    double b = (k < n - 1) ? bet[k] : 0.0;
    b1[k] = b;
    b2[k] = b * b;
  }
  __syncthreads();
  // Gershgorin bounds and the pivot floor (every wave computes the same values)
  double lo = DBL_MAX, hi = -DBL_MAX, bmax = 0.0, tnorm = 0.0;
  for (int k = lane; k < n; k += 64) {
    double off = fabs(b1[k]) + (k > 0 ? fabs(b1[k - 1]) : 0.0);
    lo = fmin(lo, al[k] - off);
    hi = fmax(hi, al[k] + off);
    bmax = fmax(bmax, b2[k]);
    tnorm = fmax(tnorm, fabs(al[k]) + off);
  }
  for (int o = 32; o >= 1; o >>= 1) {
    lo = fmin(lo, __shfl_xor(lo, o, 64));
    hi = fmax(hi, __shfl_xor(hi, o, 64));
    bmax = fmax(bmax, __shfl_xor(bmax, o, 64));
    tnorm = fmax(tnorm, __shfl_xor(tnorm, o, 64));
  }
  const double pivmin = DBL_MIN * fmax(1.0, bmax);
  const double pad = 2.0 * DBL_EPSILON * fmax(tnorm, DBL_MIN) + 2.0 * pivmin;
  lo -= pad;
  hi += pad;
  // multisection: count(lo) <= kidx < count(hi); EIG_T probes per round,
  // probe p at lo + (hi - lo) (p + 1) / (EIG_T + 1), evaluated by thread p
  for (int it = 0; it < 64; ++it) {
    const double wdt = hi - lo;
    if (wdt <= 2.0 * DBL_EPSILON * fmax(fabs(lo), fabs(hi)) + pivmin) break;
    const double step = wdt / (double)(EIG_T + 1);
    const double x = lo + step * (double)(tid + 1);
    const unsigned long long m = __ballot(sturm_count(al, b2, n, x, pivmin) > kidx);
    if (lane == 0) smask[wv] = m;
    __syncthreads();
    int f = EIG_T;                                 // first probe with count > kidx
#pragma unroll
    for (int q = EIG_T / 64 - 1; q >= 0; --q)
      if (smask[q]) f = 64 * q + __ffsll((long long)smask[q]) - 1;
    __syncthreads();
    const double nlo = (f > 0) ? lo + step * (double)f : lo;
    const double nhi = (f < EIG_T) ? lo + step * (double)(f + 1) : hi;
    if (!(nhi - nlo < wdt)) break;   // no progress (bracket at rounding level)
    lo = nlo;
    hi = nhi;
  }
  const double th = 0.5 * (lo + hi);

  // inverse iteration: LU of T - th I with partial pivoting on thread 0; the
  // triangular solves carry the running entries in registers
  if (tid == 0) {
    const double eps_piv = DBL_EPSILON * fmax(tnorm, DBL_MIN);
    // T - th I = P L U; U has diagonal fd (stored inverted), superdiagonals fu1,
    // fu2.  Row k+1 is swapped up when its entry in column k is larger; both
    // cases are computed branch-free.
    double dcur = al[0] - th, ucur = (n > 1) ? b1[0] : 0.0;
    for (int k = 0; k < n - 1; ++k) {
      const double sub = b1[k];                   // entry (k+1, k)
      const double dnext = al[k + 1] - th;
      const double unext = (k + 1 < n - 1) ? b1[k + 1] : 0.0;
      const bool swap = fabs(dcur) < fabs(sub);
      if (!swap && fabs(dcur) < eps_piv) dcur = (dcur < 0.0 ? -eps_piv : eps_piv);
      const double p = swap ? sub : dcur;         // pivot
      const double ip = rcp_nr(p);
      const double l = (swap ? dcur : sub) * ip;
      fd[k] = ip;
      fu1[k] = swap ? dnext : ucur;
      fu2[k] = swap ? unext : 0.0;
      fl[k] = l;
      piv[k] = swap;
      const double nd = swap ? fma(-l, dnext, ucur) : fma(-l, ucur, dnext);
      ucur = swap ? -l * unext : unext;
      dcur = nd;
    }
    if (fabs(dcur) < eps_piv) dcur = (dcur < 0.0 ? -eps_piv : eps_piv);
    fd[n - 1] = rcp_nr(dcur);
    fu1[n - 1] = 0.0;
    fu2[n - 1] = 0.0;
  }
  // start vector: fixed pseudo-random entries in [-1, 1)
  for (int k = tid; k < n; k += EIG_T) {
    unsigned h = (unsigned)(k + 1) * 2654435761u;
    h ^= h >> 15;
    h *= 2246822519u;
    h ^= h >> 13;
    y[k] = (double)(h >> 8) * (2.0 / 16777216.0) - 1.0;
  }
  __syncthreads();
  for (int itr = 0; itr < 2; ++itr) {
    if (tid == 0) {
      // forward: apply L^{-1} P to y into w (cur = running entry k); input and
      // output arrays differ, so the loads run ahead of the recurrence
      double cur = y[0];
#pragma unroll 4
      for (int k = 0; k < n - 1; ++k) {
        const double nxt = y[k + 1], l = fl[k];
        const bool pk = piv[k];
        w[k] = pk ? nxt : cur;
        cur = pk ? fma(-l, nxt, cur) : fma(-l, cur, nxt);
      }
      w[n - 1] = cur;
      // backward: U x = w into y (x1 = x[k+1], x2 = x[k+2])
      double x1 = 0.0, x2 = 0.0;
#pragma unroll 4
      for (int k = n - 1; k >= 0; --k) {
        const double xk = ((w[k] - fu1[k] * x1) - fu2[k] * x2) * fd[k];
        y[k] = xk;
        x2 = x1;
        x1 = xk;
      }
    }
    __syncthreads();
    // rescale by the largest magnitude (every wave computes the same value)
    double mx = 0.0;
    for (int k = lane; k < n; k += 64) mx = fmax(mx, fabs(y[k]));
    for (int o = 32; o >= 1; o >>= 1) mx = fmax(mx, __shfl_xor(mx, o, 64));
    __syncthreads();
    const double inv = mx > 0.0 ? 1.0 / mx : 1.0;
    for (int k = tid; k < n; k += EIG_T) y[k] *= inv;
    __syncthreads();
  }
  // unit norm; sign such that the first nonzero entry is positive (wave 0)
  if (wv == 0) {
    double nr = 0.0;
    int first = n - 1;
    for (int k = lane; k < n; k += 64) {
      nr = fma(y[k], y[k], nr);
      if (y[k] != 0.0 && k < first) first = k;
    }
    nr = wave_sum_f64(nr);
    for (int o = 32; o >= 1; o >>= 1) first = min(first, __shfl_xor(first, o, 64));
    double sc = 1.0 / sqrt(nr);
    if (y[first] < 0.0) sc = -sc;
    if (lane == 0) theta[(int64_t)a * r + c] = th;
    for (int k = lane; k < n_it; k += 64) Sa[(int64_t)k * r + c] = (k < n) ? y[k] * sc : 0.0;
  }
}

hipError_t launch_tridiag_eig(const double* alpha, const double* beta, const int* neff,
                              int n_act, int n_it, int r, double* theta, double* Seig,
                              hipStream_t s) {
  (void)hipGetLastError();
  hipLaunchKernelGGL(k_tridiag_eig, dim3(r, n_act), dim3(EIG_T), 0, s, alpha, beta, neff, n_it, r,
                     theta, Seig);
  return hipGetLastError();
}

// Z[a][i][c] = sum_{k < n_eff} Q[a][k][i] Seig[a][k][c]   (fp64).
// A block owns 32 rows; thread (row rl = tid % 32, group cg = tid / 32) owns
// CPT = r / 8 (rounded up) columns.  S and the block's Q rows are staged through
// LDS 32 values of k at a time.  Each chunk is fetched into registers with
// unconditional loads (indices clamped; values past n_eff or r are masked when
// stored to LDS), the next chunk's loads in flight while the current one is
// used, so the kernel waits on memory about once per chunk.
template <int CPT>
__global__ __launch_bounds__(256) void k_ritz(const double* __restrict__ Q,
                                              const double* __restrict__ Seig,
                                              const int* __restrict__ neff, int L, int ldq,
                                              int n_it, int r, double* __restrict__ Z) {
  const int a = blockIdx.y, tid = threadIdx.x;
  const int n = neff[a];
  const int rl = tid & 31, cg = tid >> 5;
  const int r0 = blockIdx.x * 32;
  const int i = r0 + rl;
  const double* Qa = Q + (int64_t)a * ldq * L;
  const double* Sa = Seig + (int64_t)a * n_it * r;
  __shared__ double sS[32][8 * CPT + 1];
  __shared__ double sQ[32][33];
  double acc[CPT];
#pragma unroll
  for (int c = 0; c < CPT; ++c) acc[c] = 0.0;
  // a chunk: 32 x 8 CPT values of S (CPT per thread) and 32 x 32 of Q (4 per thread)
  double vs[CPT], vq[4];
  auto fetch = [&](int k0) {
    const int kl = max(min(32, n - k0) - 1, 0) + k0;   // last valid k of the chunk
#pragma unroll
    for (int q = 0; q < CPT; ++q) {
      const int e = tid + 256 * q;
      const int kr = e / (8 * CPT), c = e % (8 * CPT);
      vs[q] = Sa[(int64_t)min(k0 + kr, kl) * r + min(c, r - 1)];
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int e = tid + 256 * q;
      const int kr = e >> 5, rr = e & 31;
      vq[q] = Qa[(int64_t)min(k0 + kr, kl) * L + min(r0 + rr, L - 1)];
    }
  };
  if (n > 0) fetch(0);
  for (int k0 = 0; k0 < n; k0 += 32) {
    const int nk = min(32, n - k0);
#pragma unroll
    for (int q = 0; q < CPT; ++q) {
      const int e = tid + 256 * q;
      const int kr = e / (8 * CPT), c = e % (8 * CPT);
      sS[kr][c] = (kr < nk && c < r) ? vs[q] : 0.0;
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int e = tid + 256 * q;
      const int kr = e >> 5, rr = e & 31;
      sQ[kr][rr] = (kr < nk) ? vq[q] : 0.0;
    }
    __syncthreads();
    if (k0 + 32 < n) fetch(k0 + 32);           // in flight during the FMAs below
#pragma unroll 8
    for (int kk = 0; kk < 32; ++kk) {
      const double q = sQ[kk][rl];
#pragma unroll
      for (int c = 0; c < CPT; ++c) acc[c] = fma(q, sS[kk][cg * CPT + c], acc[c]);
    }
    __syncthreads();
  }
  if (i < L) {
    double* zr = Z + ((int64_t)a * L + i) * r + cg * CPT;
#pragma unroll
    for (int c = 0; c < CPT; ++c)
      if (cg * CPT + c < r) zr[c] = acc[c];
  }
}

hipError_t launch_ritz(const double* Q, const double* Seig, const int* neff, int n_act, int L,
                       int ldq, int n_it, int r, double* Z, hipStream_t s) {
  (void)hipGetLastError();
  const dim3 grid((unsigned)((L + 31) / 32), n_act);
  const int cpt = (r + 7) / 8;                 // r <= 128
  if (cpt <= 1) hipLaunchKernelGGL(k_ritz<1>, grid, dim3(256), 0, s, Q, Seig, neff, L, ldq, n_it, r, Z);
  else if (cpt <= 2) hipLaunchKernelGGL(k_ritz<2>, grid, dim3(256), 0, s, Q, Seig, neff, L, ldq, n_it, r, Z);
  else if (cpt <= 4) hipLaunchKernelGGL(k_ritz<4>, grid, dim3(256), 0, s, Q, Seig, neff, L, ldq, n_it, r, Z);
  else if (cpt <= 8) hipLaunchKernelGGL(k_ritz<8>, grid, dim3(256), 0, s, Q, Seig, neff, L, ldq, n_it, r, Z);
  else hipLaunchKernelGGL(k_ritz<16>, grid, dim3(256), 0, s, Q, Seig, neff, L, ldq, n_it, r, Z);
  return hipGetLastError();
}

}  // namespace slh
