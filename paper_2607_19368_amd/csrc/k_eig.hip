// Eigh(T) for the Lanczos tridiagonal and the top-r Ritz coordinates
// (Algorithm 1: lambda, V = Eigh(T); Z = Q V[:, n-k:n]).
//
// One wave per kept eigenpair.  The eigenvalue is isolated by Sturm-count
// multisection (64 probe points per round, one per lane; the count of
// negative pivots of T - x I is the number of eigenvalues below x) until the
// bracket is a few ulps wide; the eigenvector by inverse iteration with a
// partially pivoted LU of T - theta I (two solves from a fixed pseudo-random
// start).  The vector is normalised and its sign chosen so that its first
// nonzero entry is positive.  Everything is fp64.
#include "slh_device.h"
#include "slh_internal.h"

#include <float.h>

namespace slh {

#define EIG_NMAX 256

__device__ int sturm_count(const double* al, const double* b2, int n, double x, double pivmin) {
  int cnt = 0;
  double d = al[0] - x;
  if (fabs(d) < pivmin) d = -pivmin;
  cnt += d < 0.0;
  for (int i = 1; i < n; ++i) {
    d = (al[i] - x) - b2[i - 1] / d;
    if (fabs(d) < pivmin) d = -pivmin;
    cnt += d < 0.0;
  }
  return cnt;
}

// theta: [n_act][r]; Seig: [n_act][n_it][r] (row k, kept column c)
__global__ __launch_bounds__(64) void k_tridiag_eig(const double* __restrict__ alpha,
                                                    const double* __restrict__ beta,
                                                    const int* __restrict__ neff, int n_it,
                                                    int r, double* __restrict__ theta,
                                                    double* __restrict__ Seig) {
  const int c = blockIdx.x, a = blockIdx.y, lane = threadIdx.x;
  const int n = neff[a];
  const int r_eff = min(r, n);
  double* Sa = Seig + (int64_t)a * n_it * r;
  if (c < r - r_eff) {
    for (int k = lane; k < n_it; k += 64) Sa[(int64_t)k * r + c] = 0.0;
    if (lane == 0) theta[(int64_t)a * r + c] = 0.0;
    return;
  }
  const int kidx = n - r + c;   // ascending index of the wanted eigenvalue
  __shared__ double al[EIG_NMAX], b1[EIG_NMAX], b2[EIG_NMAX];
  __shared__ double y[EIG_NMAX];
  __shared__ double fu1[EIG_NMAX], fu2[EIG_NMAX], fd[EIG_NMAX], fl[EIG_NMAX];
  __shared__ int piv[EIG_NMAX];
  const double* alp = alpha + (int64_t)a * n_it;
  const double* bet = beta + (int64_t)a * n_it;
  for (int k = lane; k < n; k += 64) {
    al[k] = alp[k];
    double b = (k < n - 1) ? bet[k] : 0.0;
    b1[k] = b;
    b2[k] = b * b;
  }
  __syncthreads();
  // Gershgorin bounds and the pivot floor
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
  // multisection: count(lo) <= kidx < count(hi)
  for (int it = 0; it < 64; ++it) {
    const double wdt = hi - lo;
    if (wdt <= 2.0 * DBL_EPSILON * fmax(fabs(lo), fabs(hi)) + pivmin) break;
    const double x = lo + wdt * ((double)(lane + 1) / 65.0);
    const int cnt = sturm_count(al, b2, n, x, pivmin);
    const unsigned long long mask = __ballot(cnt > kidx);
    double nlo = lo, nhi = hi;
    if (mask) {
      const int f = __ffsll((long long)mask) - 1;
      nhi = __shfl(x, f, 64);
      if (f > 0) nlo = __shfl(x, f - 1, 64);
    } else {
      nlo = __shfl(x, 63, 64);
    }
    if (!(nhi - nlo < wdt)) break;   // no progress (bracket at rounding level)
    lo = nlo;
    hi = nhi;
  }
  const double th = 0.5 * (lo + hi);

  // inverse iteration on lane 0 (tridiagonal LU with partial pivoting)
  if (lane == 0) {
    const double eps_piv = DBL_EPSILON * fmax(tnorm, DBL_MIN);
    // factor T - th I = P L U; U has diagonal fd, superdiagonals fu1, fu2
    double dcur = al[0] - th, ucur = (n > 1) ? b1[0] : 0.0;
    for (int k = 0; k < n - 1; ++k) {
      const double sub = b1[k];                   // entry (k+1, k)
      const double dnext = al[k + 1] - th;
      const double unext = (k + 1 < n - 1) ? b1[k + 1] : 0.0;
      if (fabs(dcur) >= fabs(sub)) {
        // no interchange
        if (fabs(dcur) < eps_piv) dcur = (dcur < 0.0 ? -eps_piv : eps_piv);
        const double l = sub / dcur;
        fd[k] = dcur;
        fu1[k] = ucur;
        fu2[k] = 0.0;
        fl[k] = l;
        piv[k] = 0;
        dcur = dnext - l * ucur;
        ucur = unext;
      } else {
        // swap rows k and k+1
        const double l = dcur / sub;
        fd[k] = sub;
        fu1[k] = dnext;
        fu2[k] = unext;
        fl[k] = l;
        piv[k] = 1;
        dcur = ucur - l * dnext;
        ucur = -l * unext;
      }
    }
    if (fabs(dcur) < eps_piv) dcur = (dcur < 0.0 ? -eps_piv : eps_piv);
    fd[n - 1] = dcur;
    fu1[n - 1] = 0.0;
    fu2[n - 1] = 0.0;
    // start vector: fixed pseudo-random entries in [-1, 1)
    for (int k = 0; k < n; ++k) {
      unsigned h = (unsigned)(k + 1) * 2654435761u;
      h ^= h >> 15;
      h *= 2246822519u;
      h ^= h >> 13;
      y[k] = (double)(h >> 8) * (2.0 / 16777216.0) - 1.0;
    }
    for (int itr = 0; itr < 2; ++itr) {
      // forward: apply L^{-1} P
      for (int k = 0; k < n - 1; ++k) {
        if (piv[k]) {
          const double t = y[k];
          y[k] = y[k + 1];
          y[k + 1] = t - fl[k] * y[k];
        } else {
          y[k + 1] -= fl[k] * y[k];
        }
      }
      // backward: U x = y
      for (int k = n - 1; k >= 0; --k) {
        double v = y[k];
        if (k + 1 < n) v -= fu1[k] * y[k + 1];
        if (k + 2 < n) v -= fu2[k] * y[k + 2];
        y[k] = v / fd[k];
      }
      double mx = 0.0;
      for (int k = 0; k < n; ++k) mx = fmax(mx, fabs(y[k]));
      const double inv = mx > 0.0 ? 1.0 / mx : 1.0;
      for (int k = 0; k < n; ++k) y[k] *= inv;
    }
    double nr = 0.0;
    for (int k = 0; k < n; ++k) nr = fma(y[k], y[k], nr);
    double sc = 1.0 / sqrt(nr);
    int first = 0;
    while (first < n - 1 && y[first] == 0.0) ++first;
    if (y[first] < 0.0) sc = -sc;
    for (int k = 0; k < n; ++k) y[k] *= sc;
    theta[(int64_t)a * r + c] = th;
  }
  __syncthreads();
  for (int k = lane; k < n_it; k += 64) Sa[(int64_t)k * r + c] = (k < n) ? y[k] : 0.0;
}

hipError_t launch_tridiag_eig(const double* alpha, const double* beta, const int* neff,
                              int n_act, int n_it, int r, double* theta, double* Seig,
                              hipStream_t s) {
  (void)hipGetLastError();
  hipLaunchKernelGGL(k_tridiag_eig, dim3(r, n_act), dim3(64), 0, s, alpha, beta, neff, n_it, r,
                     theta, Seig);
  return hipGetLastError();
}

// Z[a][i][c] = sum_{k < n_eff} Q[a][k][i] Seig[a][k][c]   (fp64).
// Thread = (row, group of 16 columns); S is staged through LDS 32 rows at a time.
__global__ __launch_bounds__(256) void k_ritz(const double* __restrict__ Q,
                                              const double* __restrict__ Seig,
                                              const int* __restrict__ neff, int L, int ldq,
                                              int n_it, int r, double* __restrict__ Z) {
  const int a = blockIdx.y, tid = threadIdx.x;
  const int n = neff[a];
  const int cgroups = (r + 15) / 16;
  const int rpb = 256 / cgroups;
  const int cg = tid % cgroups;
  const int i = blockIdx.x * rpb + tid / cgroups;
  const bool active = (tid / cgroups) < rpb && i < L;
  const double* Qa = Q + (int64_t)a * ldq * L;
  const double* Sa = Seig + (int64_t)a * n_it * r;
  __shared__ double sS[32 * 128];
  double acc[16];
#pragma unroll
  for (int c = 0; c < 16; ++c) acc[c] = 0.0;
  for (int k0 = 0; k0 < n; k0 += 32) {
    const int nk = min(32, n - k0);
    for (int e = tid; e < nk * r; e += 256) sS[(e / r) * 128 + (e % r)] = Sa[(int64_t)(k0 + e / r) * r + (e % r)];
    __syncthreads();
    if (active) {
      for (int kk = 0; kk < nk; ++kk) {
        const double q = Qa[(int64_t)(k0 + kk) * L + i];
        const double* srow = sS + kk * 128 + cg * 16;
#pragma unroll
        for (int c = 0; c < 16; ++c) acc[c] = fma(q, srow[c], acc[c]);
      }
    }
    __syncthreads();
  }
  if (active) {
    double* zr = Z + ((int64_t)a * L + i) * r + cg * 16;
#pragma unroll
    for (int c = 0; c < 16; ++c)
      if (cg * 16 + c < r) zr[c] = acc[c];
  }
}

hipError_t launch_ritz(const double* Q, const double* Seig, const int* neff, int n_act, int L,
                       int ldq, int n_it, int r, double* Z, hipStream_t s) {
  (void)hipGetLastError();
  const int cgroups = (r + 15) / 16;
  const int rpb = 256 / cgroups;
  hipLaunchKernelGGL(k_ritz, dim3((unsigned)((L + rpb - 1) / rpb), n_act), dim3(256), 0, s, Q,
                     Seig, neff, L, ldq, n_it, r, Z);
  return hipGetLastError();
}

}  // namespace slh
