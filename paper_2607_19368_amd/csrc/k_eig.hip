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

  // inverse iteration: LU of T - th I with partial pivoting on lane 0; the
  // triangular solves carry the running entries in registers
  if (lane == 0) {
    const double eps_piv = DBL_EPSILON * fmax(tnorm, DBL_MIN);
    // T - th I = P L U; U has diagonal fd (stored inverted), superdiagonals fu1, fu2
    double dcur = al[0] - th, ucur = (n > 1) ? b1[0] : 0.0;
    for (int k = 0; k < n - 1; ++k) {
      const double sub = b1[k];                   // entry (k+1, k)
      const double dnext = al[k + 1] - th;
      const double unext = (k + 1 < n - 1) ? b1[k + 1] : 0.0;
      if (fabs(dcur) >= fabs(sub)) {
        // no interchange
        if (fabs(dcur) < eps_piv) dcur = (dcur < 0.0 ? -eps_piv : eps_piv);
        const double l = sub / dcur;
        fd[k] = 1.0 / dcur;
        fu1[k] = ucur;
        fu2[k] = 0.0;
        fl[k] = l;
        piv[k] = 0;
        dcur = dnext - l * ucur;
        ucur = unext;
      } else {
        // swap rows k and k+1
        const double l = dcur / sub;
        fd[k] = 1.0 / sub;
        fu1[k] = dnext;
        fu2[k] = unext;
        fl[k] = l;
        piv[k] = 1;
        dcur = ucur - l * dnext;
        ucur = -l * unext;
      }
    }
    if (fabs(dcur) < eps_piv) dcur = (dcur < 0.0 ? -eps_piv : eps_piv);
    fd[n - 1] = 1.0 / dcur;
    fu1[n - 1] = 0.0;
    fu2[n - 1] = 0.0;
  }
  // start vector: fixed pseudo-random entries in [-1, 1)
  for (int k = lane; k < n; k += 64) {
    unsigned h = (unsigned)(k + 1) * 2654435761u;
    h ^= h >> 15;
    h *= 2246822519u;
    h ^= h >> 13;
    y[k] = (double)(h >> 8) * (2.0 / 16777216.0) - 1.0;
  }
  __syncthreads();
  for (int itr = 0; itr < 2; ++itr) {
    if (lane == 0) {
      // forward: apply L^{-1} P (cur = running entry k)
      double cur = y[0];
      for (int k = 0; k < n - 1; ++k) {
        const double nxt = y[k + 1];
        if (piv[k]) {
          y[k] = nxt;
          cur = cur - fl[k] * nxt;
        } else {
          y[k] = cur;
          cur = nxt - fl[k] * cur;
        }
      }
      y[n - 1] = cur;
      // backward: U x = y (x1 = x[k+1], x2 = x[k+2])
      double x1 = 0.0, x2 = 0.0;
      for (int k = n - 1; k >= 0; --k) {
        const double xk = ((y[k] - fu1[k] * x1) - fu2[k] * x2) * fd[k];
        y[k] = xk;
        x2 = x1;
        x1 = xk;
      }
    }
    __syncthreads();
    double mx = 0.0;
    for (int k = lane; k < n; k += 64) mx = fmax(mx, fabs(y[k]));
    for (int o = 32; o >= 1; o >>= 1) mx = fmax(mx, __shfl_xor(mx, o, 64));
    const double inv = mx > 0.0 ? 1.0 / mx : 1.0;
    for (int k = lane; k < n; k += 64) y[k] *= inv;
    __syncthreads();
  }
  // unit norm; sign such that the first nonzero entry is positive
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

hipError_t launch_tridiag_eig(const double* alpha, const double* beta, const int* neff,
                              int n_act, int n_it, int r, double* theta, double* Seig,
                              hipStream_t s) {
  (void)hipGetLastError();
  hipLaunchKernelGGL(k_tridiag_eig, dim3(r, n_act), dim3(64), 0, s, alpha, beta, neff, n_it, r,
                     theta, Seig);
  return hipGetLastError();
}

// Z[a][i][c] = sum_{k < n_eff} Q[a][k][i] Seig[a][k][c]   (fp64).
// Thread = (row, group of 8 columns); S is staged through LDS 32 rows at a time
// (rows past n_eff zero-filled) and Q is read 8 rows of k at a time.
__global__ __launch_bounds__(256) void k_ritz(const double* __restrict__ Q,
                                              const double* __restrict__ Seig,
                                              const int* __restrict__ neff, int L, int ldq,
                                              int n_it, int r, double* __restrict__ Z) {
  const int a = blockIdx.y, tid = threadIdx.x;
  const int n = neff[a];
  const int cgroups = (r + 7) / 8;
  const int rpb = 256 / cgroups;
  const int cg = tid % cgroups;
  const int i = blockIdx.x * rpb + tid / cgroups;
  const bool active = (tid / cgroups) < rpb && i < L;
  const int ic = min(i, L - 1);
  const double* Qa = Q + (int64_t)a * ldq * L;
  const double* Sa = Seig + (int64_t)a * n_it * r;
  __shared__ double sS[32 * 128];
  double acc[8];
#pragma unroll
  for (int c = 0; c < 8; ++c) acc[c] = 0.0;
  for (int k0 = 0; k0 < n; k0 += 32) {
    const int nk = min(32, n - k0);
    for (int e = tid; e < 32 * 128; e += 256) {
      const int kr = e >> 7, c = e & 127;
      sS[e] = (kr < nk && c < r) ? Sa[(int64_t)(k0 + kr) * r + c] : 0.0;
    }
    __syncthreads();
    if (active) {
      for (int kk = 0; kk < nk; kk += 8) {
        double q[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) q[e] = Qa[(int64_t)min(k0 + kk + e, n - 1) * L + ic];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const double* srow = sS + (kk + e) * 128 + cg * 8;   // zero rows past nk
#pragma unroll
          for (int c = 0; c < 8; ++c) acc[c] = fma(q[e], srow[c], acc[c]);
        }
      }
    }
    __syncthreads();
  }
  if (active) {
    double* zr = Z + ((int64_t)a * L + i) * r + cg * 8;
#pragma unroll
    for (int c = 0; c < 8; ++c)
      if (cg * 8 + c < r) zr[c] = acc[c];
  }
}

hipError_t launch_ritz(const double* Q, const double* Seig, const int* neff, int n_act, int L,
                       int ldq, int n_it, int r, double* Z, hipStream_t s) {
  (void)hipGetLastError();
  const int cgroups = (r + 7) / 8;
  const int rpb = 256 / cgroups;
  hipLaunchKernelGGL(k_ritz, dim3((unsigned)((L + rpb - 1) / rpb), n_act), dim3(256), 0, s, Q,
                     Seig, neff, L, ldq, n_it, r, Z);
  return hipGetLastError();
}

}  // namespace slh
