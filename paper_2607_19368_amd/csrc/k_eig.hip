// Eigh(T) for the Lanczos tridiagonal and the top-r Ritz coordinates
// (Algorithm 1: lambda, V = Eigh(T); Z = Q V[:, n-k:n]).
//
// Eigenvalues: one 256-thread workgroup per kept eigenvalue isolates it by
// Sturm-count multisection (256 probe points per round, one per thread; the
// count of negative pivots of T - x I is the number of eigenvalues below x)
// until the bracket is a few ulps wide.
// Eigenvectors: one workgroup per kept eigenvalue, inverse iteration with a
// partially pivoted LU of T - theta I from a start vector of its own.  Two
// vectors computed this way for eigenvalues g apart are orthogonal only to
// about 6e-18 |T| / g (measured on Wilkinson's W21+), and for (numerically)
// repeated eigenvalues they are independent directions of the eigenspace
// rather than an orthonormal basis of it.  So kept eigenvalues whose
// consecutive gaps are at most EIG_CLUSTER |T| (|T| the Gershgorin bound) form
// clusters, and one workgroup per window then orthonormalises each cluster's
// vectors in ascending order (modified Gram-Schmidt, two passes).  Outside
// clusters the vectors are orthogonal to about 6e-12.  Each vector is
// normalised and its sign chosen so that its first nonzero entry is positive.
// Everything is fp64.
#include "slh_device.h"
#include "slh_internal.h"

#include <float.h>

namespace slh {

#define EIG_NMAX 256
#define EIG_CLUSTER 1e-6

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

// T of window a into LDS (al: diagonal, b1: off-diagonal, b2: its squares) and
// its Gershgorin interval [lo, hi], |T| bound tnorm and largest b^2 (every wave
// computes the same values).
struct TriInfo {
  double lo, hi, tnorm, bmax;
};
__device__ __forceinline__ TriInfo load_tridiag(const double* __restrict__ alp,
                                                const double* __restrict__ bet, int n, double* al,
                                                double* b1, double* b2) {
  const int tid = threadIdx.x, lane = tid & 63;
  for (int k = tid; k < n; k += EIG_T) {
    al[k] = alp[k];
    const double b = (k < n - 1) ? bet[k] : 0.0;
    b1[k] = b;
    b2[k] = b * b;
  }
  __syncthreads();
  TriInfo t;
  t.lo = DBL_MAX;
  t.hi = -DBL_MAX;
  t.bmax = 0.0;
  t.tnorm = 0.0;
  for (int k = lane; k < n; k += 64) {
    const double off = fabs(b1[k]) + (k > 0 ? fabs(b1[k - 1]) : 0.0);
    t.lo = fmin(t.lo, al[k] - off);
    t.hi = fmax(t.hi, al[k] + off);
    t.bmax = fmax(t.bmax, b2[k]);
    t.tnorm = fmax(t.tnorm, fabs(al[k]) + off);
  }
  for (int o = 32; o >= 1; o >>= 1) {
    t.lo = fmin(t.lo, __shfl_xor(t.lo, o, 64));
    t.hi = fmax(t.hi, __shfl_xor(t.hi, o, 64));
    t.bmax = fmax(t.bmax, __shfl_xor(t.bmax, o, 64));
    t.tnorm = fmax(t.tnorm, __shfl_xor(t.tnorm, o, 64));
  }
  return t;
}

// theta: [n_act][r], ascending kept eigenvalues (zero for the r - r_eff
// leading columns of a window that stopped after n_eff < r steps).
__global__ __launch_bounds__(EIG_T) void k_eig_values(const double* __restrict__ alpha,
                                                      const double* __restrict__ beta,
                                                      const int* __restrict__ neff, int n_it,
                                                      int r, double* __restrict__ theta) {
  const int c = blockIdx.x, a = blockIdx.y, tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int n = neff[a];
  const int r_eff = min(r, n);
  if (c < r - r_eff) {
    if (tid == 0) theta[(int64_t)a * r + c] = 0.0;
    return;
  }
  const int kidx = n - r + c;   // ascending index of the wanted eigenvalue
  __shared__ double al[EIG_NMAX], b1[EIG_NMAX], b2[EIG_NMAX];
  __shared__ unsigned long long smask[EIG_T / 64];
  const TriInfo ti = load_tridiag(alpha + (int64_t)a * n_it, beta + (int64_t)a * n_it, n, al, b1, b2);
  const double pivmin = DBL_MIN * fmax(1.0, ti.bmax);
  const double pad = 2.0 * DBL_EPSILON * fmax(ti.tnorm, DBL_MIN) + 2.0 * pivmin;
  double lo = ti.lo - pad, hi = ti.hi + pad;
  // multisection: count(lo) <= kidx < count(hi); EIG_T probes per round,
  // probe p at lo + (hi - lo) (p + 1) / (EIG_T + 1), evaluated by thread p.
  // The bracket is narrowed to 2 eps max(|theta|, |T|): the Sturm count is
  // exact only for a matrix within about eps |T| of T, so narrower brackets of
  // small eigenvalues would not make them more accurate.
  const double wstop = 2.0 * DBL_EPSILON * ti.tnorm + pivmin;
  for (int it = 0; it < 64; ++it) {
    const double wdt = hi - lo;
    if (wdt <= fmax(2.0 * DBL_EPSILON * fmax(fabs(lo), fabs(hi)) + pivmin, wstop)) break;
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
  if (tid == 0) theta[(int64_t)a * r + c] = 0.5 * (lo + hi);
}

// Unit norm and the sign rule (first nonzero entry positive) for y[0..n), into
// column k of Sa (rows n..n_it-1 zero); wave 0 only.
__device__ __forceinline__ void store_unit_column(const double* y, int n, int n_it, int r, int k,
                                                  double* Sa) {
  const int lane = threadIdx.x & 63;
  double nr = 0.0;
  int first = n - 1;
  for (int i = lane; i < n; i += 64) {
    nr = fma(y[i], y[i], nr);
    if (y[i] != 0.0 && i < first) first = i;
  }
  nr = wave_sum_f64(nr);
  for (int o = 32; o >= 1; o >>= 1) first = min(first, __shfl_xor(first, o, 64));
  double sc = 1.0 / sqrt(nr);
  if (y[first] < 0.0) sc = -sc;
  for (int i = lane; i < n_it; i += 64) Sa[(int64_t)i * r + k] = (i < n) ? y[i] * sc : 0.0;
}

// Seig: [n_act][n_it][r] (row k, kept column c); rows n_eff.. are zero.
__global__ __launch_bounds__(EIG_T) void k_eig_vectors(const double* __restrict__ alpha,
                                                       const double* __restrict__ beta,
                                                       const int* __restrict__ neff, int n_it,
                                                       int r, const double* __restrict__ theta,
                                                       double* __restrict__ Seig) {
  const int c = blockIdx.x, a = blockIdx.y, tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int n = neff[a];
  const int r_eff = min(r, n);
  double* Sa = Seig + (int64_t)a * n_it * r;
  if (c < r - r_eff) {
    for (int k = tid; k < n_it; k += EIG_T) Sa[(int64_t)k * r + c] = 0.0;
    return;
  }
  const double th = theta[(int64_t)a * r + c];
  __shared__ double al[EIG_NMAX], b1[EIG_NMAX], b2[EIG_NMAX];
  __shared__ double y[EIG_NMAX], w[EIG_NMAX];
  __shared__ double fu1[EIG_NMAX], fu2[EIG_NMAX], fd[EIG_NMAX], fl[EIG_NMAX];
  __shared__ int piv[EIG_NMAX];
  const TriInfo ti = load_tridiag(alpha + (int64_t)a * n_it, beta + (int64_t)a * n_it, n, al, b1, b2);
  // LU of T - th I with partial pivoting on thread 0; the triangular solves
  // carry the running entries in registers
  if (tid == 0) {
    const double eps_piv = DBL_EPSILON * fmax(ti.tnorm, DBL_MIN);
    // T - th I = P L U; U has diagonal fd (stored inverted), superdiagonals fu1,
    // fu2.  Row i+1 is swapped up when its entry in column i is larger; both
    // cases are computed branch-free.
    double dcur = al[0] - th, ucur = (n > 1) ? b1[0] : 0.0;
    for (int i = 0; i < n - 1; ++i) {
      const double sub = b1[i];                   // entry (i+1, i)
      const double dnext = al[i + 1] - th;
      const double unext = (i + 1 < n - 1) ? b1[i + 1] : 0.0;
      const bool swap = fabs(dcur) < fabs(sub);
      if (!swap && fabs(dcur) < eps_piv) dcur = (dcur < 0.0 ? -eps_piv : eps_piv);
      const double p = swap ? sub : dcur;         // pivot
      const double ip = rcp_nr(p);
      const double l = (swap ? dcur : sub) * ip;
      fd[i] = ip;
      fu1[i] = swap ? dnext : ucur;
      fu2[i] = swap ? unext : 0.0;
      fl[i] = l;
      piv[i] = swap;
      const double nd = swap ? fma(-l, dnext, ucur) : fma(-l, ucur, dnext);
      ucur = swap ? -l * unext : unext;
      dcur = nd;
    }
    if (fabs(dcur) < eps_piv) dcur = (dcur < 0.0 ? -eps_piv : eps_piv);
    fd[n - 1] = rcp_nr(dcur);
    fu1[n - 1] = 0.0;
    fu2[n - 1] = 0.0;
  }
  // start vector: fixed pseudo-random entries in [-1, 1), a different
  // sequence for each kept column (independent directions in a repeated
  // eigenspace)
  for (int i = tid; i < n; i += EIG_T) {
    unsigned h = (unsigned)(i + 1) * 2654435761u + (unsigned)c * 0x9E3779B9u;
    h ^= h >> 15;
    h *= 2246822519u;
    h ^= h >> 13;
    y[i] = (double)(h >> 8) * (2.0 / 16777216.0) - 1.0;
  }
  __syncthreads();
  for (int itr = 0; itr < 2; ++itr) {
    if (tid == 0) {
      // forward: apply L^{-1} P to y into w (cur = running entry i); input and
      // output arrays differ, so the loads run ahead of the recurrence
      double cur = y[0];
#pragma unroll 4
      for (int i = 0; i < n - 1; ++i) {
        const double nxt = y[i + 1], l = fl[i];
        const bool pk = piv[i];
        w[i] = pk ? nxt : cur;
        cur = pk ? fma(-l, nxt, cur) : fma(-l, cur, nxt);
      }
      w[n - 1] = cur;
      // backward: U x = w into y (x1 = x[i+1], x2 = x[i+2])
      double x1 = 0.0, x2 = 0.0;
#pragma unroll 4
      for (int i = n - 1; i >= 0; --i) {
        const double xi = ((w[i] - fu1[i] * x1) - fu2[i] * x2) * fd[i];
        y[i] = xi;
        x2 = x1;
        x1 = xi;
      }
    }
    __syncthreads();
    // rescale by the largest magnitude (every wave computes the same value)
    double mx = 0.0;
    for (int i = lane; i < n; i += 64) mx = fmax(mx, fabs(y[i]));
    for (int o = 32; o >= 1; o >>= 1) mx = fmax(mx, __shfl_xor(mx, o, 64));
    __syncthreads();
    const double inv = mx > 0.0 ? 1.0 / mx : 1.0;
    for (int i = tid; i < n; i += EIG_T) y[i] *= inv;
    __syncthreads();
  }
  if (wv == 0) store_unit_column(y, n, n_it, r, c, Sa);
}

// Per window: the kept columns of each cluster (consecutive kept eigenvalues
// at most EIG_CLUSTER |T| apart) orthonormalised in ascending order by
// modified Gram-Schmidt, two passes, against the cluster's earlier columns;
// then unit norm and the sign rule again.  Windows without clusters only read
// theta and T.
__global__ __launch_bounds__(EIG_T) void k_eig_orth(const double* __restrict__ alpha,
                                                    const double* __restrict__ beta,
                                                    const int* __restrict__ neff, int n_it, int r,
                                                    const double* __restrict__ theta,
                                                    double* __restrict__ Seig) {
  const int a = blockIdx.x, tid = threadIdx.x, wv = tid >> 6;
  const int n = neff[a];
  const int c_lo = r - min(r, n);
  double* Sa = Seig + (int64_t)a * n_it * r;
  __shared__ double al[EIG_NMAX], b1[EIG_NMAX], b2[EIG_NMAX];
  __shared__ double y[EIG_NMAX], tha[EIG_NMAX];
  __shared__ double red[EIG_T / 64];
  // the kept eigenvalues in LDS (the cluster scan below is sequential)
  for (int c = threadIdx.x; c < r; c += EIG_T) tha[c] = theta[(int64_t)a * r + c];
  const TriInfo ti = load_tridiag(alpha + (int64_t)a * n_it, beta + (int64_t)a * n_it, n, al, b1, b2);
  const double ctol = EIG_CLUSTER * ti.tnorm;
  for (int c = c_lo; c < r;) {
    int c1 = c;
    while (c1 + 1 < r && tha[c1 + 1] - tha[c1] <= ctol) ++c1;
    for (int k = c + 1; k <= c1; ++k) {
      if (tid < n) y[tid] = Sa[(int64_t)tid * r + k];
      __syncthreads();
      for (int pass = 0; pass < 2; ++pass) {
        for (int p = c; p < k; ++p) {
          const double sp = (tid < n) ? Sa[(int64_t)tid * r + p] : 0.0;
          const double d = block_sum_f64((tid < n) ? y[tid] * sp : 0.0, red);
          if (tid < n) y[tid] = fma(-d, sp, y[tid]);
          __syncthreads();
        }
      }
      if (wv == 0) store_unit_column(y, n, n_it, r, k, Sa);
      __syncthreads();               // column k is read for the next members
    }
    c = c1 + 1;
  }
}

hipError_t launch_tridiag_eig(const double* alpha, const double* beta, const int* neff,
                              int n_act, int n_it, int r, double* theta, double* Seig,
                              hipStream_t s) {
  (void)hipGetLastError();
  if (n_it > EIG_NMAX || r > n_it) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_eig_values, dim3(r, n_act), dim3(EIG_T), 0, s, alpha, beta, neff, n_it, r,
                     theta);
  hipLaunchKernelGGL(k_eig_vectors, dim3(r, n_act), dim3(EIG_T), 0, s, alpha, beta, neff, n_it,
                     r, theta, Seig);
  hipLaunchKernelGGL(k_eig_orth, dim3(n_act), dim3(EIG_T), 0, s, alpha, beta, neff, n_it, r, theta,
                     Seig);
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
