// Short windows (the local backend of section 3.5, default window 16 in
// section 5.1): the whole spectral step of one window -- Lanczos with full
// re-orthogonalisation on the window's operator (Algorithm 2), Eigh of the
// tridiagonal matrix and the top-r Ritz coordinates (Algorithm 1) -- in one
// 64-lane wavefront per window.
//
// For L <= 32 tokens the operator Phi_w Phi_w^T is an L x L matrix.  It is formed
// once in fp64 from the window's fp32 feature rows (Phi is read once), after
// which every Lanczos matvec is an L x L product held in registers.  The Krylov
// recurrence, the breakdown rule and the column and sign conventions are those
// of the long-sequence path; only the summation order of the matvec differs
// (the operator is the same).
//
// Eigh(T): each kept eigenvalue is isolated by Sturm-count multisection (GR
// lanes x PPL probes per round), its eigenvector by inverse iteration with a
// partially pivoted LU of T - theta I.  Eigenvalues closer than 1e-6 |T| form
// clusters whose vectors are computed one after another, each orthogonalised
// against the cluster's earlier vectors inside every iteration, so that the
// basis stays orthonormal also where Ritz values coincide (a null space inside
// the Krylov space).  Everything after the feature map is fp64.  A window is a
// serial chain of dependent steps, so the kernel is latency-bound: reductions
// use DPP lane permutations and the scalar unit rather than LDS round trips.
#include "slh_device.h"
#include "slh_internal.h"

#include <float.h>

namespace slh {

// ---- wavefront arithmetic -------------------------------------------------
// v from the lane given by the DPP control CTRL (all rows and banks enabled)
template <int CTRL>
__device__ __forceinline__ double dpp_f64(double v) {
  const int lo = __builtin_amdgcn_mov_dpp(__double2loint(v), CTRL, 0xF, 0xF, false);
  const int hi = __builtin_amdgcn_mov_dpp(__double2hiint(v), CTRL, 0xF, 0xF, false);
  return __hiloint2double(hi, lo);
}
constexpr int DPP_XOR1 = 0xB1;          // quad_perm [1, 0, 3, 2]
constexpr int DPP_XOR2 = 0x4E;          // quad_perm [2, 3, 0, 1]
constexpr int DPP_HALF_MIRROR = 0x141;  // lane i <-> 7 - i within each 8
constexpr int DPP_MIRROR = 0x140;       // lane i <-> 15 - i within each 16

__device__ __forceinline__ double lane_f64(double v, int l) {
  return __hiloint2double(__builtin_amdgcn_readlane(__double2hiint(v), l),
                          __builtin_amdgcn_readlane(__double2loint(v), l));
}

// Sum over the GR consecutive lanes that share a row; each pair of partners adds
// the same two values, so every lane of the group ends with the same bits.
template <int GR>
__device__ __forceinline__ double group_sum(double v) {
  if constexpr (GR >= 2) v += dpp_f64<DPP_XOR1>(v);
  if constexpr (GR >= 4) v += dpp_f64<DPP_XOR2>(v);
  return v;
}

// Sum over all 64 lanes, identical in every lane: within quads and rows of 16
// by DPP, then the four row sums through the scalar unit in a fixed order.
__device__ __forceinline__ double wave_allsum(double v) {
  v += dpp_f64<DPP_XOR1>(v);
  v += dpp_f64<DPP_XOR2>(v);
  v += dpp_f64<DPP_HALF_MIRROR>(v);
  v += dpp_f64<DPP_MIRROR>(v);
  return (lane_f64(v, 0) + lane_f64(v, 16)) + (lane_f64(v, 32) + lane_f64(v, 48));
}

__device__ __forceinline__ double rcp_refined(double d) {
  const double r = __builtin_amdgcn_rcp(d);
  return fma(r, fma(-d, r, 1.0), r);
}

// LM: the largest window length the instance handles (16 or 32).  Lane l owns
// row i = l / GR of the operator and its columns [p JC, (p + 1) JC), p = l % GR;
// in the eigensolve the same GR lanes serve kept column c = i.
template <int LM>
__global__ __launch_bounds__(64) void k_local(const float* __restrict__ Phi, int m, int L, int n_it,
                                              int r, double tol, const double* __restrict__ q1,
                                              double* __restrict__ Q, double* __restrict__ alpha,
                                              double* __restrict__ beta, int* __restrict__ neff,
                                              double* __restrict__ theta, double* __restrict__ Z) {
  constexpr int GR = 64 / LM, JC = LM / GR;
  constexpr int GC = 64;                     // feature columns staged at a time
  constexpr int PPL = 2;                     // multisection probes per lane
  constexpr int NPR = GR * PPL;              // probes per eigenvalue per round
  const int a = blockIdx.x, lane = threadIdx.x;
  const int i = lane / GR, p = lane % GR, jb = p * JC;
  const int ldq = n_it + 1;

  __shared__ double sPd[GC][LM + 1];         // feature columns (fp64), column-major
  __shared__ double sQ[LM + 1][LM + 1];      // Lanczos basis, vector-major
  __shared__ double sv[LM], sh[LM + 1], sal[LM], sbe[LM], sth[LM];
  __shared__ double sS[LM][LM + 1];          // eigenvectors: [k][kept column]

  // unused basis rows must read as zero in the Gram-Schmidt products
  for (int e = lane; e < (LM + 1) * (LM + 1); e += 64) (&sQ[0][0])[e] = 0.0;

  // ---- the window's operator A = Phi_w Phi_w^T (fp64 sums of exact products).
  // Feature columns arrive 256 at a time (every load of a chunk in flight at
  // once) and pass through LDS as fp64, 64 columns at a time.
  double A[JC];
#pragma unroll
  for (int t = 0; t < JC; ++t) A[t] = 0.0;
  const float* Pa = Phi + (int64_t)a * L * m;
  for (int c0 = 0; c0 < m; c0 += 256) {
    // item u = sub-chunk s (64 columns) x t: float4 e = t * 64 + lane of the
    // sub-chunk's LM x 16 float4, row e / 16, column 64 s + 4 (e % 16)
    float4 v[LM];
#pragma unroll
    for (int u = 0; u < LM; ++u) {
      const int s4 = u / (LM / 4), e = (u % (LM / 4)) * 64 + lane;
      const int row = e / 16, col = c0 + 64 * s4 + 4 * (e % 16);
      // unconditional load (rows past the window re-read its last row, whose
      // finite values are then scaled to zero): a load under a guard would be
      // issued alone and waited for before the next one
      const float4 t4 = *(const float4*)(Pa + (int64_t)min(row, L - 1) * m + col);
      const float keep = (row < L) ? 1.0f : 0.0f;
      v[u] = make_float4(t4.x * keep, t4.y * keep, t4.z * keep, t4.w * keep);
    }
#pragma unroll
    for (int s4 = 0; s4 < 4; ++s4) {
#pragma unroll
      for (int t = 0; t < LM / 4; ++t) {
        const int e = t * 64 + lane, row = e / 16, cl = 4 * (e % 16);
        const float4 x = v[s4 * (LM / 4) + t];
        sPd[cl][row] = x.x;
        sPd[cl + 1][row] = x.y;
        sPd[cl + 2][row] = x.z;
        sPd[cl + 3][row] = x.w;
      }
      __syncthreads();
#pragma unroll 4
      for (int cc = 0; cc < GC; ++cc) {
        const double xi = sPd[cc][i];
#pragma unroll
        for (int t = 0; t < JC; ++t) A[t] = fma(xi, sPd[cc][jb + t], A[t]);
      }
      __syncthreads();
    }
  }

  // ---- Lanczos with two classical Gram-Schmidt passes (rows >= L stay zero)
  double qi = (i < L) ? q1[(int64_t)a * L + i] : 0.0;
  if (p == 0) sQ[0][i] = qi;
  __syncthreads();
  double qprev = 0.0, bprev = 0.0, amax = 0.0;
  int n = n_it;
  bool broke = false;
  for (int j = 0; j < n_it; ++j) {
    // this lane's entries of q_j, of basis vector i and of basis vectors jb.. at
    // row i, read once per step (the basis does not change within the step)
    double qj[JC], qrow[JC], qcol[JC];
#pragma unroll
    for (int t = 0; t < JC; ++t) {
      qj[t] = sQ[j][jb + t];
      qrow[t] = sQ[i][jb + t];
      qcol[t] = sQ[jb + t][i];
    }
    double zp = 0.0;
#pragma unroll
    for (int t = 0; t < JC; ++t) zp = fma(A[t], qj[t], zp);
    double z = group_sum<GR>(zp);
    const double al = wave_allsum(p == 0 ? qi * z : 0.0);
    z = z - al * qi;
    z = z - bprev * qprev;
#pragma unroll 1
    for (int pass = 0; pass < 2; ++pass) {
      if (p == 0) sv[i] = z;
      __syncthreads();
      double hp = 0.0;                        // h_k for k = i over this lane's entries of z
#pragma unroll
      for (int t = 0; t < JC; ++t) hp = fma(qrow[t], sv[jb + t], hp);
      const double h = group_sum<GR>(hp);
      if (p == 0) sh[i] = (i <= j) ? h : 0.0;
      __syncthreads();
      double cp = 0.0;                        // (Q h)_i over this lane's range of k
#pragma unroll
      for (int t = 0; t < JC; ++t) cp = fma(qcol[t], sh[jb + t], cp);
      z -= group_sum<GR>(cp);
    }
    const double b = sqrt(wave_allsum(p == 0 ? z * z : 0.0));
    amax = fmax(amax, fabs(al));
    if (lane == 0) {
      sal[j] = al;
      sbe[j] = b;
    }
    if (b <= tol * amax) {
      n = j + 1;
      broke = true;
      break;
    }
    qprev = qi;
    bprev = b;
    qi = z / b;
    if (p == 0) sQ[j + 1][i] = qi;
    __syncthreads();
  }
  __syncthreads();

  // ---- outputs of the Krylov phase
  for (int k = lane; k < n_it; k += 64) {
    alpha[(int64_t)a * n_it + k] = (k < n) ? sal[k] : 0.0;
    beta[(int64_t)a * n_it + k] = (k < n) ? sbe[k] : 0.0;
  }
  if (lane == 0) neff[a] = n;
  {
    double* Qa = Q + (int64_t)a * ldq * L;
    const int kmax = broke ? n : n + 1;       // q_{n+1} exists only without breakdown
    for (int e = lane; e < ldq * L; e += 64) {
      const int k = e / L, ii = e - k * L;
      Qa[e] = (k < kmax) ? sQ[k][ii] : 0.0;
    }
  }

  // ---- Eigh(T): T = tridiag(beta_0..beta_{n-2}; alpha_0..alpha_{n-1}; same).
  // T lives in registers (ak, bk; zero past the matrix) and every loop over its
  // rows is unrolled to LM with uniform guards, so the serial recurrences below
  // never wait on LDS.
  double ak[LM], bk[LM];
#pragma unroll
  for (int k = 0; k < LM; ++k) {
    ak[k] = (k < n) ? sal[k] : 0.0;
    bk[k] = (k < n - 1) ? sbe[k] : 0.0;
  }
  // Gershgorin interval, |T| bound and pivot floor (every lane, same order)
  double glo = DBL_MAX, ghi = -DBL_MAX, tnorm = 0.0, bmax = 0.0;
#pragma unroll
  for (int k = 0; k < LM; ++k) {
    if (k < n) {
      const double bl = (k > 0) ? fabs(bk[k - 1]) : 0.0, br = fabs(bk[k]);
      glo = fmin(glo, ak[k] - (bl + br));
      ghi = fmax(ghi, ak[k] + (bl + br));
      tnorm = fmax(tnorm, fabs(ak[k]) + (bl + br));
      bmax = fmax(bmax, br * br);
    }
  }
  const double pivmin = DBL_MIN * fmax(1.0, bmax);
  const double atol = 2.0 * DBL_EPSILON * fmax(tnorm, DBL_MIN) + pivmin;
  glo -= atol;
  ghi += atol;
  const int r_eff = min(r, n);
  const int c = i;                              // kept column of this lane group
  const bool valid = (c < r) && (c >= r - r_eff);
  const int kidx = n - r + c;                   // ascending index of its eigenvalue
  // multisection: count(lo) <= kidx < count(hi); probe q of the group at
  // lo + (hi - lo) (q + 1) / (NPR + 1), q = p * PPL + s
  double lo = glo, hi = ghi;
  bool done = !valid;
#pragma unroll 1
  for (int it = 0; it < 96; ++it) {
    if (!(hi - lo > atol)) done = true;
    if (__ballot(!done) == 0ull) break;
    const double step = (hi - lo) * (1.0 / (double)(NPR + 1));
    double d[PPL], x[PPL];
    int cnt[PPL];
#pragma unroll
    for (int s = 0; s < PPL; ++s) {
      x[s] = lo + step * (double)(p * PPL + s + 1);
      d[s] = ak[0] - x[s];
      if (fabs(d[s]) < pivmin) d[s] = -pivmin;
      cnt[s] = d[s] < 0.0;
    }
#pragma unroll
    for (int k = 1; k < LM; ++k) {
      if (k < n) {
        const double b2 = bk[k - 1] * bk[k - 1];
#pragma unroll
        for (int s = 0; s < PPL; ++s) {
          d[s] = fma(-b2, rcp_refined(d[s]), ak[k] - x[s]);
          if (fabs(d[s]) < pivmin) d[s] = -pivmin;
          cnt[s] += d[s] < 0.0;
        }
      }
    }
    // first probe of the group whose count exceeds kidx (probes ascend with
    // q = p * PPL + s); bit s * GR + p of gm is probe p * PPL + s
    unsigned gm = 0;
#pragma unroll
    for (int s = 0; s < PPL; ++s) {
      const unsigned long long bm = __ballot(cnt[s] > kidx);
      gm |= (unsigned)((bm >> (i * GR)) & ((1ull << GR) - 1)) << (s * GR);
    }
    unsigned ord = 0;
#pragma unroll
    for (int s = 0; s < PPL; ++s)
#pragma unroll
      for (int pp = 0; pp < GR; ++pp) ord |= ((gm >> (s * GR + pp)) & 1u) << (pp * PPL + s);
    const int f = ord ? __ffs(ord) - 1 : NPR;
    if (!done) {
      const double nlo = (f > 0) ? lo + step * (double)f : lo;
      const double nhi = (f < NPR) ? lo + step * (double)(f + 1) : hi;
      if (!(nhi - nlo < hi - lo)) done = true;   // bracket at rounding level
      lo = nlo;
      hi = nhi;
    }
  }
  const double th = 0.5 * (lo + hi);
  if (p == 0) sth[c] = th;
  __syncthreads();
  // cluster level: number of directly preceding kept eigenvalues within 1e-6 |T|
  const double ctol = 1e-6 * tnorm;
  int level = 0;
  if (valid)
    while (c - level - 1 >= r - r_eff && th - sth[c - level - 1] <= ctol) ++level;
  int maxlev = level;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) maxlev = max(maxlev, __shfl_xor(maxlev, o, 64));
  const double eps_piv = DBL_EPSILON * fmax(tnorm, DBL_MIN);
#pragma unroll 1
  for (int lev = 0; lev <= maxlev; ++lev) {
    if (valid && p == 0 && level == lev) {
      // start: fixed pseudo-random entries in [-1, 1)
      double y[LM], fd[LM], fu1[LM];
#pragma unroll
      for (int k = 0; k < LM; ++k) {
        unsigned hsh = (unsigned)(k + 1 + 977 * lev) * 2654435761u;
        hsh ^= hsh >> 15;
        hsh *= 2246822519u;
        hsh ^= hsh >> 13;
        y[k] = (double)(hsh >> 8) * (2.0 / 16777216.0) - 1.0;
        fd[k] = 0.0;
        fu1[k] = 0.0;
      }
#pragma unroll 1
      for (int itr = 0; itr < 2; ++itr) {
        // LU of T - th I with partial pivoting (row k + 1 swapped up when its
        // entry in column k is larger), eliminating the right-hand side y in the
        // same pass: y[k] becomes the transformed right-hand side of pivot row k,
        // fd[k] the inverted pivot, fu1[k] / fu2_k the two entries right of it
        // (fu2_k = bk[k + 1] exactly where rows were swapped)
        double dcur = ak[0] - th, ucur = bk[0], ycur = y[0];
        unsigned swapm = 0;
#pragma unroll
        for (int k = 0; k < LM - 1; ++k) {
          if (k < n - 1) {
            const double sub = bk[k], dnext = ak[k + 1] - th, unext = bk[k + 1], ynext = y[k + 1];
            const bool swap = fabs(dcur) < fabs(sub);
            if (!swap && fabs(dcur) < eps_piv) dcur = (dcur < 0.0) ? -eps_piv : eps_piv;
            const double ip = rcp_refined(swap ? sub : dcur);
            const double l = (swap ? dcur : sub) * ip;
            fd[k] = ip;
            fu1[k] = swap ? dnext : ucur;
            y[k] = swap ? ynext : ycur;
            swapm |= (unsigned)swap << k;
            const double nd = swap ? fma(-l, dnext, ucur) : fma(-l, ucur, dnext);
            ycur = swap ? fma(-l, ynext, ycur) : fma(-l, ycur, ynext);
            ucur = swap ? -l * unext : unext;
            dcur = nd;
          }
        }
        if (fabs(dcur) < eps_piv) dcur = (dcur < 0.0) ? -eps_piv : eps_piv;
        double x1 = ycur * rcp_refined(dcur), x2 = 0.0;   // x_{n-1}
        double mx = fabs(x1);
#pragma unroll
        for (int k = 0; k < LM; ++k)
          if (k == n - 1) y[k] = x1;
#pragma unroll
        for (int k = LM - 2; k >= 0; --k) {
          if (k < n - 1) {
            const double fu2 = ((swapm >> k) & 1u) ? bk[k + 1] : 0.0;
            const double xk = ((y[k] - fu1[k] * x1) - fu2 * x2) * fd[k];
            y[k] = xk;
            mx = fmax(mx, fabs(xk));
            x2 = x1;
            x1 = xk;
          }
        }
        // orthogonalise against the cluster's earlier vectors (modified Gram-Schmidt)
        for (int cq = c - level; cq < c; ++cq) {
          double dt = 0.0;
#pragma unroll
          for (int k = 0; k < LM; ++k)
            if (k < n) dt = fma(sS[k][cq], y[k], dt);
          mx = 0.0;
#pragma unroll
          for (int k = 0; k < LM; ++k)
            if (k < n) {
              y[k] = fma(-dt, sS[k][cq], y[k]);
              mx = fmax(mx, fabs(y[k]));
            }
        }
        const double inv = (mx > 0.0) ? 1.0 / mx : 1.0;
#pragma unroll
        for (int k = 0; k < LM; ++k) y[k] *= inv;
      }
      // unit norm; the first nonzero entry positive
      double nr = 0.0, firstv = 0.0;
#pragma unroll
      for (int k = 0; k < LM; ++k)
        if (k < n) {
          nr = fma(y[k], y[k], nr);
          if (firstv == 0.0) firstv = y[k];
        }
      double sc = (nr > 0.0) ? 1.0 / sqrt(nr) : 0.0;
      if (firstv < 0.0) sc = -sc;
#pragma unroll
      for (int k = 0; k < LM; ++k)
        if (k < n) sS[k][c] = y[k] * sc;
    }
    __syncthreads();
  }
  if (p == 0 && c < r) theta[(int64_t)a * r + c] = valid ? th : 0.0;

  // ---- Ritz coordinates Z = Q S[:, n - r : n] (leading columns zero when r > n)
  for (int e = lane; e < L * r; e += 64) {
    const int ii = e / r, cc = e - ii * r;
    double zv = 0.0;
    if (cc >= r - r_eff)
      for (int k = 0; k < n; ++k) zv = fma(sQ[k][ii], sS[k][cc], zv);
    Z[((int64_t)a * L + ii) * r + cc] = zv;
  }
}

bool local_supported(int L, int n_it, int r) {
  return L >= 1 && L <= 32 && n_it <= L && r <= n_it;
}

hipError_t launch_local(const float* Phi, int n_act, int m, int L, int n_it, int r, double tol,
                        const double* q1, double* Q, double* alpha, double* beta, int* neff,
                        double* theta, double* Z, hipStream_t s) {
  (void)hipGetLastError();
  if (!local_supported(L, n_it, r) || m % 256 != 0) return hipErrorInvalidValue;
  if (n_act <= 0) return hipSuccess;
  if (L <= 16)
    hipLaunchKernelGGL(k_local<16>, dim3(n_act), dim3(64), 0, s, Phi, m, L, n_it, r, tol, q1, Q,
                       alpha, beta, neff, theta, Z);
  else
    hipLaunchKernelGGL(k_local<32>, dim3(n_act), dim3(64), 0, s, Phi, m, L, n_it, r, tol, q1, Q,
                       alpha, beta, neff, theta, Z);
  return hipGetLastError();
}

}  // namespace slh
