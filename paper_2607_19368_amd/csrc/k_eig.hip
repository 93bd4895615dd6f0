// Eigh(T) for the Lanczos tridiagonal and the top-r Ritz coordinates
// (Algorithm 1: lambda, V = Eigh(T); Z = Q V[:, n-k:n]).
//
// One 256-thread workgroup per kept eigenpair (k_eig_pairs).  Its eigenvalue
// by Sturm-count multisection (256 probe points per round, one per thread; the
// sign changes along the leading principal minors of T - x I count the
// eigenvalues below x) until the bracket is a few ulps wide; then its vector.
// Eigenvalues more than EIG_TWIST_GAP |T| from every other eigenvalue of T
// (two more Sturm counts) take the twisted factorisation
// (twisted_vector: two pivot recurrences and two product recurrences, no
// iteration); the others inverse iteration with a partially pivoted LU of
// T - theta I from a start vector of its own.  Two
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

#include <algorithm>

namespace slh {

#define EIG_NMAX 256
#define EIG_CLUSTER 1e-6
#define EIG_TWIST_GAP 1e-9

// 1/d from the hardware reciprocal refined by one Newton step (d a normal number)
__device__ __forceinline__ double rcp_nr(double d) {
  const double r = __builtin_amdgcn_rcp(d);
  return fma(r, fma(-d, r, 1.0), r);
}

// Number of eigenvalues of T below x: the sign changes along the leading
// principal minors q_k = det(T_k - x I) (Sturm sequence), from q_(-1) = 0,
// q_0 = 1 and q_(k+1) = (alpha_k - x) q_k - beta_(k-1)^2 q_(k-1); a change at
// k is a negative pivot q_k / q_(k-1) of the LDL^T factorisation of T - x I.
// Each step's rounding errors are those of the pivot recurrence (a relative
// error on alpha_k - x and on the beta^2 term), but no division is needed.
// The caller scales T and x by a power of two so that |T| <= 1 (an exact
// scaling), stores an[k] = alpha_k and b2s[k] = beta_(k-1)^2 raised to at
// least EIG_B2MIN (b2s[0] unused), so that two consecutive minors never both
// vanish, and gives both arrays 8 entries beyond n rounded down to a multiple
// of 8.  The pair (q_k, q_(k-1)) is rescaled by a power of two every 8 steps:
// in 8 steps it grows at most 3^8 times and shrinks at most (EIG_B2MIN / 3)^8,
// far from overflow and underflow (raising beta^2 to EIG_B2MIN moves no
// eigenvalue by more than 2^-53 |T|).  A change is a difference of sign bits:
// each step shifts the sign of q_k into a mask, and every 8 steps the
// differences of neighbouring bits are counted.  An exact zero q_k needs no
// rule of its own: its neighbours q_(k-1) and q_(k+1) = -beta_(k-1)^2 q_(k-1)
// have opposite signs, so the pair of steps counts one change whatever the
// zero's sign bit (the pivot form counts a zero pivot as negative and the
// next one, of the same pair, as positive).
#define EIG_B2MIN 0x1p-110
__device__ __forceinline__ void minors_step(double a, double b2, double xn, double& pm, double& pc,
                                            uint32_t& sg) {
  const double pn = fma(a - xn, pc, -(b2 * pm));
  sg = __builtin_amdgcn_alignbit(sg, f64_hi(pn), 31);   // (sg << 1) | sign bit of q
  pm = pc;
  pc = pn;
}
// cnt8 <= 8 steps from operands A (alpha) and B (beta^2), 2 per double2
__device__ __forceinline__ void minors_8(const double2 (&A)[4], const double2 (&B)[4], int cnt8,
                                         double xn, double& pm, double& pc, uint32_t& sg,
                                         int& cnt) {
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    if (2 * u < cnt8) minors_step(A[u].x, B[u].x, xn, pm, pc, sg);
    if (2 * u + 1 < cnt8) minors_step(A[u].y, B[u].y, xn, pm, pc, sg);
  }
  cnt += __builtin_popcount((sg ^ (sg >> 1)) & ((1u << cnt8) - 1u));
  const int e = __builtin_amdgcn_frexp_exp(fmax(fabs(pc), fabs(pm)));
  pc = __builtin_amdgcn_ldexp(pc, -e);
  pm = __builtin_amdgcn_ldexp(pm, -e);
}
__device__ __forceinline__ void minors_load(const double2* a2, const double2* c2, int q,
                                            double2 (&A)[4], double2 (&B)[4]) {
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    A[u] = a2[4 * q + u];
    B[u] = c2[4 * q + u];
  }
}
__device__ __forceinline__ int sturm_count(const double* an, const double* b2s, int n, double xn) {
  double pm = 0.0, pc = 1.0;
  uint32_t sg = 0;   // sign bits, newest lowest; q_0 = 1 > 0
  int cnt = 0;
  const int n8 = __builtin_amdgcn_readfirstlane(n >> 3), rem = __builtin_amdgcn_readfirstlane(n & 7);
  const double2* a2 = reinterpret_cast<const double2*>(an);
  const double2* c2 = reinterpret_cast<const double2*>(b2s);
  // two operand buffers in turn: the next 8 steps' operands are read while
  // these 8 run
  double2 A0[4], B0[4], A1[4], B1[4];
  minors_load(a2, c2, 0, A0, B0);
  int q = 0;
  for (; q + 2 <= n8; q += 2) {
    minors_load(a2, c2, q + 1, A1, B1);
    minors_8(A0, B0, 8, xn, pm, pc, sg, cnt);
    minors_load(a2, c2, q + 2, A0, B0);
    minors_8(A1, B1, 8, xn, pm, pc, sg, cnt);
  }
  if (q < n8) {   // one full group left, then the remainder from the next
    minors_load(a2, c2, q + 1, A1, B1);
    minors_8(A0, B0, 8, xn, pm, pc, sg, cnt);
    minors_8(A1, B1, rem, xn, pm, pc, sg, cnt);
  } else {
    minors_8(A0, B0, rem, xn, pm, pc, sg, cnt);
  }
  return cnt;
}

#define EIG_T 256                // threads per eigenpair (vectors, orthonormalisation)
#define EIG_VT 256               // threads per eigenvalue: one multisection probe each (512 measured slower: 43 against 36 us at n = 96)

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

// The eigenvalue of ascending index kidx of the tridiagonal in LDS (al, b1;
// Gershgorin information ti) by Sturm-count multisection; every thread of the
// block calls it and gets the value.  On return an, b2s hold T / 2^esc (the
// operands of the minors recurrence, |T| / 2^esc < 1).  smask: EIG_VT / 64
// words of LDS.
__device__ double multisect(const double* al, const double* b1, int n, const TriInfo& ti, int kidx,
                            double* an, double* b2s, unsigned long long* smask, int& esc) {
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const double pivmin = DBL_MIN * fmax(1.0, ti.bmax);
  esc = (ti.tnorm > 0.0) ? __builtin_amdgcn_frexp_exp(ti.tnorm) : 0;
  for (int k = tid; k < n; k += EIG_VT) {
    an[k] = __builtin_amdgcn_ldexp(al[k], -esc);
    const double bs = (k > 0) ? __builtin_amdgcn_ldexp(b1[k - 1], -esc) : 0.0;
    b2s[k] = fmax(bs * bs, EIG_B2MIN);
  }
  __syncthreads();
  const double pad = 2.0 * DBL_EPSILON * fmax(ti.tnorm, DBL_MIN) + 2.0 * pivmin;
  double lo = ti.lo - pad, hi = ti.hi + pad;
  // multisection: count(lo) <= kidx < count(hi); EIG_VT probes per round,
  // probe p at lo + (hi - lo) (p + 1) / (EIG_VT + 1), evaluated by thread p.
  // The bracket is narrowed to 2 eps max(|theta|, |T|): the Sturm count is
  // exact only for a matrix within about eps |T| of T, so narrower brackets of
  // small eigenvalues would not make them more accurate.
  const double wstop = 2.0 * DBL_EPSILON * ti.tnorm + pivmin;
  for (int it = 0; it < 64; ++it) {
    const double wdt = hi - lo;
    if (wdt <= fmax(2.0 * DBL_EPSILON * fmax(fabs(lo), fabs(hi)) + pivmin, wstop)) break;
    const double step = wdt / (double)(EIG_VT + 1);
    const double x = lo + step * (double)(tid + 1);
    const unsigned long long m =
        __ballot(sturm_count(an, b2s, n, __builtin_amdgcn_ldexp(x, -esc)) > kidx);
    if (lane == 0) smask[wv] = m;
    __syncthreads();
    int f = EIG_VT;                                 // first probe with count > kidx
#pragma unroll
    for (int q = EIG_VT / 64 - 1; q >= 0; --q)
      if (smask[q]) f = 64 * q + __ffsll((long long)smask[q]) - 1;
    __syncthreads();
    const double nlo = (f > 0) ? lo + step * (double)f : lo;
    const double nhi = (f < EIG_VT) ? lo + step * (double)(f + 1) : hi;
    if (!(nhi - nlo < wdt)) break;   // no progress (bracket at rounding level)
    lo = nlo;
    hi = nhi;
  }
  return 0.5 * (lo + hi);
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

// The leading (fw) or trailing principal minors q_s of T - th I, s = 0 .. n - 1
// along rows i = s (fw) or i = n - 1 - s, q_(-1) = 1: q_s = A_s q_(s-1) - B_s
// q_(s-2), with the operands of the scaled matrix of multisect in step order
// (A_s = (alpha_i - th) / 2^esc; B_s = beta_(i-1)^2 / 4^esc going down, beta_i^2
// / 4^esc going up), zero past n up to a multiple of 8 and 16-byte aligned.
// One FMA per step on the dependent chain; the pair (q_s, q_(s-1)) is rescaled
// by a power of two after every 8 steps as in sturm_count.  minors_chain runs
// the chain on one lane and keeps only the pair entering each group of 8 steps
// (ck[2 g], ck[2 g + 1]); minors_group then replays group g from its pair --
// the same operations in the same order, so the same values -- into qn[i] =
// q_s and qd[i] = q_(s-1), one scale for both, so that the pivot of row i is
// qn[i] / qd[i] (times 2^esc).  The groups replay side by side, a thread each.
__device__ __forceinline__ void minors_load8(const double* A, const double* B, int s0,
                                             double2 (&a)[4], double2 (&b)[4]) {
  const double2* a2 = reinterpret_cast<const double2*>(A + s0);
  const double2* b2 = reinterpret_cast<const double2*>(B + s0);
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    a[u] = a2[u];
    b[u] = b2[u];
  }
}
__device__ __forceinline__ double minors_step(double a, double b, double& pm, double& pc) {
  const double pn = fma(a, pc, -(b * pm));
  pm = pc;
  pc = pn;
  return pn;
}
__device__ __forceinline__ void minors_chain(const double* A, const double* B, int n, double* ck) {
  n = __builtin_amdgcn_readfirstlane(n);
  double pm = 0.0, pc = 1.0;
  auto run8 = [&](int s0, const double2 (&a)[4], const double2 (&b)[4]) {
    ck[s0 / 4] = pm;
    ck[s0 / 4 + 1] = pc;
#pragma unroll
    for (int u = 0; u < 4; ++u) {        // steps past n change nothing that is kept
      minors_step(a[u].x, b[u].x, pm, pc);
      minors_step(a[u].y, b[u].y, pm, pc);
    }
    const int e = __builtin_amdgcn_frexp_exp(fmax(fabs(pc), fabs(pm)));
    pc = __builtin_amdgcn_ldexp(pc, -e);
    pm = __builtin_amdgcn_ldexp(pm, -e);
  };
  // the operands of the next 8 steps are read while these run
  double2 a0[4], b0[4], a1[4], b1[4];
  minors_load8(A, B, 0, a0, b0);
  int s0 = 0;
  for (; s0 + 8 < n; s0 += 16) {
    minors_load8(A, B, s0 + 8, a1, b1);
    run8(s0, a0, b0);
    if (s0 + 16 < n) minors_load8(A, B, s0 + 16, a0, b0);
    run8(s0 + 8, a1, b1);
  }
  if (s0 < n) run8(s0, a0, b0);
}
__device__ __forceinline__ void minors_group(const double* A, const double* B, int n, bool fw,
                                             const double* ck, int g, double* qn, double* qd) {
  double2 a[4], b[4];
  minors_load8(A, B, 8 * g, a, b);
  double pm = ck[2 * g], pc = ck[2 * g + 1];
  auto put = [&](int s, double pq, double pn) {
    if (s < n) {
      const int i = fw ? s : n - 1 - s;
      qn[i] = pn;
      qd[i] = pq;
    }
  };
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    double pq = pc;
    put(8 * g + 2 * u, pq, minors_step(a[u].x, b[u].x, pm, pc));
    pq = pc;
    put(8 * g + 2 * u + 1, pq, minors_step(a[u].y, b[u].y, pm, pc));
  }
}

// One wave: x_s = A_s x_(s-1) + B_s for s = 0 .. cnt - 1 (cnt <= 256), from
// x_(-1) = x0, as a scan of affine maps instead of cnt dependent steps: lane
// l composes the maps of its four steps 4 l .. 4 l + 3, the lanes' maps are
// combined in lane order by a Hillis-Steele scan (shuffles), and each lane then
// runs its four steps from the value its predecessors leave.  ld(s, A, B)
// gives step s's coefficients (only called for s < cnt); st(s, x) receives
// x_s.  Every lane of the wave must call it.
template <class LD, class ST>
__device__ __forceinline__ void wave_affine_scan(int cnt, double x0, LD ld, ST st) {
  const int lane = threadIdx.x & 63;
  double A[4], B[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int s2 = 4 * lane + e;
    A[e] = 1.0;
    B[e] = 0.0;
    if (s2 < cnt) ld(s2, A[e], B[e]);
  }
  double a = 1.0, b = 0.0;                       // the lane's map: x -> a x + b
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    b = fma(A[e], b, B[e]);
    a = A[e] * a;
  }
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const double pa = __shfl_up(a, off, 64), pb = __shfl_up(b, off, 64);
    if (lane >= off) {                            // this map after the earlier lanes'
      b = fma(a, pb, b);
      a = a * pa;
    }
  }
  // value entering the lane: the inclusive map of the lanes before, applied to x0
  const double qa = __shfl_up(a, 1, 64), qb = __shfl_up(b, 1, 64);
  double x = (lane == 0) ? x0 : fma(qa, x0, qb);
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int s2 = 4 * lane + e;
    if (s2 < cnt) {
      x = fma(A[e], x, B[e]);
      st(s2, x);
    }
  }
}

// Eigenvector of an isolated eigenvalue th of the unreduced tridiagonal T by
// the twisted factorisation (Parlett and Dhillon): the top-down pivots dp of
// T - th I = L D L^T and the bottom-up pivots dm of U D U^T (ratios of
// consecutive leading and trailing principal minors: the two minors
// recurrences run by lane 0 of waves 0 and 1 side by side, their groups of 8
// steps replayed and the divisions made by every thread; each pivot below pivmin in magnitude replaced by
// -pivmin), the twist gamma_k = dp_k + dm_k - (alpha_k - th), k the index of
// the smallest |gamma_k| (the first of equals), and z with z_k = 1 solving
// N_k^T z = e_k:
// z_i = -(beta_i / dp_i) z_(i+1) below k, z_i = -(beta_(i-1) / dm_i) z_(i-1)
// above (the two lanes again).  Then (T - th I) z = gamma_k e_k in exact
// arithmetic, and one inverse-iteration step with the same factors,
// x = (T - th I)^-1 z, squares the error the first solve leaves (a vector
// from one solve is orthogonal to a neighbour's only to about eps |T| / gap).
// Accepted (true, x / |x|_inf in y) when every entry is finite and
// |(T - th I) x|_inf <= 64 eps |T| |x|_inf, the level inverse iteration
// reaches; every thread of the block must call it (it contains barriers).
// dp, dm, ratios and scratch use the caller's LDS arrays; an, b2s and esc are
// the scaled operands multisect leaves.
__device__ __forceinline__ bool twisted_vector(const double* al, const double* b1, const double* b2,
                                            const double* an, const double* b2s, int esc,
                                            int n, double th, double tnorm, double pivmin,
                                            double* dp, double* dm, double* rat, double* sc,
                                            double* tw, double* y) {
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  __shared__ int kst;
  __shared__ double mred[2][EIG_T / 64];
  __shared__ double qm[4][EIG_NMAX];              // leading minors (qn, qd), then trailing
  __shared__ __align__(16) double mop[4][EIG_NMAX + 8];   // A, B going down, then going up
  __shared__ double ck[2][EIG_NMAX / 4];          // the pairs entering each group of 8 steps
  const double thn = __builtin_amdgcn_ldexp(th, -esc);
  const int ng = (n + 7) >> 3;                    // groups of 8 steps per direction
  for (int s = tid; s < 8 * ng; s += EIG_T) {
    const bool in = s < n;
    mop[0][s] = in ? an[s] - thn : 0.0;
    mop[1][s] = in ? b2s[s] : 0.0;
    mop[2][s] = in ? an[n - 1 - s] - thn : 0.0;
    mop[3][s] = in ? b2s[min(n - s, n - 1)] : 0.0;
  }
  __syncthreads();
  if (tid == 0 || tid == 64) {
    // wave-uniform in the one active lane, so indices and branches stay scalar
    const int h = __builtin_amdgcn_readfirstlane(tid) == 0 ? 0 : 2;
    minors_chain(mop[h], mop[h + 1], n, ck[h / 2]);
  }
  __syncthreads();
  if (tid < 2 * ng) {
    const bool fw = tid < ng;
    const int h = fw ? 0 : 2;
    minors_group(mop[h], mop[h + 1], n, fw, ck[h / 2], fw ? tid : tid - ng, qm[h], qm[h + 1]);
  }
  __syncthreads();
  // The pivots, dp_i = q_i / q_(i-1) of the leading minors and dm_i of the
  // trailing ones; a pivot below pivmin in magnitude (or no number: a zero
  // minor before it) becomes -pivmin, and the pivot after a replaced one is
  // formed from the replacement, (alpha - th) - beta^2 / (-pivmin), as the
  // pivot recurrence d_i = (alpha_i - th) - beta^2 / d_(i-1) does.  Then
  // |gamma_k| into sc and the ratios rat[i] = beta_i / dp_i (i < n - 1) and
  // y[i] = beta_(i-1) / dm_i (i > 0).
  auto small = [&](double d) { return !(fabs(d) >= pivmin); };
  auto ratio = [&](int h, int k) { return __builtin_amdgcn_ldexp(qm[h][k] / qm[h + 1][k], esc); };
  for (int i = tid; i < n; i += EIG_T) {
    const double am = al[i] - th;
    double p = (i > 0 && small(ratio(0, i - 1))) ? am + b2[i - 1] / pivmin : ratio(0, i);
    double q = (i < n - 1 && small(ratio(2, i + 1))) ? am + b2[i] / pivmin : ratio(2, i);
    if (small(p)) p = -pivmin;
    if (small(q)) q = -pivmin;
    dp[i] = p;
    dm[i] = q;
    sc[i] = fabs(p + q - am);
    rat[i] = (i < n - 1) ? b1[i] / p : 0.0;
    y[i] = (i > 0) ? b1[i - 1] / q : 0.0;
  }
  __syncthreads();
  if (wv == 0) {
    // smallest |gamma| and its first index: lane scan, then lanes by pairs
    double gm = DBL_MAX;
    int gk = n;
    for (int i = lane; i < n; i += 64)
      if (sc[i] < gm) {
        gm = sc[i];
        gk = i;
      }
    for (int o = 32; o >= 1; o >>= 1) {
      const double og = __shfl_xor(gm, o, 64);
      const int ok = __shfl_xor(gk, o, 64);
      if (og < gm || (og == gm && ok < gk)) {
        gm = og;
        gk = ok;
      }
    }
    if (lane == 0) kst = gk;
  }
  __syncthreads();
  const int k = __builtin_amdgcn_readfirstlane(kst);
  // z into sc: wave 0 goes down from k, wave 1 up (z_i = -rat_i z_(i+1) and
  // z_i = -y_i z_(i-1), products as affine scans)
  if (wv < 2) {
    const bool dn = wv == 0;
    if (dn && lane == 0) sc[k] = 1.0;
    wave_affine_scan(dn ? k : n - 1 - k, 1.0,
                     [&](int s2, double& A, double& Bc) {
                       A = dn ? -rat[k - 1 - s2] : -y[k + 1 + s2];
                       Bc = 0.0;
                     },
                     [&](int s2, double x) { sc[dn ? k - 1 - s2 : k + 1 + s2] = x; });
  }
  __syncthreads();
  // One inverse-iteration step with the same factors, x = (T - th I)^-1 z,
  // T - th I = N_k D_k N_k^T (N_k unit, l_i = rat[i] below the diagonal above
  // row k, u_i = y[i + 1] above it below row k; D_k = dp above k, gamma_k at
  // k, dm below): N_k t = z from either end towards k (the two lanes), then
  // t_k and t / D_k, then N_k^T x = t outwards from k.  Skipped when gamma_k
  // is below pivmin (z is then exact to working precision).
  const double gk = dp[k] + dm[k] - (al[k] - th);
  const bool refine = fabs(gk) >= pivmin;         // the same in every thread
  if (refine && wv < 2) {
    const bool dn = wv == 0;                      // wave 0: rows 0 .. k - 1, wave 1: n - 1 .. k + 1
    wave_affine_scan(dn ? k : n - 1 - k, 0.0,
                     [&](int s2, double& A, double& Bc) {
                       const int i = dn ? s2 : n - 1 - s2;
                       A = dn ? (i > 0 ? -rat[i - 1] : 0.0) : (i < n - 1 ? -y[i + 1] : 0.0);
                       Bc = sc[i];
                     },
                     [&](int s2, double x) { tw[dn ? s2 : n - 1 - s2] = x; });
  }
  __syncthreads();
  for (int i = tid; i < n && refine; i += EIG_T) {
    double t = tw[i], d;
    if (i < k) {
      d = dp[i];
    } else if (i > k) {
      d = dm[i];
    } else {
      t = sc[k];
      if (k > 0) t = fma(-rat[k - 1], tw[k - 1], t);
      if (k < n - 1) t = fma(-y[k + 1], tw[k + 1], t);
      d = gk;
    }
    dp[i] = t / d;                              // each thread rewrites only its own dp[i]
  }
  __syncthreads();
  if (refine && wv < 2) {
    const bool dn = wv == 0;
    const double xk = dp[k];
    if (dn && lane == 0) sc[k] = xk;
    wave_affine_scan(dn ? k : n - 1 - k, xk,
                     [&](int s2, double& A, double& Bc) {
                       const int i = dn ? k - 1 - s2 : k + 1 + s2;
                       A = dn ? -rat[i] : -y[i];
                       Bc = dp[i];
                     },
                     [&](int s2, double x) { sc[dn ? k - 1 - s2 : k + 1 + s2] = x; });
  }
  __syncthreads();
  // residual and size (block maxima), finiteness
  double rmax = 0.0, zmax = 0.0;
  bool fin = true;
  for (int i = tid; i < n; i += EIG_T) {
    const double zi = sc[i];
    double ri = (al[i] - th) * zi;
    if (i > 0) ri = fma(b1[i - 1], sc[i - 1], ri);
    if (i < n - 1) ri = fma(b1[i], sc[i + 1], ri);
    fin = fin && isfinite(zi) && isfinite(ri);
    rmax = fmax(rmax, fabs(ri));
    zmax = fmax(zmax, fabs(zi));
  }
  for (int o = 32; o >= 1; o >>= 1) {
    rmax = fmax(rmax, __shfl_xor(rmax, o, 64));
    zmax = fmax(zmax, __shfl_xor(zmax, o, 64));
  }
  const bool allfin = __syncthreads_and(fin);
  if (lane == 0) {
    mred[0][wv] = rmax;
    mred[1][wv] = zmax;
  }
  __syncthreads();
  rmax = 0.0;
  zmax = 0.0;
  for (int q = 0; q < EIG_T / 64; ++q) {
    rmax = fmax(rmax, mred[0][q]);
    zmax = fmax(zmax, mred[1][q]);
  }
  const bool ok = allfin && zmax > 0.0 && rmax <= 64.0 * DBL_EPSILON * tnorm * zmax;
  if (ok) {
    for (int i = tid; i < n; i += EIG_T) y[i] = sc[i] / zmax;
  }
  __syncthreads();
  return ok;
}

// Seig: [n_act][n_it][r] (row k, kept column c); rows n_eff.. are zero.
// theta: [n_act][r], ascending kept eigenvalues (zero for the r - r_eff
// leading columns of a window that stopped after n_eff < r steps); Seig
// [n_act][n_it][r] their vectors.  Block (c, a): kept eigenpair c of window a,
// its eigenvalue by multisection, then its vector.
__global__ __launch_bounds__(EIG_T) void k_eig_pairs(const double* __restrict__ alpha,
                                                     const double* __restrict__ beta,
                                                     const int* __restrict__ neff, int n_it,
                                                     int r, double* __restrict__ theta,
                                                     double* __restrict__ Seig) {
  const int c = blockIdx.x, a = blockIdx.y, tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int n = neff[a];
  const int r_eff = min(r, n);
  double* Sa = Seig + (int64_t)a * n_it * r;
  if (c < r - r_eff) {
    if (tid == 0) theta[(int64_t)a * r + c] = 0.0;
    for (int k = tid; k < n_it; k += EIG_T) Sa[(int64_t)k * r + c] = 0.0;
    return;
  }
  __shared__ double al[EIG_NMAX], b1[EIG_NMAX], b2[EIG_NMAX];
  __shared__ double y[EIG_NMAX], w[EIG_NMAX];
  __shared__ double fu1[EIG_NMAX], fu2[EIG_NMAX], fd[EIG_NMAX], fl[EIG_NMAX];
  __shared__ int piv[EIG_NMAX];
  __shared__ __align__(16) double an[EIG_NMAX + 8], b2s[EIG_NMAX + 8];
  __shared__ unsigned long long smask[EIG_VT / 64];
  __shared__ int cnt2[2];
  const TriInfo ti = load_tridiag(alpha + (int64_t)a * n_it, beta + (int64_t)a * n_it, n, al, b1, b2);
  int esc = 0;
  const double th = multisect(al, b1, n, ti, n - r + c, an, b2s, smask, esc);
  if (tid == 0) theta[(int64_t)a * r + c] = th;
  // An eigenvalue alone in [th - EIG_TWIST_GAP |T|, th + EIG_TWIST_GAP |T|)
  // (two Sturm counts) takes the twisted factorisation (its vector is then
  // accurate to about eps |T| / gap, and the clusters of kept eigenvalues are
  // orthonormalised later); if that fails its residual test, and for
  // (numerically) repeated eigenvalues, inverse iteration below.
  {
    const double ctol = EIG_TWIST_GAP * ti.tnorm;
    if (tid < 2)
      cnt2[tid] = sturm_count(an, b2s, n, __builtin_amdgcn_ldexp(tid ? th + ctol : th - ctol, -esc));
    __syncthreads();
    if (cnt2[1] - cnt2[0] == 1 &&
        twisted_vector(al, b1, b2, an, b2s, esc, n, th, ti.tnorm, DBL_MIN * fmax(1.0, ti.bmax), fd, fl, fu1,
                       fu2, w, y)) {
      if (wv == 0) store_unit_column(y, n, n_it, r, c, Sa);
      return;
    }
  }
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
// then unit norm and the sign rule again.  The clusters are independent: wave
// w of the workgroup takes clusters w, w + 4, ..., staging a cluster's columns
// in its own LDS slice when they fit (else reading them from Seig), with wave
// sums for the dot products and no workgroup barriers.  Windows without
// clusters only read theta and T.
constexpr int EIG_ORTH_LDS = 3072;             // doubles of LDS per wave
__global__ __launch_bounds__(EIG_T) void k_eig_orth(const double* __restrict__ alpha,
                                                    const double* __restrict__ beta,
                                                    const int* __restrict__ neff, int n_it, int r,
                                                    const double* __restrict__ theta,
                                                    double* __restrict__ Seig) {
  const int a = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int n = neff[a];
  const int c_lo = r - min(r, n);
  double* Sa = Seig + (int64_t)a * n_it * r;
  __shared__ double al[EIG_NMAX], b1[EIG_NMAX], b2[EIG_NMAX];
  __shared__ double tha[EIG_NMAX];
  __shared__ int cstart[EIG_NMAX], ncl;
  __shared__ double cb[EIG_T / 64][EIG_ORTH_LDS];
  for (int c = tid; c < r; c += EIG_T) tha[c] = theta[(int64_t)a * r + c];
  const TriInfo ti = load_tridiag(alpha + (int64_t)a * n_it, beta + (int64_t)a * n_it, n, al, b1, b2);
  const double ctol = EIG_CLUSTER * ti.tnorm;
  // clusters of two or more kept columns, as start indices (cstart[q], end
  // before the next start), found by one thread
  if (tid == 0) {
    int q = 0;
    for (int c = c_lo; c < r;) {
      int c1 = c;
      while (c1 + 1 < r && tha[c1 + 1] - tha[c1] <= ctol) ++c1;
      if (c1 > c) {
        cstart[2 * q] = c;
        cstart[2 * q + 1] = c1;
        ++q;
      }
      c = c1 + 1;
    }
    ncl = q;
  }
  __syncthreads();
  double* wb = cb[wv];
  for (int q = wv; q < ncl; q += EIG_T / 64) {
    const int c = cstart[2 * q], c1 = cstart[2 * q + 1], s = c1 - c + 1;
    const bool staged = s * n <= EIG_ORTH_LDS;
    // column p of the cluster (p < s): LDS slice or Seig
    auto colp = [&](int p, int i) -> double {
      return staged ? wb[p * n + i] : Sa[(int64_t)i * r + c + p];
    };
    if (staged) {
      for (int p = 0; p < s; ++p)
        for (int i = lane; i < n; i += 64) wb[p * n + i] = Sa[(int64_t)i * r + c + p];
    }
    for (int k = 1; k < s; ++k) {
      double y[EIG_NMAX / 64];
#pragma unroll
      for (int t = 0; t < EIG_NMAX / 64; ++t) {
        const int i = lane + 64 * t;
        y[t] = (i < n) ? colp(k, i) : 0.0;
      }
      for (int pass = 0; pass < 2; ++pass) {
        for (int p = 0; p < k; ++p) {
          double d = 0.0;
#pragma unroll
          for (int t = 0; t < EIG_NMAX / 64; ++t) {
            const int i = lane + 64 * t;
            if (i < n) d = fma(y[t], colp(p, i), d);
          }
          d = wave_sum_f64(d);
#pragma unroll
          for (int t = 0; t < EIG_NMAX / 64; ++t) {
            const int i = lane + 64 * t;
            if (i < n) y[t] = fma(-d, colp(p, i), y[t]);
          }
        }
      }
      // unit norm and the sign rule (first nonzero entry positive), into the
      // slice (for the later members) and Seig
      double nr = 0.0;
      int first = n - 1;
#pragma unroll
      for (int t = 0; t < EIG_NMAX / 64; ++t) {
        const int i = lane + 64 * t;
        if (i < n) {
          nr = fma(y[t], y[t], nr);
          if (y[t] != 0.0 && i < first) first = i;
        }
      }
      nr = wave_sum_f64(nr);
      for (int o = 32; o >= 1; o >>= 1) first = min(first, __shfl_xor(first, o, 64));
      double yo = 0.0;                           // this lane's entry of slot first >> 6
#pragma unroll
      for (int t = 0; t < EIG_NMAX / 64; ++t) yo = (t == (first >> 6)) ? y[t] : yo;
      const double yf = __shfl(yo, first & 63, 64);
      double sc = 1.0 / sqrt(nr);
      if (yf < 0.0) sc = -sc;
#pragma unroll
      for (int t = 0; t < EIG_NMAX / 64; ++t) {
        const int i = lane + 64 * t;
        if (i < n) {
          const double v = y[t] * sc;
          if (staged) wb[k * n + i] = v;
          Sa[(int64_t)i * r + c + k] = v;
        }
      }
    }
  }
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

static hipError_t launch_ritz(const double* Q, const double* Seig, const int* neff, int n_act, int L,
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

// The cluster orthonormalisation of k_eig_orth and the Ritz coordinates of
// k_ritz in one kernel, when S (n_it x r) and a block's Q rows (n_it x 32) fit
// in LDS together: every block stages all of S and its 32 rows of Q with one
// round of loads, repeats the (small, deterministic) orthonormalisation of the
// clustered columns on its copy of S -- the same arithmetic as k_eig_orth, so
// every block holds the same S -- and forms its rows of Z.  The clusters of a
// window are found in parallel (a cluster of two or more kept columns starts
// where the gap below is above EIG_CLUSTER |T| and the gap above is not) and
// shared out to the waves, which need no barriers between them.
constexpr int RZ_LDS = 16384;                  // doubles of dynamic LDS (128 KiB)
constexpr int RZ_NMAX = 128;                   // largest n_it of the fused path
__global__ __launch_bounds__(256) void k_ritz_orth(const double* __restrict__ Q,
                                                   const double* __restrict__ Seig,
                                                   const int* __restrict__ neff,
                                                   const double* __restrict__ alpha,
                                                   const double* __restrict__ beta,
                                                   const double* __restrict__ theta, int L,
                                                   int ldq, int n_it, int r,
                                                   double* __restrict__ Z) {
  extern __shared__ double rzs[];
  // S row-major with a padded row stride rs = r + 1, so that a column (the
  // Gram-Schmidt reads) spreads over the LDS banks
  const int rs = r + 1;
  const int n4r = (n_it + 3) & ~3;               // rows allocated (k steps of 4)
  double* sS = rzs;                              // [k][c], k < n (rows n .. n4 - 1 zero)
  double* sQ = rzs + n4r * rs;                   // [k][32]
  __shared__ double tha[EIG_NMAX], mred[4];
  __shared__ int cst[EIG_NMAX], ncl;
  const int a = blockIdx.y, tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int n = neff[a];
  const int ntile = (L + 31) / 32;
  const int r0 = blockIdx.x * 32;                // first tile; then every gridDim.x-th
  const int c_lo = r - min(r, n);
  const double* Sa = Seig + (int64_t)a * n_it * r;
  const double* Qa = Q + (int64_t)a * ldq * L;
  const double* al = alpha + (int64_t)a * n_it;
  const double* be = beta + (int64_t)a * n_it;
  if (tid == 0) ncl = 0;
  // one round of loads: S, the block's Q rows, theta and the Gershgorin terms
  {
    const int ns = n * r, nq = n * 32;
    for (int e0 = tid; e0 < ns + nq; e0 += 256 * 24) {
      double v[24];
#pragma unroll
      for (int u = 0; u < 24; ++u) {
        const int e = min(e0 + 256 * u, ns + nq - 1);
        v[u] = (e < ns) ? Sa[e] : Qa[(int64_t)((e - ns) >> 5) * L + min(r0 + ((e - ns) & 31), L - 1)];
      }
#pragma unroll
      for (int u = 0; u < 24; ++u) {
        const int e = e0 + 256 * u;
        if (e < ns) sS[(e / r) * rs + e % r] = v[u];
        else if (e < ns + nq) sQ[e - ns] = v[u];
      }
    }
    // rows n .. n4 - 1 of S and Q zero (the last step of 4 of the products)
    const int n4 = (n + 3) & ~3;
    for (int e = tid; e < (n4 - n) * rs; e += 256) sS[n * rs + e] = 0.0;
    for (int e = tid; e < (n4 - n) * 32; e += 256) sQ[n * 32 + e] = 0.0;
  }
  for (int c = tid; c < r; c += 256) tha[c] = theta[(int64_t)a * r + c];
  double tn = 0.0;
  for (int k = tid; k < n; k += 256) {
    const double off = ((k < n - 1) ? fabs(be[k]) : 0.0) + ((k > 0) ? fabs(be[k - 1]) : 0.0);
    tn = fmax(tn, fabs(al[k]) + off);
  }
  for (int o = 32; o >= 1; o >>= 1) tn = fmax(tn, __shfl_xor(tn, o, 64));
  if (lane == 0) mred[wv] = tn;
  __syncthreads();
  const double ctol = EIG_CLUSTER * fmax(fmax(mred[0], mred[1]), fmax(mred[2], mred[3]));
  for (int c = c_lo + tid; c < r; c += 256) {
    const bool start = c == c_lo || tha[c] - tha[c - 1] > ctol;
    if (start && c + 1 < r && tha[c + 1] - tha[c] <= ctol) {
      int c1 = c + 1;
      while (c1 + 1 < r && tha[c1 + 1] - tha[c1] <= ctol) ++c1;
      const int q = atomicAdd(&ncl, 1);
      cst[2 * q] = c;
      cst[2 * q + 1] = c1;
    }
  }
  __syncthreads();
  for (int q = wv; q < ncl; q += 4) {
    const int c = cst[2 * q], c1 = cst[2 * q + 1];
    for (int k = c + 1; k <= c1; ++k) {
      double y[EIG_NMAX / 64];
#pragma unroll
      for (int t = 0; t < EIG_NMAX / 64; ++t) {
        const int i = lane + 64 * t;
        y[t] = (i < n) ? sS[i * rs + k] : 0.0;
      }
      for (int pass = 0; pass < 2; ++pass) {
        for (int p = c; p < k; ++p) {
          double d = 0.0;
#pragma unroll
          for (int t = 0; t < EIG_NMAX / 64; ++t) {
            const int i = lane + 64 * t;
            if (i < n) d = fma(y[t], sS[i * rs + p], d);
          }
          d = wave_sum_f64(d);
#pragma unroll
          for (int t = 0; t < EIG_NMAX / 64; ++t) {
            const int i = lane + 64 * t;
            if (i < n) y[t] = fma(-d, sS[i * rs + p], y[t]);
          }
        }
      }
      double nr = 0.0;
      int first = n - 1;
#pragma unroll
      for (int t = 0; t < EIG_NMAX / 64; ++t) {
        const int i = lane + 64 * t;
        if (i < n) {
          nr = fma(y[t], y[t], nr);
          if (y[t] != 0.0 && i < first) first = i;
        }
      }
      nr = wave_sum_f64(nr);
      for (int o = 32; o >= 1; o >>= 1) first = min(first, __shfl_xor(first, o, 64));
      double yo = 0.0;
#pragma unroll
      for (int t = 0; t < EIG_NMAX / 64; ++t) yo = (t == (first >> 6)) ? y[t] : yo;
      const double yf = __shfl(yo, first & 63, 64);
      double sc = 1.0 / sqrt(nr);
      if (yf < 0.0) sc = -sc;
#pragma unroll
      for (int t = 0; t < EIG_NMAX / 64; ++t) {
        const int i = lane + 64 * t;
        if (i < n) sS[i * rs + k] = y[t] * sc;
      }
    }
  }
  __syncthreads();
  // Z rows, 32 per tile, on the fp64 matrix cores: Z_tile = Q_tile^T S as
  // 16 x 16 blocks (v_mfma_f64_16x16x4f64: lane l holds A[l % 16][l / 16] and
  // B[l / 16][l % 16] of a 16 x 4 by 4 x 16 step, and D[l / 16 + 4 v][l % 16],
  // v < 4); wave w takes the column blocks w, w + 4, ... of both row halves.
  // The block's later tiles (every gridDim.x-th) have their Q rows fetched
  // into registers while the current tile is multiplied.
  typedef double f64x4 __attribute__((ext_vector_type(4)));
  const int n4 = (n + 3) & ~3, nct = (r + 15) / 16;
  const int li = lane & 15, lk = lane >> 4;
  constexpr int QPT = RZ_NMAX * 32 / 256;         // Q values per thread and tile, at most
  double qn[QPT];
  auto fetch_q = [&](int t0) {
#pragma unroll
    for (int u = 0; u < QPT; ++u) {
      const int e = tid + 256 * u;
      if (e < n * 32) qn[u] = Qa[(int64_t)(e >> 5) * L + min(t0 * 32 + (e & 31), L - 1)];
    }
  };
  int tile = blockIdx.x;
  if (tile + (int)gridDim.x < ntile) fetch_q(tile + gridDim.x);
  for (;;) {
    for (int ct = wv; ct < nct; ct += 4) {
      const int jb = ct * 16 + li, jc = min(jb, r - 1);
      f64x4 acc0 = {0.0, 0.0, 0.0, 0.0}, acc1 = {0.0, 0.0, 0.0, 0.0};
#pragma unroll 2
      for (int k0 = 0; k0 < n4; k0 += 4) {
        const int kk = k0 + lk;
        const double b = sS[kk * rs + jc];
        const double a0 = sQ[kk * 32 + li], a1 = sQ[kk * 32 + 16 + li];
        acc0 = __builtin_amdgcn_mfma_f64_16x16x4f64(a0, b, acc0, 0, 0, 0);
        acc1 = __builtin_amdgcn_mfma_f64_16x16x4f64(a1, b, acc1, 0, 0, 0);
      }
      if (jb < r) {
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int i0 = tile * 32 + lk + 4 * v, i1 = i0 + 16;
          if (i0 < L) Z[((int64_t)a * L + i0) * r + jb] = acc0[v];
          if (i1 < L) Z[((int64_t)a * L + i1) * r + jb] = acc1[v];
        }
      }
    }
    tile += gridDim.x;
    if (tile >= ntile) break;
    __syncthreads();                              // sQ of the last tile read by all
#pragma unroll
    for (int u = 0; u < QPT; ++u) {
      const int e = tid + 256 * u;
      if (e < n * 32) sQ[e] = qn[u];
    }
    __syncthreads();
    if (tile + (int)gridDim.x < ntile) fetch_q(tile + gridDim.x);
  }
}

static hipError_t launch_ritz_orth(const double* Q, const double* Seig, const int* neff,
                                     const double* alpha, const double* beta,
                                     const double* theta, int n_act, int L, int ldq, int n_it,
                                     int r, double* Z, int n_cu, hipStream_t s) {
  const size_t lds = (size_t)((n_it + 3) & ~3) * (r + 33) * sizeof(double);
  auto k = k_ritz_orth;
  if (lds > 65536) {
    const hipError_t e = hipFuncSetAttribute((const void*)k, hipFuncAttributeMaxDynamicSharedMemorySize,
                                             (int)lds);
    if (e != hipSuccess) return e;
  }
  // one round of resident blocks (as many per CU as their LDS allows, 160 KiB
  // per CU): one tile per block while the tiles fit, else each block loops
  // over tiles (S staged and orthonormalised once per block)
  const int64_t ntile = (L + 31) / 32;
  const int64_t bpc = std::max<int64_t>(1, 163840 / (int64_t)(lds + 4096));
  const int64_t per_win = std::max<int64_t>(1, bpc * std::max(1, n_cu) / std::max(1, n_act));
  const unsigned bx = (unsigned)std::min<int64_t>(ntile, per_win);
  hipLaunchKernelGGL(k, dim3(bx, n_act), dim3(256), lds, s, Q, Seig, neff, alpha, beta, theta, L,
                     ldq, n_it, r, Z);
  return hipSuccess;
}

hipError_t launch_eigh_ritz(const double* alpha, const double* beta, const int* neff, int n_act,
                            int n_it, int r, double* theta, double* Seig, const double* Q, int L,
                            int ldq, double* Z, int n_cu, hipStream_t s) {
  (void)hipGetLastError();
  if (n_it > EIG_NMAX || r > n_it || r > 128 || r < 1) return hipErrorInvalidValue;
  static_assert(EIG_VT == EIG_T, "one block size for the pairs");
  hipLaunchKernelGGL(k_eig_pairs, dim3(r, n_act), dim3(EIG_T), 0, s, alpha, beta, neff, n_it, r,
                     theta, Seig);
  if ((int64_t)((n_it + 3) & ~3) * (r + 33) <= RZ_LDS && n_it <= RZ_NMAX) {
    const hipError_t e = launch_ritz_orth(Q, Seig, neff, alpha, beta, theta, n_act, L, ldq, n_it, r,
                                          Z, n_cu, s);
    if (e != hipSuccess) return e;
    return hipGetLastError();
  }
  hipLaunchKernelGGL(k_eig_orth, dim3(n_act), dim3(EIG_T), 0, s, alpha, beta, neff, n_it, r, theta,
                     Seig);
  return launch_ritz(Q, Seig, neff, n_act, L, ldq, n_it, r, Z, s);
}

}  // namespace slh
