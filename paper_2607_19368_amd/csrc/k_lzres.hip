// Implicit Lanczos with full re-orthogonalization (Algorithm 2; operator of
// Eq. 4, A v = Phi (Phi^T v)) for one window whose Phi fits in the register
// files of the device, as one persistent kernel for the whole run.
//
// Block b of nb (one per compute unit) holds rows [RB b, RB b + RB) of Phi in
// registers for the whole run, loaded once, and its rows of the basis Q in
// LDS.  Each step is the same computation as the pass and the reduction of
// the streaming path (k_lz_step, k_lz_reduce: q_j by the second Gram-Schmidt
// pass of step j-1 in row space, u = A q_j from the row dots with t~ and the
// Lanczos relation, z1 by the three-term recurrence, then t~ = Phi^T z1 / |z1|
// and h2 = Q_j^T z1), in two phases:
//   rows     every block: its rows of q_j and z1, and its partials of Phi^T z1,
//            of h2 and of |z1|^2 (alpha~ = |t~|^2 it sums from the t~ it holds);
//   columns  block b: t~ over its m / nb columns (written to every copy of t~);
//            h2 entries b, b + nb, ...; |z1|^2 (every block).
// The scalars of a step (alpha, beta, the breakdown test) are computed by
// every block from the same reduced values in the same order, so all blocks
// agree and leave the loop together.  Results are bitwise reproducible.
//
// The blocks synchronise only through the data they exchange, with no
// barrier: every value passed between blocks is written with an agent-scope
// atomic store (coherent across the device's L2 caches) carrying its step in
// its two lowest mantissa bits (1 + (step & 1); a perturbation of at most
// 3 ulp, the same for every reader), and a reader polls each value it needs
// until the tag is that of the step it waits for.  The buffers are zeroed
// (tag 0, never valid) before the launch; every slot in use is rewritten at
// every step, and no block can rewrite a slot of step e + 1 before every
// reader has consumed step e's value (it first needs values that those
// readers produce after reading), so the two tags suffice.  Every wait is
// bounded: after LR_SPIN polls (or w.spin) a block sets an error word and leaves, and the
// others, seeing it, leave too.  A block's own stores are acknowledged
// before its waves start polling: its polls and its stores share the CU's path
// to memory, and its stores are what the other blocks are waiting for.  The
// host launches the kernel only when all nb blocks are resident at once (one
// per compute unit; checked with the occupancy calculator).
#include "slh_device.h"
#include "slh_internal.h"

namespace slh {

namespace {

constexpr int LR_T = 256;          // threads per block at m = 1024 (one wave per SIMD); 512 at m = 2048
constexpr int LR_SPIN = 1 << 20;   // polls before a barrier gives up

__device__ __forceinline__ void st_flag(unsigned* p, unsigned v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ unsigned ld_flag(unsigned* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// bar: [LR_ERR] error word
constexpr int LR_ERR = LZ_BAR_ERR;
// copies of t~ (T holds [ldq][m] doubles)
__host__ __device__ constexpr int res_copies(int ldq) { return ldq < 8 ? ldq : 8; }

// v tagged with step e into *p
__device__ __forceinline__ void st_tag(double* p, double v, int e) {
  const long long x = (__double_as_longlong(v) & ~3LL) | (long long)(1 + (e & 1));
  __hip_atomic_store((long long*)p, x, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// two tagged values into p[0..1] (16-byte aligned) with one coherent 16-byte
// store; each half carries its own tag, so the store need not be atomic as a whole
__device__ __forceinline__ void st_tag2(double* p, double v0, double v1, int e) {
  typedef long long ll2 __attribute__((ext_vector_type(2)));
  ll2 x;
  x.x = (__double_as_longlong(v0) & ~3LL) | (long long)(1 + (e & 1));
  x.y = (__double_as_longlong(v1) & ~3LL) | (long long)(1 + (e & 1));
  // s_nop: a VALU write to the data registers of a store wider than 8 bytes
  // must not follow it directly (the compiler adds this wait state only to
  // stores of its own)
  asm volatile("global_store_dwordx4 %0, %1, off sc1\n\ts_nop 1" : : "v"(p), "v"(x) : "memory");
}
__device__ __forceinline__ long long ld_raw(double* p) {
  return __hip_atomic_load((long long*)p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ bool tag_is(long long x, int e) { return (int)(x & 3) == 1 + (e & 1); }

// v[u] = *addr(u) of step e for the u with bit u of act set (0 for the others),
// polling until every tag matches; false after spin polls or when the error
// word is set (the error word is then set)
template <int N, class ADDR>
__device__ __forceinline__ bool ld_wait(ADDR addr, unsigned act, int e, unsigned* bar, int spin,
                                        double (&v)[N]) {
  long long x[N];
#pragma unroll
  for (int u = 0; u < N; ++u) x[u] = ((act >> u) & 1) ? ld_raw(addr(u)) : 0;
  bool ok = true;
  for (int s = 0;; ++s) {
    bool all = true;
#pragma unroll
    for (int u = 0; u < N; ++u) all = all && (((act >> u) & 1) == 0 || tag_is(x[u], e));
    if (all) break;
    if (s > spin || ((s & 63) == 63 && ld_flag(bar + LR_ERR) != 0)) {
      st_flag(bar + LR_ERR, 1u);
      ok = false;
      break;
    }
#pragma unroll
    for (int u = 0; u < N; ++u)
      if (((act >> u) & 1) && !tag_is(x[u], e)) x[u] = ld_raw(addr(u));
  }
#pragma unroll
  for (int u = 0; u < N; ++u) v[u] = ((act >> u) & 1) ? __longlong_as_double(x[u]) : 0.0;
  return ok;
}

// Every store this thread issued acknowledged (vmcnt counts stores as well as
// loads here), then a block barrier: the block's polls that follow do not
// compete in the CU's memory path with its own stores, which other blocks are
// waiting for.
__device__ __forceinline__ void stores_done_barrier() {
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
}

// true in every thread when no thread of the block saw a failure (a barrier)
__device__ __forceinline__ bool block_ok(bool ok) {
  __shared__ int bad;
  if (threadIdx.x == 0) bad = 0;
  __syncthreads();
  if (!ok) bad = 1;
  __syncthreads();
  return bad == 0;
}

// The float4 of one Phi row as an opaque value at its point of use, so that its
// conversion to fp64 is not hoisted (the converted rows would need twice the
// registers).
__device__ __forceinline__ float4 pin4(float4 x) {
  asm volatile("" : "+v"(x.x), "+v"(x.y), "+v"(x.z), "+v"(x.w));
  return x;
}

// three block sums at once (fixed order: wave sums, then the NW waves in order)
template <int NW>
__device__ __forceinline__ void block_sum3(double& a, double& b, double& c, double (*red)[NW]) {
  a = wave_sum_f64(a);
  b = wave_sum_f64(b);
  c = wave_sum_f64(c);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) {
    red[0][threadIdx.x >> 6] = a;
    red[1][threadIdx.x >> 6] = b;
    red[2][threadIdx.x >> 6] = c;
  }
  __syncthreads();
  a = red[0][0];
  b = red[1][0];
  c = red[2][0];
#pragma unroll
  for (int w = 1; w < NW; ++w) {
    a += red[0][w];
    b += red[1][w];
    c += red[2][w];
  }
}

// The held rows of Phi marked as rewritten (an empty statement, in place), so
// that their fp64 conversions are neither hoisted out of the step loop nor
// shared between a step's two uses (converted once they would need twice the
// registers).  In place: the registers must all be VGPRs, or each one held in
// an accumulation register is moved out and back.
template <int RB, int NH>
__device__ __forceinline__ void launder_rows(float4 (&ph)[RB][NH]) {
#pragma unroll
  for (int r = 0; r < RB; ++r)
#pragma unroll
    for (int h = 0; h < NH; ++h)
      asm volatile("" : "+v"(ph[r][h].x), "+v"(ph[r][h].y), "+v"(ph[r][h].z), "+v"(ph[r][h].w));
}

}  // namespace

// RB rows per block; CPL = m / NT columns per lane (the lane's columns are
// 64 CPL w + 256 h + 4 lane + e for wave w, h < CPL / 4, e < 4).
// Workspace use: Spart [m / CB][nb][CB] (CB = m / nb), H2part [nb][ldq + 1], H2 [ldq + 1],
// T [C][m] with C = res_copies(ldq) (t~ written to every copy, block b reading
// copy b mod C, so that the blocks' polls of t~ spread over C times as many
// lines); outputs alpha, beta, neff, stop and Q[1..] as the streaming path.
// A block waits for its own stores before it starts polling (stores_done_barrier).
// Dynamic LDS: the block's rows of Q, (n_it + 1) (RB + 1) doubles.
// NT threads per block (NW = NT / 64 waves); INPLACE: the held rows fit in
// VGPRs (two waves per SIMD: 128 floats a lane) and are laundered in place once
// per use, else (one wave per SIMD, 256 floats a lane, part of them in
// accumulation registers) each use goes through pin4.
template <int RB, int CPL, int NT, bool SPIN>
__global__ __launch_bounds__(NT, 1) void k_lz_resident(LanczosWS w, unsigned* bar,
                                                       const double* __restrict__ q1) {
  constexpr int NW = NT / 64, NH = CPL / 4, KG = NT / RB, QS = RB + 1;   // QS: row stride of Qs (bank spread)
  constexpr bool INPLACE = RB * CPL <= 128;
  static_assert(CPL % 4 == 0 && RB % 8 == 0 && NT % RB == 0, "shape");
  const int b = blockIdx.x, nb = gridDim.x, tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int L = w.L, m = w.m, n_it = w.n_it, ldq = w.ldq, hs = ldq + 1;
  // SPIN: the wait limit from w.spin (SLH_OPT_WAIT_POLLS), else the constant
  const int spin = SPIN ? (w.spin > 0 ? w.spin : LR_SPIN) : LR_SPIN;
  const int r0 = b * RB;
  const int cb = wv * 64 * CPL + 4 * lane;
  extern __shared__ double Qs[];                 // [n_it + 1][QS]
  __shared__ double h2s[256], gs[256], als[256], bes[256];
  __shared__ double prw[NW][RB];
  __shared__ double zs[RB], qr[RB], qmr[RB], sgr[RB];
  __shared__ double rq[KG][RB + 1], rg[KG][RB + 1];
  __shared__ double red[3][NW];
  __shared__ double cpart[NT];
  const int ntc = res_copies(ldq);
  double* Spart = w.Spart;
  double* Hpart = w.H2part;
  double* H2 = w.H2;
  double* Tv = w.T;
  double* const Tr = w.T + (int64_t)(b % ntc) * m;   // the copy of t~ this block reads

  // the block's rows of Phi (rows past L are zero) and of q_0
  float4 ph[RB][NH];
#pragma unroll
  for (int r = 0; r < RB; ++r) {
    const int row = min(r0 + r, L - 1);
#pragma unroll
    for (int h = 0; h < NH; ++h) ph[r][h] = *(const float4*)(w.Phi + (int64_t)row * m + cb + 256 * h);
  }
  if (r0 + RB > L) {
#pragma unroll
    for (int r = 0; r < RB; ++r)
      if (r0 + r >= L) {
#pragma unroll
        for (int h = 0; h < NH; ++h) ph[r][h] = make_float4(0.f, 0.f, 0.f, 0.f);
      }
  }
  if (tid < RB) {
    const double q = (r0 + tid < L) ? q1[r0 + tid] : 0.0;
    Qs[tid] = q;
    zs[tid] = q;
  }
  __syncthreads();

  // partials of Phi^T zs over the block's rows, tagged with step e
  auto col_partials = [&](int e) {
    double col[CPL];
#pragma unroll
    for (int c = 0; c < CPL; ++c) col[c] = 0.0;
    if constexpr (INPLACE) launder_rows(ph);
#pragma unroll
    for (int r = 0; r < RB; ++r) {
      const double z = zs[r];
#pragma unroll
      for (int h = 0; h < NH; ++h) {
        const float4 x = INPLACE ? ph[r][h] : pin4(ph[r][h]);
        col[4 * h + 0] = fma((double)x.x, z, col[4 * h + 0]);
        col[4 * h + 1] = fma((double)x.y, z, col[4 * h + 1]);
        col[4 * h + 2] = fma((double)x.z, z, col[4 * h + 2]);
        col[4 * h + 3] = fma((double)x.w, z, col[4 * h + 3]);
      }
    }
    // column c of block b at ((c / CB) nb + b) CB + c % CB: the partials a block
    // reduces are contiguous (CB = m / nb, a multiple of 4)
    const int CB = m / nb;
#pragma unroll
    for (int h = 0; h < NH; ++h) {
      const int c = cb + 256 * h;
      double* dst = Spart + ((int64_t)(c / CB) * nb + b) * CB + c % CB;
#pragma unroll
      for (int q = 0; q < 4; q += 2) st_tag2(dst + q, col[4 * h + q], col[4 * h + q + 1], e);
    }
  };
  // t over the block's columns from the partials of step e (scaled by 1 / |z1|
  // when norm, |z1|^2 summed here from its partials first) into every copy,
  // tagged with step e; with kh >= 0 first the h2 entry kh.  Thread = (column
  // cl < CB, partial lane pl < NT / CB).  false when a wait failed.
  auto col_reduce = [&](bool norm, double& z2v, int e, int kh) -> bool {
    const int CB = m / nb;
    const int64_t base = (int64_t)b * nb * CB + tid;
    stores_done_barrier();
    double v[CPL], zv[1], hv[1];
    bool ok = ld_wait<CPL>([&](int u) { return Spart + base + u * NT; }, (1u << CPL) - 1u, e, bar, spin, v);
    if (norm)
      ok = ld_wait<1>([&](int) { return Hpart + (int64_t)tid * hs + ldq; }, tid < nb ? 1u : 0u, e,
                      bar, spin, zv) && ok;
    ok = ld_wait<1>([&](int) { return Hpart + (int64_t)tid * hs + kh; }, (kh >= 0 && tid < nb) ? 1u : 0u,
                    e, bar, spin, hv) && ok;
    if (!block_ok(ok)) return false;
    if (norm || kh >= 0) {
      double d2 = 0.0;
      if (!norm) zv[0] = 0.0;
      block_sum3(zv[0], hv[0], d2, red);
      if (norm) z2v = zv[0];
      if (kh >= 0 && tid == 0) st_tag(H2 + kh, hv[0], e);
    }
    double sm = 0.0;
#pragma unroll
    for (int u = 0; u < CPL; ++u) sm += v[u];
    // a column's partial lanes within a wave lie CB lanes apart: an xor
    // butterfly over them (both lanes of a pair get the same sum), then the
    // waves' sums (for CB >= 64, the column's lanes) in order
    for (int o = CB; o < 64; o <<= 1) sm += __shfl_xor(sm, o);
    const int SD = CB < 64 ? 64 : CB;
    if (lane < CB) cpart[tid] = sm;
    __syncthreads();
    // thread (copy r, column cl) sums the column (the same sum in every copy)
    for (int q = tid; q < CB * ntc; q += NT) {
      const int cl = q % CB, r = q / CB;
      double S = 0.0;
      for (int p = 0; p < NT / SD; ++p) S += cpart[p * SD + cl];
      const double t = norm ? (z2v > 0.0 ? S / sqrt(z2v) : 0.0) : S;
      st_tag(Tv + (int64_t)r * m + b * CB + cl, t, e);
    }
    stores_done_barrier();
    return true;
  };
  // sum over the blocks of the h2 partial k (or |z1|^2 for k = ldq) of step e
  auto hpart_sum = [&](int k, int e, double& out) -> bool {
    stores_done_barrier();
    double hv[1];
    const bool ok = ld_wait<1>([&](int) { return Hpart + (int64_t)tid * hs + k; }, tid < nb ? 1u : 0u,
                               e, bar, spin, hv);
    if (!block_ok(ok)) return false;
    double d1 = 0.0, d2 = 0.0;
    block_sum3(hv[0], d1, d2, red);
    out = hv[0];
    return true;
  };

  // t_0 = Phi^T q_0 and its |t_0|^2 partials: step 0 of the tags
  col_partials(0);
  double z2 = 0.0;
  if (!col_reduce(false, z2, 0, -1)) return;

  double amax = 0.0;
  const int idx = ((lane >> 5) & 1) * 4 + ((lane >> 4) & 1) * 2 + ((lane >> 3) & 1);
  for (int j = 0; j < n_it; ++j) {
    // ---- rows: the reduced values of the previous step (tags of step j),
    // those of this step tagged j + 1.  A wave takes its row dots as soon as its
    // own entries of t~ have arrived (the scalars of the step wait for values
    // of every block).
    double tv[CPL], h1[1];
    bool ok = ld_wait<CPL>([&](int u) { return Tr + cb + 256 * (u >> 2) + (u & 3); }, (1u << CPL) - 1u,
                           j, bar, spin, tv);
    // Phi t~ of the block's rows: 4 CPL products per lane and row, summed over
    // the wave 8 rows at a time (into prw), then over the NW waves
    if constexpr (INPLACE) launder_rows(ph);
#pragma unroll
    for (int r8 = 0; r8 < RB; r8 += 8) {
      double d[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        double x = 0.0;
#pragma unroll
        for (int h = 0; h < NH; ++h) {
          const float4 y = INPLACE ? ph[r8 + e][h] : pin4(ph[r8 + e][h]);
          x = fma((double)y.x, tv[4 * h + 0], x);
          x = fma((double)y.y, tv[4 * h + 1], x);
          x = fma((double)y.z, tv[4 * h + 2], x);
          x = fma((double)y.w, tv[4 * h + 3], x);
        }
        d[e] = x;
      }
      const double tot = wave_sum8_f64(d);
      if ((lane & 7) == 0) prw[wv][r8 + idx] = tot;
    }
    ok = ld_wait<1>([&](int) { return H2 + tid; }, tid < j ? 1u : 0u, j, bar, spin, h1) && ok;
    if (!block_ok(ok)) return;
    const double h2v = h1[0];
    // this thread's share of alpha~ = |t~|^2: every block holds all of t~ and
    // sums it in the same order, so every block gets the same value
    double apv = 0.0;
#pragma unroll
    for (int u = 0; u < CPL; ++u) apv = fma(tv[u], tv[u], apv);
    if (tid < j) h2s[tid] = h2v;
    __syncthreads();
    // g = T_{j-1} h2 (alpha_k on the diagonal, beta_k beside it; beta_{j-1} is
    // not part of T_{j-1}); alpha~ = |t~|^2, |h2|^2 and h2^T g
    double gi = 0.0;
    if (tid < j) {
      gi = als[tid] * h2v;
      if (tid > 0) gi = fma(bes[tid - 1], h2s[tid - 1], gi);
      if (tid + 1 < j) gi = fma(bes[tid], h2s[tid + 1], gi);
      gs[tid] = gi;
    }
    double alpha_t = apv, hh = h2v * h2v, hth = h2v * gi;
    block_sum3(alpha_t, hh, hth, red);
    double alpha = alpha_t, beta = 0.0, h2last = 0.0, ibeta = 0.0;
    if (j > 0) {
      const double b2 = z2 - hh;
      beta = b2 > 0.0 ? sqrt(b2) : 0.0;
      if (!(beta > w.tol * amax)) {             // breakdown: n_eff stays j
        if (b == 0 && tid == 0) {
          w.beta[j - 1] = beta;
          w.stop[0] = 1;
        }
        return;
      }
      h2last = h2s[j - 1];
      alpha = (z2 * alpha_t - hth) / (beta * beta) - 2.0 * h2last;
      // (the 256-thread kernel multiplies by 1 / beta below: one division per
      // step rather than two per row on the block's dependent path; at 512
      // threads the extra value held costs more than the divisions)
      if constexpr (NT <= 256) ibeta = 1.0 / beta;
    }
    amax = fmax(amax, fabs(alpha));
    if (tid == 0) {
      als[j] = alpha;
      if (j > 0) bes[j - 1] = beta;
      if (b == 0) {
        if (j > 0) w.beta[j - 1] = beta;
        w.alpha[j] = alpha;
        w.neff[0] = j + 1;
      }
    }
    // Q_{j-1} h2 and Q_{j-1} g of each row: thread = (row i, k-group kg)
    {
      const int i = tid % RB, kg = tid / RB;
      double aq = 0.0, ag = 0.0;
      for (int k = kg; k < j; k += KG) {
        const double qk = Qs[k * QS + i];
        aq = fma(qk, h2s[k], aq);
        ag = fma(qk, gs[k], ag);
      }
      rq[kg][i] = aq;
      rg[kg][i] = ag;
    }
    __syncthreads();
    if (tid < RB) {
      const int i = tid, row = r0 + i;
      double sub = 0.0, sg = 0.0;
      for (int q = 0; q < KG; ++q) {
        sub += rq[q][i];
        sg += rg[q][i];
      }
      double q = Qs[i], qm = 0.0;                 // j = 0: q_0
      if (j > 0) {
        if constexpr (NT <= 256) q = (row < L) ? (zs[i] - sub) * ibeta : 0.0;
        else q = (row < L) ? (zs[i] - sub) / beta : 0.0;
        qm = Qs[(j - 1) * QS + i];
        Qs[j * QS + i] = q;
        if (row < L) w.Q[(int64_t)j * L + row] = q;
      }
      qr[i] = q;
      qmr[i] = qm;
      sgr[i] = sg;
    }
    __syncthreads();
    // z1 of the block's rows, and their partial of |z1|^2 (wave 0 holds the RB rows)
    if (tid < 64) {
      double z = 0.0;
      if (tid < RB) {
        const int i = tid;
        double u = prw[0][i];
#pragma unroll
        for (int q = 1; q < NW; ++q) u += prw[q][i];
        const double q = qr[i];
        if constexpr (NT <= 256) {
          if (j > 0) u = (fma(sqrt(z2), u, -sgr[i]) - beta * h2last * q) * ibeta;
        } else {
          if (j > 0) u = (fma(sqrt(z2), u, -sgr[i]) - beta * h2last * q) / beta;
        }
        z = (u - alpha * q) - beta * qmr[i];
        z = (r0 + i < L) ? z : 0.0;
        zs[i] = z;
      }
      const double zz = wave_sum_f64(z * z);
      if (tid == 0) st_tag(Hpart + (int64_t)b * hs + ldq, zz, j + 1);
    }
    __syncthreads();
    // partials of Phi^T z1, then of h2 = Q_j^T z1 (k <= j): the h2 partials are
    // read only after the column partials have been reduced, so they are formed
    // while those travel
    col_partials(j + 1);
    if constexpr (NT <= 256) {
      // four threads per entry k (four lanes of a wave), RB / 4 rows each
      for (int t = tid; t < 4 * (j + 1); t += NT) {
        const int k = t >> 2, p4 = t & 3;
        const double* qk = Qs + k * QS + p4 * (RB / 4);
        const double* zq = zs + p4 * (RB / 4);
        double a2[2] = {0.0, 0.0};
#pragma unroll
        for (int i = 0; i < RB / 4; ++i) a2[i & 1] = fma(qk[i], zq[i], a2[i & 1]);
        double v = a2[0] + a2[1];
        v += __shfl_xor(v, 1);
        v += __shfl_xor(v, 2);
        if (p4 == 0) st_tag(Hpart + (int64_t)b * hs + k, v, j + 1);
      }
    } else {
      for (int k = tid; k <= j; k += NT) {
        double a4[4] = {0.0, 0.0, 0.0, 0.0};
        const double* qk = Qs + k * QS;
#pragma unroll
        for (int i = 0; i < RB; ++i) a4[i & 3] = fma(qk[i], zs[i], a4[i & 3]);
        st_tag(Hpart + (int64_t)b * hs + k, (a4[0] + a4[1]) + (a4[2] + a4[3]), j + 1);
      }
    }
    // ---- columns: |z1|^2 (every block), t~_{j+1}, h2
    int k0 = b;                                   // h2 entries of this block: b, b + nb, ...
    if (j + 1 < n_it) {
      if (!col_reduce(true, z2, j + 1, b <= j ? b : -1)) return;
      k0 = b + nb;
    } else {
      if (!hpart_sum(ldq, j + 1, z2)) return;
    }
    for (int k = k0; k <= j; k += nb) {
      double v = 0.0;
      if (!hpart_sum(k, j + 1, v)) return;
      if (tid == 0) st_tag(H2 + k, v, j + 1);
    }
  }
  // beta of the last step (reported; T does not use it)
  if (b == 0) {
    double hv[1];
    const bool ok = ld_wait<1>([&](int) { return H2 + tid; }, tid < n_it ? 1u : 0u, n_it, bar, spin, hv);
    if (!block_ok(ok)) return;
    double hh2 = hv[0] * hv[0], d1 = 0.0, d2 = 0.0;
    block_sum3(hh2, d1, d2, red);
    if (tid == 0) {
      const double b2 = z2 - hh2;
      w.beta[n_it - 1] = b2 > 0.0 ? sqrt(b2) : 0.0;
    }
  }
}

// Everything the kernel expects before it starts, in one launch: q_0 into
// Q[0], alpha, beta, n_eff, the breakdown flag and max |alpha| cleared (the
// streaming path's k_lz_start), and the status word and every buffer of tagged
// values zeroed (tag 0: not yet written).
struct ResClear {
  double* p[6];
  int64_t n[6];   // doubles
};
__global__ void k_lz_res_prep(LanczosWS w, const double* __restrict__ q1, ResClear z) {
  const int64_t t0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t st = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = t0; i < w.L; i += st) w.Q[i] = q1[i];
  for (int64_t i = t0; i < w.n_it; i += st) {
    w.alpha[i] = 0.0;
    w.beta[i] = 0.0;
  }
  if (t0 == 0) {
    w.stop[0] = 0;
    w.neff[0] = 0;
    w.amax[0] = 0.0;
    w.amax[1] = 0.0;
  }
#pragma unroll
  for (int q = 0; q < 6; ++q)
    for (int64_t i = t0; i < z.n[q]; i += st) z.p[q][i] = 0.0;
}

namespace {
struct ResShape {
  int rb, nb, nt;   // rows per block, blocks, threads per block
};
// The resident kernel's shape, or rb = 0 when it does not qualify: one window,
// m of 1024 (256 threads, 4 columns a lane) or 2048 (512 threads, 4 columns a
// lane), rb of 32 or 16 rows a block, nb = ceil(L / rb) rounded up to a power of
// two, dividing m, at most one block per compute unit and per row group of the
// workspace, n_it <= 256
ResShape res_shape(const LanczosWS& w, int n_cu) {
  ResShape s{0, 0, 0};
  if (w.n_act != 1 || (w.m != 1024 && w.m != 2048) || w.n_it > 256 || w.n_it < 1) return s;
  const int nt = w.m == 2048 ? 512 : LR_T;
  for (int rb : {32, 16}) {
    int nb = 1;                                // ceil(L / rb) rounded up to a power of two
    while (nb * rb < w.L) nb *= 2;             // (blocks past the last row hold zeros)
    if (nb > n_cu || nb > w.G3 || (nb & (nb - 1)) != 0 || w.m % nb != 0 || w.m / nb > nt ||
        w.m / nb < 4)
      continue;   // (G3 row groups: the rows of Spart and H2part)
    s.rb = rb;
    s.nb = nb;
    s.nt = nt;
    return s;
  }
  return s;
}
template <int RB, int CPL, int NT, bool SPIN>
hipError_t launch_res_t(const LanczosWS& w, const ResShape& sh, unsigned* bar, const double* q1,
                        bool check, hipStream_t s) {
  auto k = k_lz_resident<RB, CPL, NT, SPIN>;
  const size_t lds = (size_t)(w.n_it + 1) * (RB + 1) * sizeof(double);
  if (lds > 65536) {
    const hipError_t e =
        hipFuncSetAttribute((const void*)k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  if (check) {
    int per_cu = 0;
    const hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, (const void*)k, NT, lds);
    if (e != hipSuccess) return e;
    return per_cu >= 1 ? hipSuccess : hipErrorInvalidConfiguration;
  }
  hipLaunchKernelGGL(k, dim3(sh.nb), dim3(NT), lds, s, w, bar, q1);
  return hipGetLastError();
}
template <bool SPIN>
hipError_t launch_res_s(const LanczosWS& w, const ResShape& sh, unsigned* bar, const double* q1,
                        bool check, hipStream_t s) {
  if (w.m == 2048) return sh.rb == 32 ? launch_res_t<32, 4, 512, SPIN>(w, sh, bar, q1, check, s)
                                      : launch_res_t<16, 4, 512, SPIN>(w, sh, bar, q1, check, s);
  return sh.rb == 32 ? launch_res_t<32, 4, LR_T, SPIN>(w, sh, bar, q1, check, s)
                     : launch_res_t<16, 4, LR_T, SPIN>(w, sh, bar, q1, check, s);
}
// a wait limit other than the built-in one (SLH_OPT_WAIT_POLLS) takes an
// instantiation of its own, so that the limit stays a constant in the other
hipError_t launch_res(const LanczosWS& w, const ResShape& sh, unsigned* bar, const double* q1,
                      bool check, hipStream_t s) {
  return w.spin > 0 ? launch_res_s<true>(w, sh, bar, q1, check, s)
                    : launch_res_s<false>(w, sh, bar, q1, check, s);
}
}  // namespace

bool lanczos_resident_ok(const LanczosWS& w, int n_cu) {
  const ResShape sh = res_shape(w, n_cu);
  if (sh.rb == 0) return false;
  (void)hipGetLastError();
  return launch_res(w, sh, nullptr, nullptr, true, nullptr) == hipSuccess;
}

size_t lanczos_resident_bar_words(int n_cu) {
  (void)n_cu;
  return (size_t)LR_ERR + 32;   // the error word on a line of its own
}

hipError_t launch_lanczos_resident(const LanczosWS& w, const double* q1_act, unsigned* bar,
                                   int n_cu, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  (void)hipGetLastError();
  const ResShape sh = res_shape(w, n_cu);
  if (sh.rb == 0) return hipErrorInvalidValue;
  const int64_t hs = w.ldq + 1;
  ResClear z;
  const double* const bufs[6] = {(const double*)bar, w.Spart, w.H2part, w.T, w.Apart, w.H2};
  const int64_t lens[6] = {(int64_t)lanczos_resident_bar_words(n_cu) / 2, (int64_t)sh.nb * w.m,
                           (int64_t)sh.nb * hs, (int64_t)res_copies(w.ldq) * w.m, 0, hs};
  for (int q = 0; q < 6; ++q) {
    z.p[q] = const_cast<double*>(bufs[q]);
    z.n[q] = lens[q];
  }
  hipLaunchKernelGGL(k_lz_res_prep, dim3(256), dim3(256), 0, s, w, q1_act, z);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (e0) {
    e = hipEventRecord(e0, s);
    if (e != hipSuccess) return e;
  }
  e = launch_res(w, sh, bar, q1_act, false, s);
  if (e != hipSuccess) return e;
  if (e1) e = hipEventRecord(e1, s);
  return e;
}

}  // namespace slh
