// Implicit Lanczos with full re-orthogonalization (Algorithm 2; operator of
// Eq. 4, A v = Phi (Phi^T v), never forming the N x N kernel).
//
// Each window runs its own recurrence; all windows advance in lockstep (grid
// dimension y = window).  Vectors and every reduction are fp64; Phi is fp32.
//
// A run is k_lz_start (q_0), k_lz_init (partials of Phi^T q_0), k_lz_reduce
// (t_0 = Phi^T q_0), then per step j one pass and (but for the last step) one
// reduction:
//   k_lz_step    one read of the step's Phi rows: q_j (second Gram-Schmidt pass
//                of step j-1, in row space), u = A q_j from the row dots with
//                t~_j, z1 = u - alpha_j q_j - beta_{j-1} q_{j-1} (the
//                three-term recurrence, i.e. the first pass), and the partials
//                of Phi^T z1, of h2 = Q_j^T z1 and of |z1|^2 per block of rows.
//   k_lz_reduce  t~_{j+1} = Phi^T z1 / |z1| with the partials of |t~|^2, and h2
//                and |z1|^2 for the next pass.
// t~_{j+1} differs from Phi^T q_{j+1} by the rounding-level h2 term, which the
// next pass carries into u and alpha through the Lanczos relation (see
// k_lz_step); the basis Q stays fully re-orthogonalized in row space.
// k_lz_h2sum and k_lz_last_beta give beta of the last step.  All partial sums are
// combined in a fixed order, so results are bitwise reproducible.  alpha_j and
// beta_j are those of Algorithm 2: alpha_j = q_j^T A q_j, beta_j the norm after
// re-orthogonalization.
#include "slh_device.h"
#include "slh_internal.h"

#include <hip/hip_ext.h>

#include <algorithm>
#include <type_traits>

namespace slh {

// The same over each 16-lane quarter (DPP only): lane l holds the quarter sum
// of value index ((l>>3)&1)*4 + ((l>>2)&1)*2 + ((l>>1)&1).  The 4-lane step
// pairs lane i with 7 - i of its 8-lane group (row_half_mirror), which, like
// i ^ 4, joins the two halves of the group.
__device__ __forceinline__ double quarter_sum8_f64(const double (&v)[8]) {
  const int lane = threadIdx.x & 63;
  double w[4];
  const bool b8 = lane & 8;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const double keep = b8 ? v[e + 4] : v[e];
    const double send = b8 ? v[e] : v[e + 4];
    w[e] = keep + dpp_f64<DPP_ROR8>(send);
  }
  double x[2];
  const bool b4 = lane & 4;
#pragma unroll
  for (int e = 0; e < 2; ++e) {
    const double keep = b4 ? w[e + 2] : w[e];
    const double send = b4 ? w[e] : w[e + 2];
    x[e] = keep + dpp_f64<DPP_HALF_MIRROR>(send);
  }
  const bool b2 = lane & 2;
  double y = (b2 ? x[1] : x[0]) + dpp_f64<DPP_XOR2>(b2 ? x[0] : x[1]);
  y += dpp_f64<DPP_XOR1>(y);
  return y;
}

// Sum of src[g * ld] over g < G with 16 loads in flight (fixed order).
// Every batch issues its 16 loads unconditionally (index clamped to G - 1, the
// surplus values masked to zero afterwards), so a ragged tail costs one round
// trip rather than one per element.
__device__ __forceinline__ double sum_strided(const double* __restrict__ src, int64_t ld, int G) {
  constexpr int NF = 16;
  double acc[NF];
#pragma unroll
  for (int e = 0; e < NF; ++e) acc[e] = 0.0;
  for (int g = 0; g < G; g += NF) {
    double v[NF];
#pragma unroll
    for (int e = 0; e < NF; ++e) v[e] = src[(int64_t)min(g + e, G - 1) * ld];
#pragma unroll
    for (int e = 0; e < NF; ++e) acc[e] += (g + e < G) ? v[e] : 0.0;
  }
#pragma unroll
  for (int h = NF / 2; h >= 1; h >>= 1) {
#pragma unroll
    for (int e = 0; e < h; ++e) acc[e] += acc[e + h];
  }
  return acc[0];
}

// Column reduction by one block of 512 threads over 16 columns: returns, in
// threads < 16, sum_{g<G} src[g*ld + c0 + threadIdx.x] (0 past ncol).  Thread
// (cl = tid & 15, pl = tid >> 4) sums rows pl, pl + 32, ...; the four partial
// lanes of a column within a wave are added by two butterflies and the 8 waves'
// sums in LDS, all in a fixed order.  All threads must call it.
__device__ __forceinline__ double colsum16(const double* __restrict__ src, int64_t ld, int G,
                                           int c0, int ncol) {
  __shared__ double red[8][17];
  const int tid = threadIdx.x, cl = tid & 15, pl = tid >> 4;
  const int col = c0 + cl;
  double acc = 0.0;
  if (col < ncol) {
    const int cnt = (G - pl + 31) / 32;
    acc = sum_strided(src + (int64_t)pl * ld + col, (int64_t)32 * ld, cnt > 0 ? cnt : 0);
  }
  acc = swap16_add(acc, acc);                   // + lane ^ 16
  acc = swap32_add(acc, acc);                   // + lane ^ 32
  if ((tid & 63) < 16) red[tid >> 6][cl] = acc;
  __syncthreads();
  double t = 0.0;
  if (tid < 16 && col < ncol) {
    for (int w = 0; w < 8; ++w) t += red[w][cl];
  }
  __syncthreads();
  return t;
}

// |z1|^2 of window a: the sum over the row groups of H2part[g][ldq], by a block
// of 512 threads in a fixed order (every caller gets the same bits).  Split in
// a load part (four clamped loads per thread and batch, for G3 <= 2048 one
// batch) and the reduction, so that a caller can put other loads in flight
// between them.
struct Z2Part {
  double v[4];
};
__device__ __forceinline__ Z2Part z2_load(const LanczosWS& w, int a, int g0) {
  const int hs = w.ldq + 1, G = w.G3, tid = threadIdx.x;
  const double* src = w.H2part + (int64_t)a * G * hs + w.ldq;
  Z2Part p;
#pragma unroll
  for (int e = 0; e < 4; ++e) p.v[e] = src[(int64_t)min(g0 + tid + 512 * e, G - 1) * hs];
  return p;
}
__device__ __forceinline__ double z2_add(const Z2Part& p, int G, int g0, double acc) {
#pragma unroll
  for (int e = 0; e < 4; ++e) acc += (g0 + (int)threadIdx.x + 512 * e < G) ? p.v[e] : 0.0;
  return acc;
}
__device__ __forceinline__ double z2_sum(const LanczosWS& w, int a, double* red) {
  double acc = 0.0;
  for (int g0 = 0; g0 < w.G3; g0 += 4 * 512) acc = z2_add(z2_load(w, a, g0), w.G3, g0, acc);
  return block_sum_f64(acc, red);
}

// Block g of nx = ceil(j / 16) + 1 (512 threads): H2[k] = sum over the row
// groups of the h2 partials for k in [16 g, 16 g + 16) (k < j), or, for the
// last block, |z1|^2 (slot ldq).
// stopped: the window broke down (nothing is written; the flag is read by the
// caller alongside the loads rather than before them).
__device__ __forceinline__ void h2_reduce_block(const LanczosWS& w, int a, int j, int g, int nx,
                                                int stopped) {
  const int hs = w.ldq + 1;
  const double* hp = w.H2part + (int64_t)a * w.G3 * hs;
  double* dst = w.H2 + (int64_t)a * hs;
  if (g == nx - 1) {
    __shared__ double red[8];
    const double v = z2_sum(w, a, red);
    if (threadIdx.x == 0 && !stopped) dst[w.ldq] = v;
  } else {
    const int c0 = g * 16;
    const double v = colsum16(hp, hs, w.G3, c0, j);
    if (threadIdx.x < 16 && c0 + threadIdx.x < j && !stopped) dst[c0 + threadIdx.x] = v;
  }
}

// ---------------------------------------------------------------------------
// The pass over Phi.  A block owns NCH chunks of RC = 16 consecutive rows and
// all m columns of them; 8 waves, wave = (row subset p, 256-column slice sl),
// sl = wave % ns, p = wave / ns; the WPS = RC / RPW subsets of RPW rows each
// cover a chunk (waves with p >= WPS, when ns does not divide 8, take no rows
// and load those of the last subset).  Lane = 4 columns (one float4 per row) of
// the wave's slice.  A chunk's rows are held in registers; when another chunk
// follows, they are copied to LDS after the row dots so that the next chunk's
// loads are in flight while this chunk's column sums are taken.
// ---------------------------------------------------------------------------
constexpr int LZ_RC = 16;

struct StepGeom {
  int sl, p;
  bool rows;
};
template <int RPW>
__device__ __forceinline__ StepGeom step_geom(int m) {
  constexpr int WPS = LZ_RC / RPW;
  const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const int ns = m >> 8;
  StepGeom gm;
  gm.sl = wave % ns;
  gm.p = wave / ns;
  gm.rows = gm.p < WPS;
  return gm;
}

// The float4 of one Phi row as an opaque value at its point of use, so that its
// conversion to fp64 is not hoisted: otherwise every row of the chunk is held
// converted (twice the registers) across the phases that use it.
__device__ __forceinline__ float4 pin_row(float4 x) {
  asm volatile("" : "+v"(x.x), "+v"(x.y), "+v"(x.z), "+v"(x.w));
  return x;
}

// Column partials of the block (4 per lane of each slice; the WPS row subsets of
// a slice are combined through cr in a fixed order) into Spart[a][g][:].
template <int WPS>
__device__ __forceinline__ void lz_store_colsums(const LanczosWS& w, int a, int g,
                                                 const StepGeom& gm, double (&col)[4],
                                                 double (*cr)[256]) {
  const int lane = threadIdx.x & 63, ns = w.m >> 8;
  if (WPS > 1) {
    if (gm.rows && gm.p > 0) {
#pragma unroll
      for (int e = 0; e < 4; ++e) cr[(gm.p - 1) * ns + gm.sl][4 * lane + e] = col[e];
    }
    __syncthreads();
    if (gm.rows && gm.p == 0) {
      for (int q = 1; q < WPS; ++q) {
#pragma unroll
        for (int e = 0; e < 4; ++e) col[e] += cr[(q - 1) * ns + gm.sl][4 * lane + e];
      }
    }
  }
  if (gm.rows && gm.p == 0) {
    double* dst = w.Spart + ((int64_t)a * w.G3 + g) * w.m + gm.sl * 256 + 4 * lane;
#pragma unroll
    for (int e = 0; e < 4; ++e) dst[e] = col[e];
  }
}

// Initial pass: partials of Phi^T q_0 (t_0 before reduction), over the same row
// groups as the step's pass.
template <int RPW>
__global__ __launch_bounds__(512) void k_lz_init(LanczosWS w) {
  constexpr int WPS = LZ_RC / RPW;
  const int a = blockIdx.y, g = blockIdx.x, tid = threadIdx.x, lane = tid & 63;
  const int L = w.L, m = w.m, nch = w.NCH;
  const int r0 = g * LZ_RC * nch;
  const StepGeom gm = step_geom<RPW>(m);
  const int prow = min(gm.p, WPS - 1) * RPW;
  const float* pbase = w.Phi + (int64_t)a * L * m + gm.sl * 256 + 4 * lane;
  const double* q0 = w.Q + (int64_t)a * w.ldq * L;
  __shared__ double zs[LZ_RC];
  __shared__ double cr[WPS > 1 ? 7 : 1][256];
  double col[4] = {0.0, 0.0, 0.0, 0.0};
  for (int c = 0; c < nch; ++c) {
    const int rc0 = r0 + LZ_RC * c;
    const double z = q0[min(rc0 + (tid & (LZ_RC - 1)), L - 1)];
    float4 v[RPW];
#pragma unroll
    for (int i = 0; i < RPW; ++i) v[i] = *(const float4*)(pbase + (int64_t)min(rc0 + prow + i, L - 1) * m);
    if (tid < LZ_RC) zs[tid] = (rc0 + tid < L) ? z : 0.0;
    __syncthreads();
    if (gm.rows) {
#pragma unroll
      for (int i = 0; i < RPW; ++i) {
        const double zz = zs[gm.p * RPW + i];
        const float4 x = pin_row(v[i]);
        col[0] = fma((double)x.x, zz, col[0]);
        col[1] = fma((double)x.y, zz, col[1]);
        col[2] = fma((double)x.z, zz, col[2]);
        col[3] = fma((double)x.w, zz, col[3]);
      }
    }
    __syncthreads();
  }
  lz_store_colsums<WPS>(w, a, g, gm, col, cr);
}

// ---------------------------------------------------------------------------
// One Lanczos step j on the block's rows, with one read of their Phi rows.
// From the previous step: z1 (row space), h2 = Q_{j-1}^T z1 and |z1|^2 (reduced),
// and t~ = Phi^T z1 / |z1| with alpha~ = |t~|^2 (feature space).
//   beta_{j-1} = |z1 - Q_{j-1} h2| = sqrt(|z1|^2 - |h2|^2) (Q orthonormal), and
//     the breakdown test;
//   q_j = (z1 - Q_{j-1} h2) / beta_{j-1}     (second Gram-Schmidt pass of step
//     j-1, in row space; stored as Q[j]);
//   u = A q_j from the row dots Phi t~ = A z1 / |z1| and the Lanczos relation
//     A Q_{j-1} = Q_{j-1} T_{j-1} + beta_{j-1} q_j e^T (T_{j-1} tridiagonal of
//     the alphas and betas so far):
//       u = (|z1| Phi t~ - Q_{j-1} g - beta_{j-1} h2_{j-1} q_j) / beta_{j-1},
//       g = T_{j-1} h2;
//     alpha_j = q_j^T A q_j = (|z1|^2 alpha~ - h2^T g) / beta_{j-1}^2 - 2 h2_{j-1};
//     (without this correction the h2 of each step would re-enter the next one
//     amplified by |A| / beta);
//   z1 = u - alpha_j q_j - beta_{j-1} q_{j-1}   (the three-term recurrence);
//   partials of Phi^T z1 (column sums), of h2 = Q_j^T z1 and of |z1|^2 over the
//   block's rows.
// Row-space work of a chunk: thread = (row rl < 16, k-group kg < 32); MAXT =
// slots of k = kg + 32 t per thread, 32 MAXT >= n_it.
// dry = 1 (timing replays): q_j and z1 go to Zs, no bookkeeping, no breakdown exit.
// Dynamic LDS: 16 m floats (the staged chunk) when NCH > 1, else none.
// ---------------------------------------------------------------------------
// STAGED: blocks of NCH > 1 chunks (else NCH = 1, no LDS staging and a smaller
// register footprint, two blocks per CU).
// Unstaged: at most 128 VGPRs (four waves per SIMD), so that two blocks share a
// CU and all of the pass's blocks are resident at once.
template <int RPW, int MAXT, bool STAGED>
__global__ __launch_bounds__(512, STAGED ? 2 : 4) void k_lz_step(LanczosWS w, int j, int dry) {
  constexpr int RC = LZ_RC, WPS = RC / RPW, KG = 512 / RC;
  extern __shared__ float4 phis[];             // [RC][m / 4] staged chunk
  const int a = blockIdx.y, g = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63;
  const int L = w.L, m = w.m, hs = w.ldq + 1, nbr = m >> 4, nch = w.NCH, m4 = m >> 2;
  const int r0 = g * RC * nch;
  const StepGeom gm = step_geom<RPW>(m);
  const int rl = tid & (RC - 1), kg = tid / RC;
  const double* Qa = w.Q + (int64_t)a * w.ldq * L;
  const int jm = max(j - 1, 0);
  const int prow = min(gm.p, WPS - 1) * RPW;   // the wave's rows within a chunk
  const float* pbase = w.Phi + (int64_t)a * L * m + gm.sl * 256 + 4 * lane;
  // Every small load is issued before the Phi rows, so waiting for them leaves
  // the Phi loads in flight.  Every load is unconditional, with clamped indices
  // (surplus values are unused): a load under a branch would make the compiler
  // wait, where the branches join, as if the other path had issued no later
  // loads, i.e. for most of the Phi rows.
  const double* H2a = w.H2 + (int64_t)a * hs;
  const double h2v = H2a[min(tid, jm)];        // n_it <= 512
  const double z2 = H2a[w.ldq];
  const double apv = w.Apart[(int64_t)a * nbr + min(tid, nbr - 1)];
  const double alv = w.alpha[(int64_t)a * w.n_it + min(tid, jm)];
  const double bev = w.beta[(int64_t)a * w.n_it + min(tid, jm)];
  // the neighbours of entry tid of h2 and beta, for g = T_{j-1} h2 without an
  // LDS exchange, and h2_{j-1}
  const double h2p = H2a[max(min(tid - 1, jm), 0)], h2n = H2a[min(tid + 1, jm)];
  const double bep = w.beta[(int64_t)a * w.n_it + max(min(tid - 1, jm), 0)];
  const double h2l = H2a[jm];
  const int stopped = w.stop[a];
  const double amax0 = w.amax[2 * a + (j & 1)];   // max |alpha| before step j
  double tv[4];
  {
    const double* tt = w.T + ((int64_t)a * w.ldq + (j & 1)) * m + gm.sl * 256 + 4 * lane;
#pragma unroll
    for (int e = 0; e < 4; ++e) tv[e] = tt[e];
  }
  // keep the t~ loads ahead of the Phi rows (the first row dot needs them; issued
  // after the rows, waiting for them would wait for every row)
  __builtin_amdgcn_sched_barrier(0);
  // a chunk's loads: Q[k][row] for k = kg + KG t < j, z1 and q_{j-1} of the
  // thread's row, the wave's Phi rows
  double qv[MAXT], zp, qp;
  float4 v[RPW];
  auto load_chunk = [&](int c) {
    const int rc0 = r0 + RC * c;
    const int irc = min(rc0 + rl, L - 1);
#pragma unroll
    for (int t = 0; t < MAXT; ++t) qv[t] = Qa[(int64_t)min(kg + KG * t, jm) * L + irc];
    zp = w.Z1[(int64_t)a * L + irc];
    qp = Qa[(int64_t)jm * L + irc];            // q_{j-1}, or q_0 when j = 0
#pragma unroll
    for (int i = 0; i < RPW; ++i) v[i] = *(const float4*)(pbase + (int64_t)min(rc0 + prow + i, L - 1) * m);
  };
  load_chunk(0);
  if (stopped) return;
  __shared__ double h2s[264], gs[264];
  __shared__ double rq[KG][RC + 1], rg[KG][RC + 1];
  __shared__ double pr[RC][9];
  __shared__ double zs[RC];
  __shared__ double cr[WPS > 1 ? 7 : 1][256];
  // g = T_{j-1} h2 (alpha_i on the diagonal, beta_i beside it; beta_{j-1} is
  // not part of T_{j-1}) from the loaded neighbours; |t~|^2 (alpha~), |h2|^2 and
  // h2^T g summed as block_sum_f64 does (wave butterflies, then the 8 waves in
  // order), with h2 and g put in LDS, under one barrier
  const int wv = tid >> 6;
  __shared__ double red3[3][8];
  {
    double gi = 0.0;
    if (tid < j) {
      gi = alv * h2v;
      if (tid > 0) gi = fma(bep, h2p, gi);
      if (tid + 1 < j) gi = fma(bev, h2n, gi);
      h2s[tid] = h2v;
      gs[tid] = gi;
    }
    const double va = wave_sum_f64((tid < nbr) ? apv : 0.0);
    const double vh = wave_sum_f64((tid < j) ? h2v * h2v : 0.0);
    const double vg = wave_sum_f64((tid < j) ? h2v * gi : 0.0);
    if (lane == 0) {
      red3[0][wv] = va;
      red3[1][wv] = vh;
      red3[2][wv] = vg;
    }
  }
  __syncthreads();
  double alpha_t = 0.0, hh = 0.0, hth = 0.0;
  for (int q = 0; q < 8; ++q) {
    alpha_t += red3[0][q];
    hh += red3[1][q];
    hth += red3[2][q];
  }
  double alpha = alpha_t, beta = 0.0, h2last = 0.0;
  if (j > 0) {
    const double b2 = z2 - hh;
    beta = b2 > 0.0 ? sqrt(b2) : 0.0;
    if (!dry && !(beta > w.tol * amax0)) {     // breakdown: n_eff stays j
      if (g == 0 && tid == 0) {
        w.beta[(int64_t)a * w.n_it + j - 1] = beta;
        w.stop[a] = 1;
      }
      return;
    }
    h2last = h2l;
    alpha = (z2 * alpha_t - hth) / (beta * beta) - 2.0 * h2last;
  }
  if (!dry && g == 0 && tid == 0) {
    if (j > 0) w.beta[(int64_t)a * w.n_it + j - 1] = beta;
    w.alpha[(int64_t)a * w.n_it + j] = alpha;
    w.amax[2 * a + ((j + 1) & 1)] = fmax(amax0, fabs(alpha));   // the other slot:
    w.neff[a] = j + 1;                                          // read by the next step
  }
  const double zn = sqrt(z2);
  double* qdst = dry ? w.Zs + (int64_t)a * 2 * L : w.Q + ((int64_t)a * w.ldq + j) * L;
  double* zdst = dry ? w.Zs + ((int64_t)a * 2 + 1) * L : w.Z1 + (int64_t)a * L;
  double col[4] = {0.0, 0.0, 0.0, 0.0};      // Phi^T z1 over the block's rows
  double h2acc[MAXT];                         // Q[k] z1 over this thread's rows
#pragma unroll
  for (int t = 0; t < MAXT; ++t) h2acc[t] = 0.0;
  double qz = 0.0, zz = 0.0;                  // q_j . z1 and |z1|^2 (threads < RC)
  const int idx = ((lane >> 5) & 1) * 4 + ((lane >> 4) & 1) * 2 + ((lane >> 3) & 1);
  // one chunk; MORE: another chunk follows (stage this one in LDS, prefetch the next)
  // Phi t~ over rows [i0, i1) of the wave: 4 products per lane summed over the
  // wave (8 rows per butterfly), into pr (then summed over the slices)
  auto dots = [&](int i0, int i1) {
    if (gm.rows) {
#pragma unroll
      for (int b = i0; b < i1; b += 8) {
        double d[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          if (b + e < i1) {
            const float4 y = pin_row(v[b + e]);
            double x = (double)y.x * tv[0];
            x = fma((double)y.y, tv[1], x);
            x = fma((double)y.z, tv[2], x);
            d[e] = fma((double)y.w, tv[3], x);
          } else {
            d[e] = 0.0;
          }
        }
        const double tot = wave_sum8_f64(d);
        if ((lane & 7) == 0 && b + idx < i1) pr[gm.p * RPW + b + idx][gm.sl] = tot;
      }
    }
  };
  // k-group sums Q_{j-1} h2 and Q_{j-1} g of each row: wave 0, lane = (part,
  // row), 4 parts of KG / 4 groups combined by two butterflies (fixed order)
  auto kgroup_sums = [&](double& sub, double& sub_g) {
    sub = 0.0;
    sub_g = 0.0;
    if (tid < 64 && j > 0) {
      const int k0 = (tid >> 4) * (KG / 4);
#pragma unroll
      for (int k = 0; k < KG / 4; ++k) {
        sub += rq[k0 + k][rl];
        sub_g += rg[k0 + k][rl];
      }
      sub = swap16_add(sub, sub);
      sub_g = swap16_add(sub_g, sub_g);
      sub = swap32_add(sub, sub);
      sub_g = swap32_add(sub_g, sub_g);
    }
  };
  // q_j of the thread's row (threads < RC; stored) and the remaining terms of u
  auto row_q = [&](int ir, double sub, double zpc, double qpc, double& q, double& qm) {
    q = qpc;
    qm = 0.0;
    if (j > 0) {
      q = (zpc - sub) / beta;
      qm = qpc;
      if (ir < L) qdst[ir] = q;
    }
  };
  // z1 of the thread's row (threads < RC), stored, into zs
  auto row_z = [&](int ir, double sub_g, double q, double qm) {
    double z = 0.0;
    if (ir < L) {
      double u = 0.0;
      for (int s2 = 0; s2 < (m >> 8); ++s2) u += pr[rl][s2];
      if (j > 0) u = (fma(zn, u, -sub_g) - beta * h2last * q) / beta;
      z = (u - alpha * q) - beta * qm;
      zdst[ir] = z;
    }
    zs[rl] = z;
    qz = fma(q, z, qz);
    zz = fma(z, z, zz);
  };
  // column sums over rows [i0, i1) of the wave (from LDS when staged)
  auto colsums = [&](int i0, int i1, bool from_lds) {
    if (gm.rows) {
#pragma unroll
      for (int i = i0; i < i1; ++i) {
        const double zr = zs[gm.p * RPW + i];
        const float4 x = from_lds ? phis[(gm.p * RPW + i) * m4 + gm.sl * 64 + lane] : pin_row(v[i]);
        col[0] = fma((double)x.x, zr, col[0]);
        col[1] = fma((double)x.y, zr, col[1]);
        col[2] = fma((double)x.z, zr, col[2]);
        col[3] = fma((double)x.w, zr, col[3]);
      }
    }
  };
  auto chunk = [&](int c, auto more_tag) {
    constexpr bool MORE = decltype(more_tag)::value;
    const int ir = r0 + RC * c + rl;
    // row space: Q_{j-1} h2 (for q_j) and Q_{j-1} g (for u) over this thread's k
    {
      double aq[2] = {0.0, 0.0}, ag[2] = {0.0, 0.0};
#pragma unroll
      for (int t = 0; t < MAXT; ++t) {
        if (KG * t < j && kg + KG * t < j) {
          aq[t & 1] = fma(qv[t], h2s[kg + KG * t], aq[t & 1]);
          ag[t & 1] = fma(qv[t], gs[kg + KG * t], ag[t & 1]);
        }
      }
      rq[kg][rl] = aq[0] + aq[1];
      rg[kg][rl] = ag[0] + ag[1];
    }
    double qvc[MAXT];
#pragma unroll
    for (int t = 0; t < MAXT; ++t) qvc[t] = qv[t];
    const double zpc = zp, qpc = qp;
    // Staged: q_j and the k-group sums before the row dots (they need only the
    // prologue, so this barrier falls while the chunk's Phi rows are in flight).
    // Unstaged they follow the dots (taken before, they cost the 128-VGPR
    // kernel a spill: 19.0 against 18.2 us at qwen7b).
    double sub = 0.0, sub_g = 0.0, q = 0.0, qm = 0.0;
    __syncthreads();
    kgroup_sums(sub, sub_g);
    if (tid < RC) row_q(ir, sub, zpc, qpc, q, qm);
    if constexpr (MORE) {
      // stage this chunk's Phi rows in LDS and put the next chunk's loads in flight
      dots(0, RPW);
      if (gm.rows) {
#pragma unroll
        for (int i = 0; i < RPW; ++i) phis[(gm.p * RPW + i) * m4 + gm.sl * 64 + lane] = pin_row(v[i]);
      }
      load_chunk(c + 1);
      __syncthreads();
      if (tid < RC) row_z(ir, sub_g, q, qm);
      __syncthreads();
      colsums(0, RPW, true);
    } else {
      // (taking the rows in two halves, the first half's z1 and column sums while
      // the second half arrives, measured slower: 19.7 against 18.5 us at qwen7b)
      dots(0, RPW);
      __syncthreads();
      if (tid < RC) row_z(ir, sub_g, q, qm);
      __syncthreads();
      colsums(0, RPW, false);
    }
    const double zl = zs[rl];
#pragma unroll
    for (int t = 0; t < MAXT; ++t) h2acc[t] = fma(qvc[t], zl, h2acc[t]);
    if constexpr (MORE) __syncthreads();       // before the staged rows are replaced
  };
  if constexpr (STAGED) {
    for (int c = 0; c + 1 < nch; ++c) chunk(c, std::true_type{});
  }
  chunk(nch - 1, std::false_type{});
  lz_store_colsums<WPS>(w, a, g, gm, col, cr);
  // h2 partials: k < j summed over the 16 rows of each quarter wave (8 slots per
  // butterfly), then k = j and |z1|^2 over the first 16 threads
  double* hp = w.H2part + ((int64_t)a * w.G3 + g) * hs;
  const int hidx = ((lane >> 3) & 1) * 4 + ((lane >> 2) & 1) * 2 + ((lane >> 1) & 1);
#pragma unroll
  for (int t0 = 0; t0 < MAXT; t0 += 8) {
    if (KG * t0 < j) {                         // block-uniform
      double v8[8];
#pragma unroll
      for (int e = 0; e < 8; ++e)
        v8[e] = (t0 + e < MAXT && kg + KG * (t0 + e) < j) ? h2acc[min(t0 + e, MAXT - 1)] : 0.0;
      const double tot = quarter_sum8_f64(v8);
      const int k = kg + KG * (t0 + hidx);
      // lanes that agree in the index bits hold equal sums: one of them writes
      if ((lane & 1) == 0 && t0 + hidx < MAXT && k < j) hp[k] = tot;
    }
  }
  if (tid < 64) {
    // all of wave 0 takes part in every shuffle (a lane that skips one supplies
    // no value to it): lanes RC..2RC-1 take |z1|^2 of lanes 0..RC-1
    static_assert(RC == 16, "one row of 16 lanes");
    // lanes 16-31 take zz of lanes 0-15 (a 16-lane trade of zz with itself)
    const auto zl = __builtin_amdgcn_permlane16_swap(f64_lo(zz), f64_lo(zz), false, false);
    const auto zh = __builtin_amdgcn_permlane16_swap(f64_hi(zz), f64_hi(zz), false, false);
    double t = (tid < RC) ? qz : f64_of(zl[0], zh[0]);
    t += dpp_f64<DPP_ROR8>(t);
    t = oct_sum_f64(t);
    if (tid == 0) hp[j] = t;
    if (tid == RC) hp[w.ldq] = t;
  }
}

// ---------------------------------------------------------------------------
// Reduction after the pass of step j (j = -1: the initial pass): blocks
// [0, nx) reduce h2 (k <= j) and |z1|^2 over the row groups into H2; the others
// own 16 columns (x 32 partial lanes over the row groups): t_{j+1} = (Phi^T z1)
// / |z1| (Phi^T q_0 for the initial pass) into T[(j + 1) & 1], and the block's
// partial of |t_{j+1}|^2.
// ---------------------------------------------------------------------------
// CPB columns per column block, PL = 512 / CPB partial lanes over the row groups
// (CPB grows as G3 shrinks, so that few lanes idle; see launch_reduce).
template <int CPB>
__global__ __launch_bounds__(512) void k_lz_reduce(LanczosWS w, int j) {
  constexpr int PL = 512 / CPB;                     // partial lanes per column
  constexpr int WL = CPB < 64 ? 64 / CPB : 1;       // ... of them within one wave
  const int a = blockIdx.y, tid = threadIdx.x;
  const int m = w.m, hs = w.ldq + 1;
  const int nx = (j >= 0) ? (j + 16) / 16 + 1 : 0;
  int g = blockIdx.x;
  const int stopped = w.stop[a];                    // checked after the loads are out
  if (g < nx) {
    h2_reduce_block(w, a, j + 1, g, nx, stopped);
    return;
  }
  g -= nx;
  const int cl = tid % CPB, pl = tid / CPB;
  const int c = g * CPB + cl;                       // m is a multiple of CPB
  __shared__ double red[8];
  __shared__ double rs[PL / WL][CPB + 1];
  // |z1|^2 and the column sums with both sets of loads in flight together (the
  // same |z1|^2 routine and order as the h2 block, so t and the next pass use
  // the same |z1|); the |z1|^2 reduction's barriers come after the sums' loads
  double z2acc = 0.0;
  const Z2Part zp0 = z2_load(w, a, 0);              // unconditional: valid for any j
  const int cnt = (w.G3 - pl + PL - 1) / PL;
  const double s = sum_strided(w.Spart + ((int64_t)a * w.G3 + pl) * m + c, (int64_t)PL * m,
                               cnt > 0 ? cnt : 0);
  if (stopped) return;
  z2acc = z2_add(zp0, w.G3, 0, z2acc);
  for (int g0 = 4 * 512; g0 < w.G3; g0 += 4 * 512) z2acc = z2_add(z2_load(w, a, g0), w.G3, g0, z2acc);
  // |z1|^2 as block_sum_f64 forms it (wave butterflies, then the 8 waves in
  // order: the same bits as the h2 block) and the WL partial lanes of a column
  // within a wave by butterflies, then the waves' column sums, one barrier for both
  const double zw = wave_sum_f64(z2acc);
  double sw = s;
  static_assert(CPB >= 16, "partial lanes at distances 16 and 32 only");
  if constexpr (CPB <= 16) sw = swap16_add(sw, sw);   // + lane ^ 16
  if constexpr (CPB <= 32) sw = swap32_add(sw, sw);   // + lane ^ 32
  if ((tid & 63) == 0) red[tid >> 6] = zw;
  if (pl % WL == 0) rs[pl / WL][cl] = sw;
  __syncthreads();
  if (tid < CPB) {
    double z2 = 0.0;
    for (int q = 0; q < 8; ++q) z2 += red[q];
    double S = 0.0;
    for (int q = 0; q < PL / WL; ++q) S += rs[q][cl];
    double t = S;
    if (j >= 0) t = z2 > 0.0 ? S / sqrt(z2) : 0.0;
    w.T[((int64_t)a * w.ldq + ((j + 1) & 1)) * m + c] = t;
    // |t|^2 partials per 16 columns
    double t2 = t * t;
    t2 += dpp_f64<DPP_ROR8>(t2);                    // within rows of 16 lanes, all active
    t2 = oct_sum_f64(t2);
    if ((tid & 15) == 0) w.Apart[(int64_t)a * (m >> 4) + (c >> 4)] = t2;
  }
}

// beta of the last step (reported; T does not use it): h2 and |z1|^2 of the last
// orthogonalisation are reduced as at the start of a step, then
// beta = sqrt(|z1|^2 - |h2|^2).
__global__ __launch_bounds__(512) void k_lz_h2sum(LanczosWS w) {
  const int a = blockIdx.y;
  const int j = w.n_it, nx = (j + 15) / 16 + 1;
  h2_reduce_block(w, a, j, blockIdx.x, nx, w.stop[a]);
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
    w.amax[2 * a] = 0.0;
    w.amax[2 * a + 1] = 0.0;
  }
}


// rows per wave of a 16-row chunk: 16 / (8 / ns) for ns = m / 256 column slices
static int step_rpw(int m) { return LZ_RC / (8 / (m >> 8)); }

template <int RPW>
static void launch_init_t(const LanczosWS& w, hipStream_t s) {
  hipLaunchKernelGGL(k_lz_init<RPW>, dim3(w.G3, w.n_act), dim3(512), 0, s, w);
}
static void launch_init(const LanczosWS& w, hipStream_t s) {
  switch (step_rpw(w.m)) {
    case 2: launch_init_t<2>(w, s); break;
    case 4: launch_init_t<4>(w, s); break;
    case 8: launch_init_t<8>(w, s); break;
    default: launch_init_t<16>(w, s); break;
  }
}

template <int RPW, int MAXT, bool STAGED>
static hipError_t launch_step_s(const LanczosWS& w, int j, int dry, hipStream_t s, hipEvent_t e0,
                                hipEvent_t e1) {
  const dim3 g(w.G3, w.n_act), b(512);
  auto k = k_lz_step<RPW, MAXT, STAGED>;
  const size_t lds = STAGED ? (size_t)LZ_RC * w.m * sizeof(float) : 0;
  if (lds > 65536) {
    const hipError_t e = hipFuncSetAttribute((const void*)k, hipFuncAttributeMaxDynamicSharedMemorySize,
                                             (int)lds);
    if (e != hipSuccess) return e;
  }
  if (e0) hipExtLaunchKernelGGL(k, g, b, lds, s, e0, e1, 0, w, j, dry);
  else hipLaunchKernelGGL(k, g, b, lds, s, w, j, dry);
  return hipSuccess;
}
template <int RPW, int MAXT>
static hipError_t launch_step_t(const LanczosWS& w, int j, int dry, hipStream_t s, hipEvent_t e0,
                                hipEvent_t e1) {
  if (w.NCH > 1) return launch_step_s<RPW, MAXT, true>(w, j, dry, s, e0, e1);
  return launch_step_s<RPW, MAXT, false>(w, j, dry, s, e0, e1);
}
// MAXT: the smallest slot count with 32 MAXT >= n_it
template <int RPW>
static hipError_t launch_step_m(const LanczosWS& w, int j, int dry, hipStream_t s, hipEvent_t e0,
                                hipEvent_t e1) {
  if (w.n_it <= 128) return launch_step_t<RPW, 4>(w, j, dry, s, e0, e1);
  return launch_step_t<RPW, 8>(w, j, dry, s, e0, e1);
}
static hipError_t launch_step(const LanczosWS& w, int j, int dry, hipStream_t s,
                              hipEvent_t e0 = nullptr, hipEvent_t e1 = nullptr) {
  switch (step_rpw(w.m)) {
    case 2: return launch_step_m<2>(w, j, dry, s, e0, e1);
    case 4: return launch_step_m<4>(w, j, dry, s, e0, e1);
    case 8: return launch_step_m<8>(w, j, dry, s, e0, e1);
    default: return launch_step_m<16>(w, j, dry, s, e0, e1);
  }
}

// columns per column block: 16 (32 partial lanes) for 32 or more row groups,
// wider blocks for fewer (e.g. 8 row groups per window: 64 columns x 8 lanes)
static void launch_reduce(const LanczosWS& w, int j, hipStream_t s) {
  const int nx = (j >= 0) ? (j + 16) / 16 + 1 : 0;
  if (w.G3 >= 32) hipLaunchKernelGGL(k_lz_reduce<16>, dim3(nx + w.m / 16, w.n_act), dim3(512), 0, s, w, j);
  else if (w.G3 >= 16) hipLaunchKernelGGL(k_lz_reduce<32>, dim3(nx + w.m / 32, w.n_act), dim3(512), 0, s, w, j);
  else if (w.G3 >= 8) hipLaunchKernelGGL(k_lz_reduce<64>, dim3(nx + w.m / 64, w.n_act), dim3(512), 0, s, w, j);
  else hipLaunchKernelGGL(k_lz_reduce<128>, dim3(nx + w.m / 128, w.n_act), dim3(512), 0, s, w, j);
}

hipError_t launch_lanczos_start(const LanczosWS& w, const double* q1_act, hipStream_t s) {
  hipLaunchKernelGGL(k_lz_start, dim3((w.L + 255) / 256, w.n_act), dim3(256), 0, s, w, q1_act);
  return hipGetLastError();
}

hipError_t launch_lanczos(const LanczosWS& w, const double* q1_act, hipStream_t s,
                          const hipEvent_t* ev_before, const hipEvent_t* ev_after) {
  (void)hipGetLastError();
  if (w.m % 256 != 0 || w.m > 2048 || w.n_it > 256 || w.n_it < 1 || w.NCH < 1 ||
      w.G3 != (w.L + LZ_RC * w.NCH - 1) / (LZ_RC * w.NCH))
    return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_lz_start, dim3((w.L + 255) / 256, w.n_act), dim3(256), 0, s, w, q1_act);
  launch_init(w, s);
  launch_reduce(w, -1, s);
  for (int j = 0; j < w.n_it; ++j) {
    const hipError_t e = launch_step(w, j, 0, s, ev_before ? ev_before[j] : nullptr,
                                     ev_after ? ev_after[j] : nullptr);
    if (e != hipSuccess) return e;
    if (j + 1 < w.n_it) launch_reduce(w, j, s);
  }
  hipLaunchKernelGGL(k_lz_h2sum, dim3((w.n_it + 15) / 16 + 1, w.n_act), dim3(512), 0, s, w);
  hipLaunchKernelGGL(k_lz_last_beta, dim3(w.n_act), dim3(256), 0, s, w);
  return hipGetLastError();
}

// reps x the pass of step j, launched as in launch_lanczos but dry
hipError_t launch_lanczos_passes(const LanczosWS& w, int j, int reps, hipStream_t s) {
  (void)hipGetLastError();
  for (int q = 0; q < reps; ++q) {
    const hipError_t e = launch_step(w, j, 1, s);
    if (e != hipSuccess) return e;
  }
  return hipGetLastError();
}

}  // namespace slh
