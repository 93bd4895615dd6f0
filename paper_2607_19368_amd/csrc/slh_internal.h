// Internal launcher declarations shared by the host library and the kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace slh {

// ---- preparation (k_prep.hip) ----
// Row norms of X: nrm2_fm[i] = |bf16(x_i)|^2 and nrm_x[i] = |x_i| (X as given),
// both accumulated in fp64, and rowscale[i] = fp32(s_i * sqrt(2/m)) with
// s_i = exp(nrm2_fm[i] / (2 sqrt(D))) (or 1 for the Gaussian map).
// For fp32 X it also writes the bf16 copy Xb (row stride D) unless Xb is NULL.
hipError_t launch_rownorm(const void* X, int dtype, int64_t ldx, int64_t N, int D, int m,
                          int gauss, double* nrm2_fm, double* nrm_x, double* inv_x,
                          float* rowscale, uint16_t* Xb, hipStream_t s);

// dst[a] = src[winlist[a]] (L doubles each) for a < n_act; winlist on the device.
hipError_t launch_gather_windows(double* dst, const double* src, const int* winlist, int64_t L,
                                 int n_act, hipStream_t s);

// ---- feature map (k_featmap.hip) ----
struct FeatmapArgs {
  const uint16_t* X;      // bf16 rows, global token index, row stride ldx
  int64_t ldx;
  const uint16_t* Wt;     // [m][ldw] bf16 (transposed projection, zero for k >= D)
  const float* psi;       // [m]
  const float* rowscale;  // [N] global token index
  float* Phi;             // [n_rows][m]
  const int* winlist;     // active window -> window index (n_rows / L entries)
  int64_t n_rows;         // n_act * L
  int64_t L;
  int D, m;
  int ldw;                // D rounded up to a multiple of 64
};
// n_cu: compute units of the device (picks the tile shape).  e0/e1 (may be
// NULL): receive the kernel's own start / end timestamps.
hipError_t launch_featmap(const FeatmapArgs& a, int n_cu, hipStream_t s, hipEvent_t e0 = nullptr,
                          hipEvent_t e1 = nullptr);

// ---- Lanczos (k_lanczos.hip) ----
struct LanczosWS {
  int n_act, L, m, n_it, ldq;   // ldq = n_it + 1 vectors per window
  const float* Phi;             // [n_act][L][m]
  double* Q;                    // [n_act][ldq][L]  Lanczos basis, vector-major
  double* T;                    // [n_act][ldq][m]  t_j = Phi^T z1 / |z1| of step j-1 in slot j & 1
  double* Apart;                // [n_act][m/16]    partials of |t_j|^2 (= alpha_j) per 16 columns
  double* Z1;                   // [n_act][L]       z1 of the last step (before the second pass)
  double* Spart;                // [n_act][G3][m]   partials of Phi^T z1 per row group
  double* H2part;               // [n_act][G3][ldq+1] (slot ldq: |z1|^2)
  double* H2;                   // [n_act][ldq+1]   Q^T z1 and |z1|^2
  double* Zs;                   // [n_act][2][L]    row outputs of timing replays
  double* alpha;                // [n_act][n_it]
  double* beta;                 // [n_act][n_it]
  int* neff;                    // [n_act]  steps done
  int* stop;                    // [n_act]  1 after breakdown
  double* amax;                 // [n_act][2] max |alpha| so far (breakdown scale): step j reads
                                //   slot j & 1 and writes the other
  double tol;
  int NCH;                      // chunks of 16 rows per block of the pass
  int G3;                       // row groups of 16 NCH rows (one block of the pass each)
  int spin;                     // resident kernel: polls before a wait between blocks
                                //   gives up (0: the built-in 2^20)
};
// One pass over Phi per step (k_lz_step) and one reduction.  ev_before/ev_after
// (may be NULL): n_it events each, receiving the start and end timestamps of
// the pass of every step.  Requires m % 256 == 0, m <= 2048, 1 <= n_it <= 256.
hipError_t launch_lanczos(const LanczosWS& w, const double* q1_act, hipStream_t s,
                          const hipEvent_t* ev_before = nullptr,
                          const hipEvent_t* ev_after = nullptr);
// reps x the pass of step j, launched as in launch_lanczos but dry: its rows go
// to Zs and it records no alpha, beta, n_eff or breakdown (for timing); it
// rewrites Spart and H2part
hipError_t launch_lanczos_passes(const LanczosWS& w, int j, int reps, hipStream_t s);
// q_0 of every active window into Q[a][0], alpha and beta zeroed, the
// per-window state (n_eff, stop) cleared (k_lz_start)
hipError_t launch_lanczos_start(const LanczosWS& w, const double* q1_act, hipStream_t s);

// ---- resident Lanczos (k_lzres.hip): one window whose Phi fits in the register
// files, the whole run as one persistent kernel (rows of Phi held in registers;
// the blocks exchange step-tagged values instead of meeting at barriers) ----
// true when the shape qualifies (n_act 1, m 1024 or 2048, at most 32 rows per
// compute unit, n_it <= 256) and every block of the kernel can be resident
bool lanczos_resident_ok(const LanczosWS& w, int n_cu);
// 32-bit words of the kernel's status buffer; its error word, at index
// LZ_BAR_ERR, is nonzero after a wait between blocks timed out (the run's
// results are then invalid)
size_t lanczos_resident_bar_words(int n_cu);
constexpr int LZ_BAR_ERR = 32;
// one preparation kernel (q_0 into Q[0] and the state cleared as k_lz_start
// does; the status and exchange buffers zeroed), then the persistent kernel
// (bracketed by e0 / e1 when given); the same outputs as launch_lanczos
hipError_t launch_lanczos_resident(const LanczosWS& w, const double* q1_act, unsigned* bar,
                                   int n_cu, hipStream_t s, hipEvent_t e0 = nullptr,
                                   hipEvent_t e1 = nullptr);

// ---- eigensolve + Ritz + SimHash (k_eig.hip, k_hash.hip) ----
// Eigh(T) of every active window (theta: kept eigenvalues ascending, Seig their
// vectors) and Z = Q S[:, kept] (Algorithm 1), all on stream s.
hipError_t launch_eigh_ritz(const double* alpha, const double* beta, const int* neff, int n_act,
                            int n_it, int r, double* theta, double* Seig, const double* Q, int L,
                            int ldq, double* Z, int n_cu, hipStream_t s);
hipError_t launch_simhash(const double* Z, const double* R, const int* winlist, int n_act,
                          int L, int r, int bits, uint32_t* codes, double* proj,
                          hipStream_t s);

// ---- short windows (k_local.hip): Lanczos + Eigh + Ritz of each window in one
// wavefront, on the window's explicit L x L operator (L <= 32, n_it <= L) ----
bool local_supported(int L, int n_it, int r);
hipError_t launch_local(const float* Phi, int n_act, int m, int L, int n_it, int r, double tol,
                        const double* q1, double* Q, double* alpha, double* beta, int* neff,
                        double* theta, double* Z, hipStream_t s);

// ---- normalised operator (k_norm.hip): per window s = Phi (Phi^T 1), rows of
// Phi scaled in place by s_i^-1/2 (0 where s_i <= 0); s kept in s_out ----
int normalise_groups(int n_act, int L, int m, int n_cu);   // row groups G of the column sums
hipError_t launch_normalise(float* Phi, int n_act, int L, int m, int G, double* part, double* csum,
                            double* s_out, hipStream_t s);   // part: [n_act][G][m], csum: [n_act][m]

// ---- diagnostics (k_diag.hip): per window sum(theta) / ||Phi_w||_F^2 ----
hipError_t launch_energy(const float* Phi, const double* theta, int n_act, int L, int m, int r,
                         double* rowsq, double* energy, hipStream_t s);   // rowsq: [n_act][L]

// bucket purity: tiles = ntiles (A, B) pairs of 64-position blocks of the sorted
// member order; counts[0] += pairs with cos > thresh, counts[1] += pairs
hipError_t launch_purity(const void* X, int dtype, int64_t ldx, int D, const int* sval,
                         const int* sseg, const double* nrm, int64_t N, const int* tiles,
                         int ntiles, double thresh, unsigned long long* counts, hipStream_t s);

hipError_t launch_fill_u32(uint32_t* p, int64_t n, uint32_t v, hipStream_t s);

// ---- merge (k_merge.hip) ----
struct MergeWS {
  int n_win, L, bits, chunk_k, compact, D;
  int64_t N;
  const uint8_t* route;         // [n_win] 1 = spectral (device)
  const uint32_t* codes;        // [N]
  const double* nrm_x;          // [N]
  uint32_t* keyA; uint32_t* keyB;  // [N] radix-sort keys
  int* valA; int* valB;            // [N] radix-sort values (token index)
  int* tmpi;                    // [N] representative flags / ranks (token order)
  int* segid;                   // [N] bucket ordinal per sorted position
  int* segk;                    // [N] bucket ordinal -> window-local macro rank
  int* sval;                    // [N] member token per sorted position
  int* sloc;                    // [N] window-local macro rank per sorted position
  int* mw;                      // [n_win] macro count per window
  int* wbase;                   // [n_win + 1] first global macro index per window
  int* sseg;                    // [N] global macro index per sorted position
  int* Mtot;                    // [1]
  float* part;                  // [2 * nchunks][D] partial sums of cut buckets
  int* part_seg;                // [2 * nchunks] macro of the slot, -1 if unused
  int* part_cnt;                // [2 * nchunks]
  double* part_nsum;            // [2 * nchunks] sum of member norms
  int* part_end;                // [2 * nchunks] 1 if the bucket ends in this slot
  int CH;                       // sorted positions per reduction chunk (<= 64)
  int scheme;                   // position scheme: 0 max, 1 lower median, 2 mean (half to even)
  int* posv;                    // [N] scheme != 0: representative position at each run end
  long long* pre;               // [N] scheme != 0 or target: prefix sums / remainders
  const int* tw;                // [n_win] exact target length: budget per window (NULL = off)
  int* tg;                      // [N] exact target length: scratch
};
int merge_nchunks(int64_t N, int CH);
// preserved suffix: tail tokens N .. N + K - 1 become macro-tokens *Mtot .. *Mtot + K - 1
hipError_t launch_merge_report(const int* Mtot, const unsigned* err, unsigned* out, hipStream_t s);
hipError_t launch_merge_tail(const void* X, int dtype, int64_t ldx, int D, int64_t N, int K,
                             const int* Mtot, int compact, float* E, int* P, int* tok2macro,
                             hipStream_t s);
hipError_t launch_merge(const MergeWS& w, const void* X, int dtype, int64_t ldx,
                        float* E, int* P, int* tok2macro, hipStream_t s);

// ---- adaptive routing (k_route.hip) ----
// inv_x: 1 / |x_i| per row (0 for a zero row); part: n_win * route_slices(D) * 2
int route_slices(int D);
// fused row norms + scores (one read of X) for D <= 4096: the row-norm kernel's
// outputs for the n_win * L rows plus the scores; psu: n_win * G * 2 * D doubles
// with G = route_norm_groups(L, D) (0: not available, use the two kernels)
int route_norm_groups(int L, int D);
hipError_t launch_route_norm_scores(const void* X, int dtype, int64_t ldx, int n_win, int L,
                                    int D, int m, int gauss, double* nrm2_fm, double* nrm_x,
                                    double* inv_x, float* rowscale, uint16_t* Xb, double* psu,
                                    double* part, double* scores, hipStream_t s);
hipError_t launch_route_scores(const void* X, int dtype, int64_t ldx, const double* inv_x,
                               int n_win, int L, int D, double* part, double* scores,
                               hipStream_t s);

}  // namespace slh
