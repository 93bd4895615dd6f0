/*
 * slh.h - C ABI of the Spectral-LSH hot path on AMD MI355X (gfx950).
 *
 * Spectral-LSH (arXiv 2607.19368) compresses N token embeddings X (N x D)
 * into M macro-tokens: a random-feature map Phi of the unnormalised softmax
 * kernel (section 3.2, Eq. 2-3), Lanczos with full re-orthogonalization on the
 * implicit operator Phi (Phi^T v) (Eq. 4, Algorithm 2), an eigensolve of the
 * Lanczos tridiagonal T and the top-r Ritz coordinates Z (Algorithm 1),
 * SimHash of Z (Eq. 5) and a merge of each hash bucket into one renormalised
 * mean with the bucket's max position (Eq. 7, section 3.4), ordered by that
 * position (section 3.6).  The adaptive backend (section 3.6, Eq. 8) routes
 * windows of the prompt either to that path or to chunk pooling (section 3.5).
 *
 * Notation: N tokens, D embedding width (the paper's d), m random features
 * (the paper's D), n_it Lanczos steps (the paper's r in Algorithm 2), r kept
 * Ritz vectors (the paper's k), bits SimHash bits (the paper's b).
 *
 * Conventions for every call:
 *  - Return value: SLH_OK (0) or a negative SLH_E* code.  On error no output
 *    is written and slh_last_error() describes the cause.
 *  - "device" pointers are HIP device memory of the current device, owned by
 *    the caller; "host" pointers are ordinary host memory owned by the caller.
 *    The context owns every workspace (parameters, Phi, Lanczos basis, codes,
 *    merge scratch) and frees it in slh_destroy.
 *  - All GPU work is enqueued on the stream given to slh_set_stream (default:
 *    the null stream).  Calls return without waiting for it, except where a
 *    host output is produced (noted per call).
 *  - A context is not thread-safe; separate contexts are independent.
 *  - Calls must follow the path order: [slh_route] -> slh_feature_map ->
 *    slh_lanczos -> slh_simhash -> slh_merge; calling a step before its
 *    predecessor returns SLH_ESTATE.
 */
#ifndef SLH_H
#define SLH_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct slh_ctx slh_ctx;

/* status codes */
#define SLH_OK      0
#define SLH_EINVAL (-1)   /* bad argument, size or alignment                      */
#define SLH_ENOMEM (-2)   /* device or host allocation failed                     */
#define SLH_EHIP   (-3)   /* a HIP runtime call failed (message has the details)  */
#define SLH_ESTATE (-4)   /* step called out of order                             */

/* element types of X */
#define SLH_BF16 0        /* bfloat16, raw 16-bit patterns                          */
#define SLH_F32  1        /* float32                                                */

/* options for slh_set_option (set before slh_feature_map) */
#define SLH_OPT_KERNEL        1  /* 0: unbiased for exp(x.y/sqrt(D)) (default): the
                                    Eq. 3 map times s(x) = exp(|x|^2/(2 sqrt(D)));
                                    1: the Eq. 3 map as printed (Gaussian kernel)      */
#define SLH_OPT_WINDOW_LEN    2  /* window length L (N must be a multiple of L);
                                    0 (default) = one window of N tokens.  Every step
                                    then runs independently per window (section 3.5
                                    local backend, section 3.6 adaptive backend)       */
#define SLH_OPT_POS_MODE      3  /* 0: representative positions (default), 1: compact
                                    0..M-1 (section 5.6, compressed position mode)     */
#define SLH_OPT_BREAKDOWN_TOL 4  /* Lanczos stops when beta_j <= tol * max_i alpha_i
                                    (Algorithm 2 break); default 1e-10                 */
#define SLH_OPT_TIMING        5  /* 1: record HIP events around each stage and around
                                    every pass over Phi (see slh_stage_times)          */
#define SLH_OPT_NORMALIZE     7  /* 1: the normalised operator (section 3.2 remark on
                                    row normalisation; appendix on the softmax
                                    normalisation gap): per window, row sums
                                    s = Phi (Phi^T 1) are estimated and the rows of
                                    Phi scaled by s_i^-1/2 (0 where s_i <= 0) inside
                                    slh_feature_map, so Lanczos runs on
                                    diag(s)^-1/2 Phi Phi^T diag(s)^-1/2, similar to
                                    diag(s)^-1 Phi Phi^T.  Z holds that symmetric
                                    operator's Ritz vectors (the normalised
                                    operator's are diag(s)^-1/2 Z: the same SimHash
                                    codes).  0 (default): Phi Phi^T as in Eq. 4     */
#define SLH_OPT_POS_SCHEME    8  /* macro-token positions (section 3.4): 0 max of the
                                    members' positions (default), 1 lower median,
                                    2 mean rounded half to even; macro-tokens are
                                    ordered by that position, ties (mean only) by
                                    the max position.  Chunk groups of the adaptive
                                    backend use the same scheme                     */
#define SLH_OPT_KEEP_LAST     9  /* preserved suffix (section 3.5: every backend can
                                    keep final tokens as they are; section 5.1: 12
                                    by default): the last K tokens are not
                                    compressed; each follows the compressed
                                    macro-tokens as its own macro-token (its row,
                                    its position).  Windows tile the first N - K
                                    tokens (N - K must be a multiple of
                                    WINDOW_LEN); routing, Phi and the Lanczos
                                    outputs cover those tokens only; codes, the
                                    token map and X keep N rows (tail codes are
                                    0xFFFFFFFF).  0 (default) keeps none          */
#define SLH_OPT_TARGET_LEN    10 /* exact output length T (section 3.3: clusters are
                                    merged or split until their number matches the
                                    target; no algorithm is given, this library's
                                    reading): the spectral windows share
                                    B = T - chunk macro-tokens - KEEP_LAST as
                                    floor(B/n) (+1 for the first B mod n); a window
                                    with more buckets merges runs of consecutive
                                    macro-tokens (macro k -> floor(k T_w / M_w)),
                                    one with fewer cuts buckets into contiguous
                                    member runs apportioned by size (largest
                                    remainder).  Needs POS_SCHEME 0; slh_merge
                                    fails with SLH_EINVAL when a budget leaves
                                    [1, L].  0 (default): off                       */
#define SLH_OPT_SHORT_WINDOWS 6  /* 1 (default): windows of L <= 32 tokens run Lanczos,
                                    Eigh and Ritz in one wavefront per window on the
                                    explicit L x L operator Phi_w Phi_w^T (the same
                                    operator and recurrence; section 3.5 local
                                    backend); 0: the general path for every L          */
#define SLH_OPT_RESIDENT      11 /* 1 (default): a single window whose Phi fits in the
                                    register files (m of 1024 or 2048, at most 32
                                    rows per compute unit, n_it <= 256) runs the
                                    whole Lanczos loop of Algorithm 2 as one
                                    persistent kernel that holds its rows of Phi in
                                    registers (the same recurrence; partial sums in
                                    a different grouping); 0: one pass over Phi per
                                    step for every shape                             */
#define SLH_OPT_WAIT_POLLS    12 /* polls after which a wait of the resident Lanczos
                                    kernel for a value of another block gives up
                                    (the blocks then leave and the call that reads
                                    the run's results reports SLH_EHIP); 0
                                    (default): 2^20, far beyond any wait of a
                                    healthy run (about a second).  Small values
                                    exercise that error path                       */

/*
 * Random parameters of the method, drawn from `seed` with Philox4x32-10
 * (Salmon et al., SC'11): key = (seed lo, seed hi), counter = (block lo,
 * block hi, stream, window); block n gives the uniform
 * u = ((w0 >> 5) * 2^26 + (w1 >> 6)) / 2^53 and, with w2/w3 likewise, the
 * Box-Muller pair (sqrt(-2 ln(1-u_a)) cos(2 pi u_b), ... sin(...)) as elements
 * 2n, 2n+1.  Streams: 1 = W, 2 = psi, 3 = q1, 4 = R.
 *   W[k][j]  = bf16_rne(float(n_{k*m+j} / sqrt(sqrt(D))))    (section 3.2: variance 1/sqrt(d))
 *   psi[j]   = float(2 pi u_j)                                 (section 3.2: Uniform(0, 2 pi))
 *   R[c][l]  = n_{c*bits+l}                                    (Eq. 5: r_l ~ N(0, I))
 *   q1 (window w) = first n normals of stream 3, window w, scaled to unit norm
 *                                                              (Algorithm 2 start)
 * These two calls run on the host only and touch no GPU.
 */
/* W_out: host, D*m uint16 bf16 patterns, row-major [D][m] (may be NULL);
   psi_out: host, m floats (may be NULL); R_out: host, r*bits doubles,
   row-major [r][bits] (may be NULL). */
int slh_gen_params(uint64_t seed, int64_t D, int64_t m, int32_t r, int32_t bits,
                   uint16_t *W_out, float *psi_out, double *R_out);
/* q_out: host, n doubles. */
int slh_gen_start(uint64_t seed, int64_t window, int64_t n, double *q_out);

/*
 * Create a context for prompts of N tokens of width D with m random features,
 * r kept Ritz vectors and `bits` SimHash bits (Algorithm 1 inputs).  Draws the
 * parameters (above) on the host and uploads them to the current device.
 * Limits: N >= 2; 8 <= D <= 32768 and D % 8 == 0; m % 256 == 0 and 256 <= m <= 2048;
 * 1 <= r <= 128; 1 <= bits <= 16.  *out receives the context (NULL on error).
 */
int slh_create(slh_ctx **out, int64_t N, int64_t D, int64_t m, int32_t r,
               int32_t bits, uint64_t seed);
void slh_destroy(slh_ctx *ctx);
const char *slh_last_error(const slh_ctx *ctx);

int slh_set_option(slh_ctx *ctx, int32_t key, double value);
/* stream: a hipStream_t (NULL = null stream). */
int slh_set_stream(slh_ctx *ctx, void *stream);

/*
 * Adaptive routing (section 3.6): per window, the redundancy score of Eq. 8
 * (mean cosine of each row to the normalised sum of the rows), then
 *   spectral if rho >= 16, else chunk if L <= 4, else spectral iff score >= tau;
 * tau < 0 selects the schedule tau(rho): 0.70 at rho <= 2, linear in log2(rho)
 * through 0.60 at 8 and 0.55 at 16.  Chunk windows are pooled in groups of
 * k = max(1, round-half-even(rho)) consecutive tokens (section 3.5).
 * Without this call every window takes the spectral path.
 * X: device, N rows of width D, row stride ldx elements (ldx >= D, ldx % 8 == 0,
 * 16-byte aligned).  route_out: host, n_windows bytes (1 = spectral), may be
 * NULL; scores_out: host, n_windows doubles, may be NULL.  Synchronises the
 * stream (the routing decision is made on the host from the device scores).
 */
int slh_route(slh_ctx *ctx, const void *X, int32_t x_dtype, int64_t ldx,
              double rho, double tau, uint8_t *route_out, double *scores_out);

/*
 * Step 1 (Eq. 3, Algorithm 1 first line): Phi = s(x) sqrt(2/m) cos(bf16(X) W + psi)
 * for the tokens of every spectral window, stored fp32 in the context.
 * X as for slh_route.  The row norms behind s(x) (and the member norms slh_merge
 * uses) are taken from X on every call, unless slh_route has just taken them
 * from the same X (pointer, type and stride) for this pass; a new prompt may
 * therefore be written into the same buffer between passes.  Asynchronous.
 */
int slh_feature_map(slh_ctx *ctx, const void *X, int32_t x_dtype, int64_t ldx);

/*
 * Steps 2-3 (Algorithm 2, then Eigh(T) and the top-r Ritz coordinates of
 * Algorithm 1): n_it Lanczos steps on Phi (Phi^T v) with full
 * re-orthogonalization, in fp64, from the seeded start vector of each window;
 * then the top-r eigenpairs of T (ascending; each eigenvector's first nonzero
 * entry positive) and Z = Q S[:, n-r:n] (N x r, fp64, kept in the context).
 * Requires r <= n_it <= min(L, 256).  A window whose beta_j falls below the
 * breakdown tolerance stops after n_eff = j steps (not an error): its Z then has
 * r - min(r, n_eff) leading zero columns and zero Ritz values.
 * ritz_out: host, n_spectral * r doubles (ascending per window) or NULL;
 * iters_out: host, n_spectral int32 (n_eff per window) or NULL.  If either is
 * non-NULL the call synchronises the stream; with both NULL it is asynchronous.
 */
int slh_lanczos(slh_ctx *ctx, int32_t n_it, double *ritz_out, int32_t *iters_out);

/*
 * Step 4 (Eq. 5): code_i = sum_l [R[:, l] . z_i > 0] 2^l for tokens of spectral
 * windows.  codes_out: device, N uint32 (tokens of chunk windows get
 * 0xFFFFFFFF), or NULL (codes stay in the context).  Asynchronous.
 */
int slh_simhash(slh_ctx *ctx, uint32_t *codes_out);

/*
 * Step 5 (Eq. 7; section 3.4 max positions; section 3.6 ordering): one
 * macro-token per (window, code) bucket, and per chunk group of chunk windows:
 * E = mean of the member rows of X (as given) rescaled to the mean member norm
 * (zero if the mean is zero), position = max member token index (global, 0-based;
 * or 0..M-1 in compact mode), macro-tokens in ascending position order.
 * X: the same tokens passed to slh_feature_map (their row norms from that call
 * are reused; after slh_load of codes, or for another X, they are recomputed).
 * emb_out: device, cap x D floats (row-major); pos_out: device, cap int32;
 * tok2macro_out: device, N int32 (macro index of each token), may be NULL;
 * cap >= the bound n_spectral_windows * min(L, 2^bits) + chunk groups.
 * *M_out (host) receives M.  Synchronises the stream.  SLH_ESTATE while a
 * merge from slh_merge_async has not been waited for.
 */
int slh_merge(slh_ctx *ctx, const void *X, int32_t x_dtype, int64_t ldx,
              float *emb_out, int32_t *pos_out, int32_t *tok2macro_out,
              int64_t cap, int64_t *M_out);

/*
 * Step 5 (Eq. 7; section 3.4 max positions; section 3.6 ordering) as
 * slh_merge, without waiting: the merge is enqueued on the context's
 * stream and the call returns, so that the host can enqueue the next prompt's
 * steps (slh_feature_map ...) before this one's M is known.  The outputs hold
 * the result, and M is returned, once slh_merge_wait returns for this merge.
 * At most two merges may be outstanding (SLH_ESTATE otherwise); each is waited
 * for, in order.  A later merge writes its own outputs, so the caller gives
 * consecutive merges different output buffers if it reads them after the next
 * merge was enqueued.  Same arguments and errors as slh_merge, without M_out.
 */
int slh_merge_async(slh_ctx *ctx, const void *X, int32_t x_dtype, int64_t ldx,
                    float *emb_out, int32_t *pos_out, int32_t *tok2macro_out,
                    int64_t cap);

/*
 * Waits for the oldest merge enqueued by slh_merge_async and not yet waited for
 * (spinning on an event: the stream up to that merge has finished) and stores
 * its M in *M_out (host).  SLH_ESTATE when none is outstanding; SLH_EHIP when a
 * wait between blocks of the resident Lanczos kernel of that prompt timed out.
 */
int slh_merge_wait(slh_ctx *ctx, int64_t *M_out);

/* Capacity slh_merge needs for the current routing. */
int64_t slh_merge_capacity(const slh_ctx *ctx);

/*
 * Copy an intermediate result to host memory (parity checks and diagnostics).
 * Synchronises the stream.  `bytes` must equal the size listed:
 *   SLH_OUT_PHI    n_act*L*m floats      Phi rows of the spectral windows in order
 *   SLH_OUT_ALPHA  n_act*n_it doubles    diagonal of T per window (zero past n_eff)
 *   SLH_OUT_BETA   n_act*n_it doubles    beta_1..beta_{n_it} per window
 *   SLH_OUT_Z      n_act*L*r doubles     Ritz coordinates, row-major per window
 *   SLH_OUT_PROJ   n_act*L*bits doubles  SimHash projections R^T z_i
 *   SLH_OUT_CODES  N uint32              codes (0xFFFFFFFF for chunk windows)
 *   SLH_OUT_THETA  n_act*r doubles       kept Ritz values (ascending)
 *   SLH_OUT_Q      n_act*(n_it+1)*L doubles  Lanczos basis, vector-major
 *   SLH_OUT_WINDOWS n_act int32          window index of each spectral window
 *   SLH_OUT_ROWSUM n_act*L doubles       estimated row sums s (SLH_OPT_NORMALIZE = 1)
 * (n_act = number of spectral windows.)
 */
#define SLH_OUT_PHI     1
#define SLH_OUT_ALPHA   2
#define SLH_OUT_BETA    3
#define SLH_OUT_Z       4
#define SLH_OUT_PROJ    5
#define SLH_OUT_CODES   6
#define SLH_OUT_THETA   7
#define SLH_OUT_Q       8
#define SLH_OUT_WINDOWS 9
#define SLH_OUT_ROWSUM  10
int slh_copy_out(slh_ctx *ctx, int32_t which, void *dst_host, int64_t bytes);

/*
 * Replace a stage's result with caller data so a later stage can be checked on
 * its own (step-wise parity).  src: device memory, `bytes` exactly:
 *   SLH_OUT_PHI    n_act*L*m floats  -> Phi; the next call may be slh_lanczos
 *   SLH_OUT_ALPHA  n_act*n_it doubles -> the diagonal of T per window; sets the
 *                  order n_it (r <= n_it <= min(L, 256)) and n_eff = n_it for
 *                  every window, clears beta; load first
 *   SLH_OUT_BETA   n_act*n_it doubles -> beta_1..beta_{n_it} per window (the
 *                  first n_it - 1 are T's off-diagonal)
 *   SLH_OUT_Q      n_act*(n_it+1)*L doubles -> the basis, vector-major
 *                  (after alpha, beta and Q the next call may be slh_eigh_ritz)
 *   SLH_OUT_CODES  N uint32          -> codes; the next call may be slh_merge
 * Asynchronous (device-to-device copy on the context stream), except that
 * SLH_OUT_ALPHA synchronises the stream.
 */
int slh_load(slh_ctx *ctx, int32_t which, const void *src, int64_t bytes);

/*
 * Eigh(T) and the Ritz coordinates alone (Algorithm 1: lambda, V <- Eigh(T);
 * Z <- Q V[:, n-r:n]) on the tridiagonal and basis the context holds: those
 * of the last slh_lanczos, or alpha, beta and Q given by slh_load (stage-wise
 * checks of the eigensolver on a chosen T).  slh_lanczos already includes
 * this step.  n_it must equal the order of T.  Kept eigenvalues whose gaps are
 * at most 1e-8 |T| (|T| = max_k |alpha_k| + |beta_k-1| + |beta_k|) are a
 * cluster: their vectors are orthogonalised against each other within the
 * inverse iteration.  ritz_out / iters_out as for slh_lanczos (the call
 * synchronises when either is non-NULL).  SLH_ESTATE when neither a Lanczos
 * run nor a loaded alpha, beta and Q is present.
 */
int slh_eigh_ritz(slh_ctx *ctx, int32_t n_it, double *ritz_out, int32_t *iters_out);

/*
 * Stage timings of the most recent calls, from HIP events on the context
 * stream (requires SLH_OPT_TIMING = 1 before those calls).  Fills up to n of:
 *   [0] feature map ms        [1] Lanczos loop ms (all steps, all windows)
 *   [2] sum of Phi-pass ms     [3] number of Lanczos steps those passes cover
 *   (the resident kernel of SLH_OPT_RESIDENT is timed as one pass covering all
 *   n_it steps)
 *   [4] eigensolve + Ritz ms  [5] SimHash ms   [6] merge ms
 *   [7] row normalisation ms (SLH_OPT_NORMALIZE = 1, else 0)
 *   [8] 1 when the last slh_lanczos ran the resident kernel (SLH_OPT_RESIDENT)
 * Synchronises the stream.
 */
int slh_stage_times(slh_ctx *ctx, double *ms_out, int32_t n);

/*
 * Duration of one pass over Phi without per-launch events (measurement aid for
 * the matvec of Algorithm 2, A v = Phi (Phi^T v)): the pass kernel of the final
 * step of the last slh_lanczos call (u = Phi t_j and the partials of Phi^T z1
 * on one read of Phi, with the step's re-orthogonalisation work), with that
 * step's launch configuration and data, is captured reps times as one HIP
 * graph, replayed once untimed and once between two events on the context
 * stream.  us_out: host, 1 double = elapsed microseconds / reps, so gaps
 * between graph nodes are included.  The replays write their row vectors to
 * scratch and record no step state: they rewrite only the step's partial sums,
 * never Q, alpha, beta, the Ritz pairs or codes; windows that broke down early
 * skip their passes as in the loop itself.  After a run of the resident kernel
 * (SLH_OPT_RESIDENT) the call instead launches that run reps times, each
 * kernel between two events (its preparation kernel outside them), and us_out is the kernel's mean duration over the runs after the
 * first, divided by n_it (per Lanczos step); those runs recompute the whole
 * Lanczos loop and rewrite Q, alpha and beta with the same values.  reps in
 * [1, 4096].  Synchronises the stream.  SLH_ESTATE before slh_lanczos or after a short-window
 * (single-wavefront) Lanczos run, which has no passes.
 */
int slh_time_passes(slh_ctx *ctx, int32_t reps, double *us_out);

/*
 * Spectral-energy fraction (section 5 kill test on spectral energy; rank
 * ablation): for each spectral window, sum of its r kept Ritz values divided by
 * tr(Phi_w Phi_w^T) = ||Phi_w||_F^2, the squared Frobenius norm of the rows the
 * Lanczos step used (after the row normalisation when SLH_OPT_NORMALIZE = 1);
 * 0 for a window whose rows are all zero.  Call after slh_lanczos.
 * energy_out: host, n_spectral doubles (window order of SLH_OUT_WINDOWS).
 * Synchronises the stream.  SLH_ESTATE before slh_lanczos.
 */
int slh_spectral_energy(slh_ctx *ctx, double *energy_out);

/*
 * Bucket purity (section 5 kill test on buckets): over token pairs i < j that
 * share a bucket of a spectral window, counts_out[0] = pairs whose rows of X
 * have cosine similarity > thresh (cosine 0 for a zero row), counts_out[1] =
 * all such pairs; purity = counts_out[0] / counts_out[1].  X as passed to
 * slh_merge (device, N x D, row stride ldx, x_dtype); thresh in [-1, 1] (the
 * paper uses 0.7).  Call after slh_merge.  counts_out: host, 2 int64.
 * Synchronises the stream.  SLH_ESTATE before slh_merge.
 */
int slh_bucket_purity(slh_ctx *ctx, const void *X, int32_t x_dtype, int64_t ldx, double thresh,
                      int64_t *counts_out);

/*
 * Measured ceilings for the roofline figures (measurement aids, not part of the
 * method; no context needed).  Both time `reps` launches (after one untimed
 * launch) with HIP events on `stream` (a hipStream_t, NULL = null stream) and
 * synchronise it.
 * slh_peak_read: a plain streaming read of every 16-byte word of buf (device,
 *   `bytes` long, a multiple of 16 and >= 4096, 16-byte aligned; its contents
 *   are not changed in practice) -> *gbs_out = bytes * reps / time in GB/s.  A
 *   buffer larger than the 256 MB Infinity Cache measures HBM; a smaller one
 *   read again and again measures what the cache serves.
 * slh_peak_mfma: independent chains of dense bf16 32x32x16 MFMAs with their
 *   operands in registers, two waves per SIMD on every CU -> *tflops_out in
 *   TFLOP/s.  sink: device, 16 bytes (written only in a case that does not occur).
 * reps in [1, 1000]; SLH_EINVAL for bad arguments, SLH_EHIP if a launch fails.
 */
int slh_peak_read(void *buf, int64_t bytes, int32_t reps, void *stream, double *gbs_out);
int slh_peak_mfma(int32_t reps, void *sink, void *stream, double *tflops_out);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the merge of
 * slh_merge for one window of N tokens from codes the caller supplies (what
 * slh_load(SLH_OUT_CODES) followed by slh_merge computes on a one-window
 * context: max positions, representative mode, no preserved suffix or target
 * length), with no context and no allocation.  Every workspace lives in one
 * fixed array of SLH_NOALLOC_BYTES device bytes per GPU, which the library
 * holds from its first call on that GPU until the process ends.
 * Limits: 2 <= N <= 8192; 8 <= D <= 4096, D % 8 == 0; 1 <= bits <= 16 and
 * every code < 2^bits; cap >= min(N, 2^bits).  Larger sizes are rejected with
 * SLH_EINVAL before any GPU work.
 * X: device, N x D of x_dtype, row stride ldx (ldx >= D, ldx % 8 == 0, 16-byte
 * aligned); codes: device, N uint32; emb_out: device, cap x D floats; pos_out:
 * device, cap int32; tok2macro_out: device, N int32, may be NULL; *M_out
 * (host) receives M.  stream: a hipStream_t (NULL = null stream); the call
 * synchronises it (M goes to the host).
 * Every call on one GPU uses that GPU's array and overwrites what the last call
 * left there: calls that overlap in time on one GPU (other threads, other
 * streams) race, and the caller must serialise them.  SLH_EHIP if the array's
 * device address cannot be obtained or a launch fails.
 */
#define SLH_NOALLOC_BYTES 17355008
int slh_merge_noalloc(const void *X, int32_t x_dtype, int64_t ldx, int64_t N, int64_t D,
                      const uint32_t *codes, int32_t bits, float *emb_out, int32_t *pos_out,
                      int32_t *tok2macro_out, int64_t cap, int64_t *M_out, void *stream);

/* Number of windows and of spectral windows of the current routing. */
int64_t slh_num_windows(const slh_ctx *ctx);
int64_t slh_num_spectral(const slh_ctx *ctx);

#ifdef __cplusplus
}
#endif

#endif /* SLH_H */
