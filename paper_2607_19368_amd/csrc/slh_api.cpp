// Host side of the C ABI declared in include/slh.h: argument checks, the
// method's seeded parameters, workspace ownership, and the launch sequence of
// each step.  All arithmetic of the path runs in the HIP kernels.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "slh.h"
#include "slh_internal.h"

using namespace slh;

// ---------------------------------------------------------------------------
// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11) and the derived streams.
// ---------------------------------------------------------------------------
namespace {

inline void philox4x32_10(uint32_t c[4], uint32_t k0, uint32_t k1) {
  for (int r = 0; r < 10; ++r) {
    if (r) {
      k0 += 0x9E3779B9u;
      k1 += 0xBB67AE85u;
    }
    const uint64_t p0 = (uint64_t)0xD2511F53u * c[0];
    const uint64_t p1 = (uint64_t)0xCD9E8D57u * c[2];
    const uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
    const uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
    const uint32_t n0 = hi1 ^ c[1] ^ k0, n2 = hi0 ^ c[3] ^ k1;
    c[0] = n0;
    c[1] = lo1;
    c[2] = n2;
    c[3] = lo0;
  }
}

inline void philox_block(uint64_t seed, uint32_t stream, uint32_t window, uint64_t n,
                         uint32_t out[4]) {
  out[0] = (uint32_t)n;
  out[1] = (uint32_t)(n >> 32);
  out[2] = stream;
  out[3] = window;
  philox4x32_10(out, (uint32_t)seed, (uint32_t)(seed >> 32));
}

inline double u53(uint32_t a, uint32_t b) {
  return ((double)(a >> 5) * 67108864.0 + (double)(b >> 6)) / 9007199254740992.0;
}

enum { STREAM_W = 1, STREAM_PSI = 2, STREAM_Q1 = 3, STREAM_R = 4 };

void gen_normals(uint64_t seed, uint32_t stream, uint32_t window, int64_t count, double* out) {
  const int64_t nb = (count + 1) / 2;
  for (int64_t n = 0; n < nb; ++n) {
    uint32_t w[4];
    philox_block(seed, stream, window, (uint64_t)n, w);
    const double ua = u53(w[0], w[1]), ub = u53(w[2], w[3]);
    const double rad = std::sqrt(-2.0 * std::log(1.0 - ua));
    const double ang = (2.0 * M_PI) * ub;
    out[2 * n] = rad * std::cos(ang);
    if (2 * n + 1 < count) out[2 * n + 1] = rad * std::sin(ang);
  }
}

inline uint16_t bf16_rne(float f) {
  uint32_t u;
  std::memcpy(&u, &f, 4);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

}  // namespace

// ---------------------------------------------------------------------------
// context
// ---------------------------------------------------------------------------
struct DevBuf {
  void* p = nullptr;
  size_t bytes = 0;
};

struct slh_ctx {
  int64_t N = 0, D = 0, m = 0;
  int r = 0, bits = 0;
  uint64_t seed = 0;
  int gauss = 0, compact = 0;
  int64_t L = 0, n_win = 1;
  double tol = 1e-10;
  hipStream_t stream = nullptr;
  hipStream_t cap_stream = nullptr;
  // results the host waits for (M, routing scores) arrive in pinned memory and
  // the host spins on an event rather than sleeping in a stream synchronisation
  void* pin = nullptr;
  size_t pin_bytes = 0;
  hipEvent_t ev_host = nullptr;
  // merges in flight (slh_merge_async): slot s = count & 1 of a pinned ring
  // holds (M, the resident Lanczos kernel's error word) of that merge, written
  // by the stream and marked by mq_ev[s]; mq_head merges enqueued, mq_tail waited for
  unsigned* mq_pin = nullptr;
  hipEvent_t mq_ev[2] = {nullptr, nullptr};
  int64_t mq_head = 0, mq_tail = 0;
  int mq_res[2] = {0, 0}, mq_keep[2] = {0, 0};
  int device = 0, n_cu = 256;
  std::string err;

  // routing
  std::vector<uint8_t> route_h;
  std::vector<int> winlist_h;
  int n_act = 0, chunk_k = 1;
  bool routed = false;
  bool routing_on_device = false;

  // stage: 0 ready, 1 feature map done, 2 Lanczos done, 3 SimHash done
  int stage = 0;
  int n_it = 0;
  // Row norms (s(x) of Eq. 3, the member norms of Eq. 7) are computed from X
  // by slh_route or slh_feature_map and reused only within the same pass over
  // one prompt: slh_feature_map recomputes them unless slh_route has just
  // computed them for the same X (norms_fresh), and slh_merge reuses them only
  // if they were computed for the same X in this pass.  A new prompt written
  // into the same buffer therefore never inherits the previous prompt's norms.
  const void* norms_of = nullptr;   // X (pointer, type, stride) the row norms were taken from
  int32_t norms_dtype = -1;
  int64_t norms_ldx = -1;
  bool norms_fresh = false;         // set by slh_route, consumed by slh_feature_map
  int64_t q1_L = -1;                // window length q1all was drawn for

  std::vector<DevBuf*> all;
  DevBuf Wt, psi, R, q1all, q1act, winlist, route;
  DevBuf nrm2_fm, nrm_x, inv_x, rowscale, Xb, Phi;
  DevBuf Q, T, Apart, Z1, Spart, Zs, H2part, H2, alpha, beta, neff, stop, amax;
  DevBuf theta, Seig, Z, proj, codes;
  DevBuf keyA, keyB, valA, valB, tmpi, segid, segk, sval, sloc, mw, wbase, sseg, Mtot;
  DevBuf part, part_seg, part_cnt, part_nsum, part_end;
  DevBuf rpart, scores, rsu;

  hipGraphExec_t lz_exec = nullptr;
  std::string lz_key;
  LanczosWS lz_w{};                 // workspace of the last full-size Lanczos run
  bool lz_w_valid = false;
  bool lz_res = false;              // that run used the resident kernel
  int resident = 1;                 // SLH_OPT_RESIDENT
  int wait_polls = 0;               // SLH_OPT_WAIT_POLLS (0: the built-in limit)
  DevBuf lz_bar;                    // its grid-barrier words (generation, error, arrivals)

  int short_win = 1;                // SLH_OPT_SHORT_WINDOWS
  int normalize = 0;                // SLH_OPT_NORMALIZE
  int pos_scheme = 0;               // SLH_OPT_POS_SCHEME
  int merged = 0;                   // slh_merge ran on the current codes
  int t_loaded = 0;                 // slh_load of alpha (1), beta (2), Q (4) since slh_lanczos
  int64_t Ntot = 0;                 // prompt length; N = Ntot - keep_last tokens are compressed
  int64_t keep_last = 0;            // SLH_OPT_KEEP_LAST
  int64_t target_len = 0;           // SLH_OPT_TARGET_LEN (0 = off)
  std::vector<int> tw_h;            // per-window budgets of the last merge
  std::vector<int> tw_dev_h;        // the budgets in tg_tw (uploaded to tw_dev_p)
  void* tw_dev_p = nullptr;
  DevBuf tg_tw, tg_scr;
  DevBuf dg_tiles, dg_counts;
  DevBuf posv, mg_pre;
  DevBuf nm_part, nm_csum, rowsum;
  DevBuf dg_rowsq, dg_energy;

  // timing (SLH_OPT_TIMING)
  int timing = 0;
  std::vector<hipEvent_t> ev_fb, ev_fa;    // around each fused pass
  hipEvent_t ev[12] = {};                   // stage brackets: fm, lz, eig, sh, mg
  bool ev_made = false;
  int fused_timed = 0;              // event pairs in ev_fb / ev_fa
  int passes_timed = 0;             // Lanczos steps they cover
  int norm_timed = 0;
};

namespace {

int fail(slh_ctx* c, int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  if (c) c->err = buf;
  return code;
}

#define HIP_TRY(c, expr)                                                                   \
  do {                                                                                     \
    hipError_t e_ = (expr);                                                                \
    if (e_ != hipSuccess)                                                                  \
      return fail((c), SLH_EHIP, "%s failed: %s", #expr, hipGetErrorString(e_));           \
  } while (0)

// grow-only device buffer
int ensure(slh_ctx* c, DevBuf& b, size_t bytes) {
  if (bytes == 0) bytes = 16;
  if (b.bytes >= bytes) return SLH_OK;
  if (b.p) {
    hipError_t e = hipFree(b.p);
    if (e != hipSuccess) return fail(c, SLH_EHIP, "hipFree: %s", hipGetErrorString(e));
    b.p = nullptr;
    b.bytes = 0;
  }
  hipError_t e = hipMalloc(&b.p, bytes);
  if (e != hipSuccess) {
    b.p = nullptr;
    return fail(c, SLH_ENOMEM, "hipMalloc(%zu): %s", bytes, hipGetErrorString(e));
  }
  b.bytes = bytes;
  return SLH_OK;
}

// pinned host buffer of at least `bytes`
int ensure_pinned(slh_ctx* c, size_t bytes) {
  if (c->pin_bytes >= bytes) return SLH_OK;
  if (c->pin) (void)hipHostFree(c->pin);
  c->pin = nullptr;
  c->pin_bytes = 0;
  const size_t b = std::max<size_t>(bytes, 256);
  const hipError_t e = hipHostMalloc(&c->pin, b, hipHostMallocDefault);
  if (e != hipSuccess) {
    c->pin = nullptr;
    return fail(c, SLH_ENOMEM, "hipHostMalloc(%zu): %s", b, hipGetErrorString(e));
  }
  c->pin_bytes = b;
  return SLH_OK;
}

// Wait for the work enqueued so far on the context stream by spinning on an
// event (a woken-up stream synchronisation costs tens of microseconds).
int wait_stream(slh_ctx* c) {
  hipError_t e = hipEventRecord(c->ev_host, c->stream);
  if (e != hipSuccess) return fail(c, SLH_EHIP, "hipEventRecord: %s", hipGetErrorString(e));
  while ((e = hipEventQuery(c->ev_host)) == hipErrorNotReady) {
  }
  if (e != hipSuccess) return fail(c, SLH_EHIP, "hipEventQuery: %s", hipGetErrorString(e));
  return SLH_OK;
}

#define ENSURE(c, b, bytes)                   \
  do {                                        \
    int rc_ = ensure((c), (b), (bytes));      \
    if (rc_ != SLH_OK) return rc_;            \
  } while (0)

template <class T>
T* P(DevBuf& b) {
  return (T*)b.p;
}

// Timing events only measure: no system-scope fence (cache writeback) when they
// complete, which would otherwise slow the kernels that follow them; readers
// synchronise the stream before reading them.
int make_events(slh_ctx* c, int n_fused) {
  const unsigned fl = hipEventDisableSystemFence;
  if (!c->ev_made) {
    // events made before a failed creation are kept (and destroyed with the context)
    for (auto& e : c->ev)
      if (!e) HIP_TRY(c, hipEventCreateWithFlags(&e, fl));
    c->ev_made = true;
  }
  while ((int)c->ev_fb.size() < n_fused) {
    hipEvent_t a = nullptr, b = nullptr;
    hipError_t e = hipEventCreateWithFlags(&a, fl);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&b, fl);
    if (e != hipSuccess) {
      if (a) (void)hipEventDestroy(a);
      return fail(c, SLH_EHIP, "hipEventCreateWithFlags: %s", hipGetErrorString(e));
    }
    c->ev_fb.push_back(a);
    c->ev_fa.push_back(b);
  }
  return SLH_OK;
}

void drop_graph(slh_ctx* c) {
  if (c->lz_exec) {
    (void)hipGraphExecDestroy(c->lz_exec);
    c->lz_exec = nullptr;
  }
  c->lz_key.clear();
}

int64_t window_len(const slh_ctx* c) { return c->L > 0 ? c->L : c->N; }

int check_x(slh_ctx* c, const void* X, int32_t dtype, int64_t ldx) {
  if (!X) return fail(c, SLH_EINVAL, "X is NULL");
  if (dtype != SLH_BF16 && dtype != SLH_F32) return fail(c, SLH_EINVAL, "unknown x_dtype %d", dtype);
  if (ldx < c->D || ldx % 8 != 0)
    return fail(c, SLH_EINVAL, "ldx must be >= D and a multiple of 8 (got %lld)", (long long)ldx);
  if (((uintptr_t)X) % 16 != 0) return fail(c, SLH_EINVAL, "X must be 16-byte aligned");
  return SLH_OK;
}

// row norms (and the bf16 copy of fp32 X) for the given X
int prep_norms(slh_ctx* c, const void* X, int32_t dtype, int64_t ldx) {
  ENSURE(c, c->nrm2_fm, c->N * sizeof(double));
  ENSURE(c, c->nrm_x, c->N * sizeof(double));
  ENSURE(c, c->inv_x, c->N * sizeof(double));
  ENSURE(c, c->rowscale, c->N * sizeof(float));
  uint16_t* xb = nullptr;
  if (dtype == SLH_F32) {
    ENSURE(c, c->Xb, (size_t)c->N * c->D * sizeof(uint16_t));
    xb = P<uint16_t>(c->Xb);
  }
  HIP_TRY(c, launch_rownorm(X, dtype == SLH_BF16 ? 0 : 1, ldx, c->N, (int)c->D, (int)c->m,
                            c->gauss, P<double>(c->nrm2_fm), P<double>(c->nrm_x),
                            P<double>(c->inv_x), P<float>(c->rowscale), xb, c->stream));
  c->norms_of = X;
  c->norms_dtype = dtype;
  c->norms_ldx = ldx;
  return SLH_OK;
}

bool norms_match(const slh_ctx* c, const void* X, int32_t dtype, int64_t ldx) {
  return c->norms_of == X && c->norms_dtype == dtype && c->norms_ldx == ldx;
}

void forget_norms(slh_ctx* c) {
  c->norms_of = nullptr;
  c->norms_dtype = -1;
  c->norms_ldx = -1;
  c->norms_fresh = false;
}

int upload_routing(slh_ctx* c) {
  ENSURE(c, c->winlist, std::max<size_t>(1, c->winlist_h.size()) * sizeof(int));
  ENSURE(c, c->route, std::max<size_t>(1, c->route_h.size()));
  if (!c->winlist_h.empty())
    HIP_TRY(c, hipMemcpyAsync(c->winlist.p, c->winlist_h.data(), c->winlist_h.size() * sizeof(int),
                              hipMemcpyHostToDevice, c->stream));
  HIP_TRY(c, hipMemcpyAsync(c->route.p, c->route_h.data(), c->route_h.size(),
                            hipMemcpyHostToDevice, c->stream));
  // the host vectors must stay alive until the copies complete
  HIP_TRY(c, hipStreamSynchronize(c->stream));
  c->routing_on_device = true;
  return SLH_OK;
}

int ensure_routing(slh_ctx* c) {
  return c->routing_on_device ? SLH_OK : upload_routing(c);
}

void route_all_spectral(slh_ctx* c) {
  c->route_h.assign((size_t)c->n_win, 1);
  c->winlist_h.resize((size_t)c->n_win);
  for (int64_t w = 0; w < c->n_win; ++w) c->winlist_h[(size_t)w] = (int)w;
  c->n_act = (int)c->n_win;
  c->chunk_k = 1;
  c->routing_on_device = false;
}

// Exact target length: the spectral windows share B = target - (chunk-window
// macro-tokens) - (preserved tokens), floor(B / n) each and one more for the
// first B mod n (window order).  Returns false if some budget would leave [1, L].
bool target_budgets(const slh_ctx* c, std::vector<int>& tw) {
  const int64_t L = window_len(c);
  tw.assign((size_t)c->n_win, 0);
  int64_t chunk = 0, ns = 0;
  for (int64_t w = 0; w < c->n_win; ++w) {
    if (c->route_h[(size_t)w]) ++ns;
    else chunk += (L + c->chunk_k - 1) / c->chunk_k;
  }
  const int64_t B = c->target_len - chunk - c->keep_last;
  if (ns == 0) return B == 0;
  if (B < ns || B > ns * L) return false;
  int64_t a = 0;
  for (int64_t w = 0; w < c->n_win; ++w)
    if (c->route_h[(size_t)w]) tw[(size_t)w] = (int)(B / ns + (a++ < B % ns ? 1 : 0));
  return true;
}

int64_t capacity(const slh_ctx* c) {
  const int64_t L = window_len(c);
  const int64_t per_spec = std::min<int64_t>(L, (int64_t)1 << c->bits);
  std::vector<int> tw;
  const bool tg = c->target_len > 0 && target_budgets(c, tw);
  int64_t cap = 0;
  for (int64_t w = 0; w < c->n_win; ++w)
    cap += c->route_h[(size_t)w] ? std::max<int64_t>(per_spec, tg ? tw[(size_t)w] : 0)
                                 : (L + c->chunk_k - 1) / c->chunk_k;
  return cap + c->keep_last;
}

// The captured body of slh_lanczos (graph mode): the step sequence, Eigh(T)
// and the Ritz coordinates, in one stream (a forked branch for the last beta,
// which T does not use, made the replay about 0.1 ms slower: the branches are
// synchronised across queues).  Returns the first launch error (the capture
// is ended by the caller in every case).
hipError_t launch_lanczos_graph_body(slh_ctx* c, const LanczosWS& w, const double* q1act, int na,
                                 int n_it, int L, bool res) {
  hipError_t e = res ? launch_lanczos_resident(w, q1act, P<unsigned>(c->lz_bar), c->n_cu,
                                               c->cap_stream)
                     : launch_lanczos(w, q1act, c->cap_stream);
  if (e == hipSuccess)
    e = launch_eigh_ritz(w.alpha, w.beta, w.neff, na, n_it, c->r, P<double>(c->theta),
                         P<double>(c->Seig), w.Q, L, w.ldq, P<double>(c->Z), c->n_cu, c->cap_stream);
  return e;
}

}  // namespace

// ---------------------------------------------------------------------------
// ABI
// ---------------------------------------------------------------------------
extern "C" {

int slh_gen_params(uint64_t seed, int64_t D, int64_t m, int32_t r, int32_t bits,
                   uint16_t* W_out, float* psi_out, double* R_out) {
  if (D <= 0 || m <= 0 || r <= 0 || bits <= 0) return SLH_EINVAL;
  if (W_out) {
    const double std_w = 1.0 / std::sqrt(std::sqrt((double)D));
    const int64_t total = D * m;
    std::vector<double> nrm((size_t)std::min<int64_t>(total, 1 << 20) + 1);
    // stream W in chunks of whole Philox blocks
    for (int64_t e0 = 0; e0 < total; e0 += (1 << 20)) {
      const int64_t cnt = std::min<int64_t>(1 << 20, total - e0);
      const int64_t nb0 = e0 / 2, nb = (cnt + 1) / 2;
      for (int64_t b = 0; b < nb; ++b) {
        uint32_t w[4];
        philox_block(seed, STREAM_W, 0, (uint64_t)(nb0 + b), w);
        const double ua = u53(w[0], w[1]), ub = u53(w[2], w[3]);
        const double rad = std::sqrt(-2.0 * std::log(1.0 - ua));
        const double ang = (2.0 * M_PI) * ub;
        nrm[(size_t)(2 * b)] = rad * std::cos(ang);
        nrm[(size_t)(2 * b + 1)] = rad * std::sin(ang);
      }
      for (int64_t e = 0; e < cnt; ++e) W_out[e0 + e] = bf16_rne((float)(nrm[(size_t)e] * std_w));
    }
  }
  if (psi_out) {
    for (int64_t j = 0; j < m; ++j) {
      uint32_t w[4];
      philox_block(seed, STREAM_PSI, 0, (uint64_t)j, w);
      psi_out[j] = (float)((2.0 * M_PI) * u53(w[0], w[1]));
    }
  }
  if (R_out) gen_normals(seed, STREAM_R, 0, (int64_t)r * bits, R_out);
  return SLH_OK;
}

int slh_gen_start(uint64_t seed, int64_t window, int64_t n, double* q_out) {
  if (n <= 0 || !q_out || window < 0) return SLH_EINVAL;
  gen_normals(seed, STREAM_Q1, (uint32_t)window, n, q_out);
  double s = 0.0;
  for (int64_t i = 0; i < n; ++i) s += q_out[i] * q_out[i];
  const double nrm = std::sqrt(s);
  for (int64_t i = 0; i < n; ++i) q_out[i] /= nrm;
  return SLH_OK;
}

const char* slh_last_error(const slh_ctx* c) { return c ? c->err.c_str() : "no context"; }

int slh_create(slh_ctx** out, int64_t N, int64_t D, int64_t m, int32_t r, int32_t bits,
               uint64_t seed) {
  if (!out) return SLH_EINVAL;
  *out = nullptr;
  if (N < 2 || N > (int64_t)1 << 30) return SLH_EINVAL;
  if (D < 8 || D % 8 != 0 || D > 32768) return SLH_EINVAL;
  if (m < 256 || m > 2048 || m % 256 != 0) return SLH_EINVAL;
  if (r < 1 || r > 128) return SLH_EINVAL;
  if (bits < 1 || bits > 16) return SLH_EINVAL;
  slh_ctx* c = new (std::nothrow) slh_ctx();
  if (!c) return SLH_ENOMEM;
  c->N = N;
  c->Ntot = N;
  c->D = D;
  c->m = m;
  c->r = r;
  c->bits = bits;
  c->seed = seed;
  c->n_win = 1;
  if (hipGetDevice(&c->device) != hipSuccess) {
    delete c;
    return SLH_EHIP;
  }
  hipDeviceProp_t prop;
  if (hipGetDeviceProperties(&prop, c->device) == hipSuccess) c->n_cu = prop.multiProcessorCount;
  route_all_spectral(c);
  // parameters: W transposed to [m][Dp] for K-contiguous MFMA operands, K padded
  // with zeros to a multiple of 64 so the GEMM's K tail needs no masking
  const int64_t Dp = ((D + 63) / 64) * 64;
  std::vector<uint16_t> W((size_t)(D * m)), Wt((size_t)(Dp * m), 0);
  std::vector<float> psi((size_t)m);
  std::vector<double> R((size_t)r * bits);
  slh_gen_params(seed, D, m, r, bits, W.data(), psi.data(), R.data());
  for (int64_t k = 0; k < D; ++k)
    for (int64_t j = 0; j < m; ++j) Wt[(size_t)(j * Dp + k)] = W[(size_t)(k * m + j)];
  int rc = SLH_OK;
  if ((rc = ensure(c, c->Wt, Wt.size() * 2)) || (rc = ensure(c, c->psi, psi.size() * 4)) ||
      (rc = ensure(c, c->R, R.size() * 8))) {
    slh_destroy(c);
    return rc;
  }
  if (hipMemcpy(c->Wt.p, Wt.data(), Wt.size() * 2, hipMemcpyHostToDevice) != hipSuccess ||
      hipMemcpy(c->psi.p, psi.data(), psi.size() * 4, hipMemcpyHostToDevice) != hipSuccess ||
      hipMemcpy(c->R.p, R.data(), R.size() * 8, hipMemcpyHostToDevice) != hipSuccess) {
    slh_destroy(c);
    return SLH_EHIP;
  }
  if (hipStreamCreateWithFlags(&c->cap_stream, hipStreamNonBlocking) != hipSuccess ||
      hipEventCreateWithFlags(&c->ev_host, hipEventDisableTiming) != hipSuccess ||
      hipEventCreateWithFlags(&c->mq_ev[0], hipEventDisableTiming) != hipSuccess ||
      hipEventCreateWithFlags(&c->mq_ev[1], hipEventDisableTiming) != hipSuccess ||
      hipHostMalloc((void**)&c->mq_pin, 4 * sizeof(unsigned), hipHostMallocDefault) != hipSuccess) {
    slh_destroy(c);
    return SLH_EHIP;
  }
  *out = c;
  return SLH_OK;
}

void slh_destroy(slh_ctx* c) {
  if (!c) return;
  if (c->mq_head != c->mq_tail) (void)hipStreamSynchronize(c->stream);   // merges still in flight
  drop_graph(c);
  DevBuf* bufs[] = {&c->Wt, &c->psi, &c->R, &c->q1all, &c->q1act, &c->winlist, &c->route,
                    &c->nrm2_fm, &c->nrm_x, &c->inv_x, &c->rowscale, &c->Xb, &c->Phi, &c->Q, &c->T,
                    &c->Apart, &c->Z1, &c->Spart, &c->Zs, &c->H2part, &c->H2,
                    &c->alpha, &c->beta, &c->neff, &c->stop, &c->amax, &c->theta, &c->Seig, &c->Z,
                    &c->proj, &c->codes, &c->keyA, &c->keyB, &c->valA, &c->valB, &c->tmpi,
                    &c->segid, &c->segk, &c->sval, &c->sloc, &c->mw, &c->wbase, &c->sseg,
                    &c->Mtot, &c->part, &c->part_seg, &c->part_cnt, &c->part_nsum,
                    &c->part_end, &c->rpart, &c->scores, &c->rsu, &c->lz_bar, &c->nm_part, &c->nm_csum, &c->rowsum, &c->dg_counts,
                    &c->dg_energy, &c->dg_rowsq, &c->dg_tiles, &c->mg_pre, &c->posv, &c->tg_scr,
                    &c->tg_tw};
  for (DevBuf* b : bufs)
    if (b->p) (void)hipFree(b->p);
  if (c->cap_stream) (void)hipStreamDestroy(c->cap_stream);
  if (c->ev_host) (void)hipEventDestroy(c->ev_host);
  if (c->pin) (void)hipHostFree(c->pin);
  for (auto& e : c->mq_ev)
    if (e) (void)hipEventDestroy(e);
  if (c->mq_pin) (void)hipHostFree(c->mq_pin);

  for (auto& e : c->ev)
    if (e) (void)hipEventDestroy(e);
  for (auto& e : c->ev_fb) (void)hipEventDestroy(e);
  for (auto& e : c->ev_fa) (void)hipEventDestroy(e);
  delete c;
}

int slh_set_option(slh_ctx* c, int32_t key, double v) {
  if (!c) return SLH_EINVAL;
  switch (key) {
    case SLH_OPT_KERNEL:
      if (v != 0.0 && v != 1.0) return fail(c, SLH_EINVAL, "KERNEL must be 0 or 1");
      c->gauss = (int)v;
      forget_norms(c);
      break;
    case SLH_OPT_WINDOW_LEN: {
      const int64_t L = (int64_t)v;
      if ((double)L != v || L < 0) return fail(c, SLH_EINVAL, "WINDOW_LEN must be a non-negative integer");
      const int64_t Le = L ? L : c->N;
      if (Le < 2 || c->N % Le != 0) return fail(c, SLH_EINVAL, "N must be a multiple of WINDOW_LEN >= 2");
      c->L = L;
      c->n_win = c->N / Le;
      route_all_spectral(c);
      c->routed = false;
      drop_graph(c);
      break;
    }
    case SLH_OPT_POS_MODE:
      if (v != 0.0 && v != 1.0) return fail(c, SLH_EINVAL, "POS_MODE must be 0 or 1");
      c->compact = (int)v;
      break;
    case SLH_OPT_BREAKDOWN_TOL:
      if (!(v >= 0.0)) return fail(c, SLH_EINVAL, "BREAKDOWN_TOL must be >= 0");
      c->tol = v;
      drop_graph(c);
      break;
    case SLH_OPT_TIMING:
      if (v != 0.0 && v != 1.0) return fail(c, SLH_EINVAL, "TIMING must be 0 or 1");
      c->timing = (int)v;
      drop_graph(c);
      if (c->timing && make_events(c, 0)) return SLH_EHIP;
      break;
    case SLH_OPT_KEEP_LAST: {
      const int64_t K = (int64_t)v;
      if ((double)K != v || K < 0 || c->Ntot - K < 2)
        return fail(c, SLH_EINVAL, "KEEP_LAST must be an integer in [0, N - 2]");
      const int64_t Nc = c->Ntot - K;
      const int64_t Le = c->L ? c->L : Nc;
      if (Nc % Le != 0)
        return fail(c, SLH_EINVAL, "N - KEEP_LAST must be a multiple of WINDOW_LEN");
      c->keep_last = K;
      c->N = Nc;
      c->n_win = Nc / Le;
      forget_norms(c);
      c->q1_L = -1;
      route_all_spectral(c);
      c->routed = false;
      drop_graph(c);
      break;
    }
    case SLH_OPT_TARGET_LEN: {
      const int64_t T = (int64_t)v;
      if ((double)T != v || T < 0 || T > c->Ntot)
        return fail(c, SLH_EINVAL, "TARGET_LEN must be an integer in [0, N]");
      c->target_len = T;
      break;
    }
    case SLH_OPT_POS_SCHEME:
      if (v != 0.0 && v != 1.0 && v != 2.0) return fail(c, SLH_EINVAL, "POS_SCHEME must be 0, 1 or 2");
      c->pos_scheme = (int)v;
      break;
    case SLH_OPT_NORMALIZE:
      if (v != 0.0 && v != 1.0) return fail(c, SLH_EINVAL, "NORMALIZE must be 0 or 1");
      c->normalize = (int)v;
      break;
    case SLH_OPT_SHORT_WINDOWS:
      if (v != 0.0 && v != 1.0) return fail(c, SLH_EINVAL, "SHORT_WINDOWS must be 0 or 1");
      c->short_win = (int)v;
      break;
    case SLH_OPT_RESIDENT:
      if (v != 0.0 && v != 1.0) return fail(c, SLH_EINVAL, "RESIDENT must be 0 or 1");
      c->resident = (int)v;
      break;
    case SLH_OPT_WAIT_POLLS:
      if (!(v >= 0.0 && v <= 2147483647.0) || v != (double)(int)v)
        return fail(c, SLH_EINVAL, "WAIT_POLLS must be an integer in [0, 2^31)");
      c->wait_polls = (int)v;
      break;
    default:
      return fail(c, SLH_EINVAL, "unknown option %d", key);
  }
  c->stage = 0;
  c->merged = 0;
  return SLH_OK;
}

int slh_set_stream(slh_ctx* c, void* s) {
  if (!c) return SLH_EINVAL;
  c->stream = (hipStream_t)s;
  return SLH_OK;
}

int64_t slh_num_windows(const slh_ctx* c) { return c ? c->n_win : 0; }
int64_t slh_num_spectral(const slh_ctx* c) { return c ? c->n_act : 0; }
int64_t slh_merge_capacity(const slh_ctx* c) { return c ? capacity(c) : 0; }

int slh_route(slh_ctx* c, const void* X, int32_t dtype, int64_t ldx, double rho, double tau,
              uint8_t* route_out, double* scores_out) {
  if (!c) return SLH_EINVAL;
  int rc = check_x(c, X, dtype, ldx);
  if (rc) return rc;
  if (!(rho > 0.0)) return fail(c, SLH_EINVAL, "rho must be > 0");
  const int64_t L = window_len(c);
  ENSURE(c, c->rpart, (size_t)c->n_win * route_slices((int)c->D) * 2 * sizeof(double));
  ENSURE(c, c->scores, (size_t)c->n_win * sizeof(double));
  const int G = route_norm_groups((int)L, (int)c->D);
  if (G > 0) {
    // one read of X for the row norms and the scores
    ENSURE(c, c->nrm2_fm, c->N * sizeof(double));
    ENSURE(c, c->nrm_x, c->N * sizeof(double));
    ENSURE(c, c->inv_x, c->N * sizeof(double));
    ENSURE(c, c->rowscale, c->N * sizeof(float));
    uint16_t* xb = nullptr;
    if (dtype == SLH_F32) {
      ENSURE(c, c->Xb, (size_t)c->N * c->D * sizeof(uint16_t));
      xb = P<uint16_t>(c->Xb);
    }
    ENSURE(c, c->rsu, (size_t)c->n_win * G * 2 * c->D * sizeof(double));
    HIP_TRY(c, launch_route_norm_scores(X, dtype == SLH_BF16 ? 0 : 1, ldx, (int)c->n_win, (int)L,
                                        (int)c->D, (int)c->m, c->gauss, P<double>(c->nrm2_fm),
                                        P<double>(c->nrm_x), P<double>(c->inv_x),
                                        P<float>(c->rowscale), xb, P<double>(c->rsu),
                                        P<double>(c->rpart), P<double>(c->scores), c->stream));
    c->norms_of = X;
    c->norms_dtype = dtype;
    c->norms_ldx = ldx;
  } else {
    if ((rc = prep_norms(c, X, dtype, ldx))) return rc;
    HIP_TRY(c, launch_route_scores(X, dtype == SLH_BF16 ? 0 : 1, ldx, P<double>(c->inv_x),
                                   (int)c->n_win, (int)L, (int)c->D, P<double>(c->rpart),
                                   P<double>(c->scores), c->stream));
  }
  std::vector<double> sc((size_t)c->n_win);
  if ((rc = ensure_pinned(c, sc.size() * sizeof(double)))) return rc;
  HIP_TRY(c, hipMemcpyAsync(c->pin, c->scores.p, sc.size() * sizeof(double),
                            hipMemcpyDeviceToHost, c->stream));
  if ((rc = wait_stream(c))) return rc;
  std::memcpy(sc.data(), c->pin, sc.size() * sizeof(double));
  // tau(rho): 0.70 at rho <= 2, linear in log2(rho) through 0.60 at 8 and 0.55 at 16
  double t = tau;
  if (!(tau >= 0.0)) {
    const double l2 = std::log2(rho);
    if (rho <= 2.0) t = 0.70;
    else if (rho <= 8.0) t = 0.70 - 0.05 * (l2 - 1.0);
    else if (rho < 16.0) t = 0.60 - 0.05 * (l2 - 3.0);
    else t = 0.55;
  }
  c->route_h.assign((size_t)c->n_win, 0);
  c->winlist_h.clear();
  for (int64_t w = 0; w < c->n_win; ++w) {
    bool spectral;
    if (rho >= 16.0) spectral = true;
    else if (L <= 4) spectral = false;
    else spectral = sc[(size_t)w] >= t;
    c->route_h[(size_t)w] = spectral ? 1 : 0;
    if (spectral) c->winlist_h.push_back((int)w);
  }
  c->n_act = (int)c->winlist_h.size();
  c->chunk_k = std::max(1, (int)std::nearbyint(rho));   // round half to even
  c->norms_fresh = true;
  c->routed = true;
  c->routing_on_device = false;
  drop_graph(c);
  if ((rc = upload_routing(c))) return rc;
  if (route_out) std::memcpy(route_out, c->route_h.data(), c->route_h.size());
  if (scores_out) std::memcpy(scores_out, sc.data(), sc.size() * sizeof(double));
  c->stage = 0;
  c->merged = 0;
  return SLH_OK;
}

int slh_feature_map(slh_ctx* c, const void* X, int32_t dtype, int64_t ldx) {
  if (!c) return SLH_EINVAL;
  int rc = check_x(c, X, dtype, ldx);
  if (rc) return rc;
  if ((rc = ensure_routing(c))) return rc;
  if (!(c->norms_fresh && norms_match(c, X, dtype, ldx)))
    if ((rc = prep_norms(c, X, dtype, ldx))) return rc;
  c->norms_fresh = false;
  const int64_t L = window_len(c);
  const int64_t rows = (int64_t)c->n_act * L;
  ENSURE(c, c->Phi, (size_t)std::max<int64_t>(rows, 1) * c->m * sizeof(float));
  FeatmapArgs a;
  a.X = dtype == SLH_F32 ? P<uint16_t>(c->Xb) : (const uint16_t*)X;
  a.ldx = dtype == SLH_F32 ? c->D : ldx;
  a.Wt = P<uint16_t>(c->Wt);
  a.psi = P<float>(c->psi);
  a.rowscale = P<float>(c->rowscale);
  a.Phi = P<float>(c->Phi);
  a.winlist = (c->n_act == c->n_win) ? nullptr : P<int>(c->winlist);
  a.n_rows = rows;
  a.L = L;
  a.D = (int)c->D;
  a.ldw = (int)(((c->D + 63) / 64) * 64);
  a.m = (int)c->m;
  HIP_TRY(c, launch_featmap(a, c->n_cu, c->stream, c->timing ? c->ev[0] : nullptr,
                            c->timing ? c->ev[1] : nullptr));
  if (c->normalize && c->n_act > 0) {
    const int G = normalise_groups(c->n_act, (int)L, (int)c->m, c->n_cu);
    ENSURE(c, c->nm_part, (size_t)c->n_act * G * c->m * 8);
    ENSURE(c, c->nm_csum, (size_t)c->n_act * c->m * 8);
    ENSURE(c, c->rowsum, (size_t)rows * 8);
    if (c->timing) HIP_TRY(c, hipEventRecord(c->ev[9], c->stream));
    HIP_TRY(c, launch_normalise(P<float>(c->Phi), c->n_act, (int)L, (int)c->m, G,
                                P<double>(c->nm_part), P<double>(c->nm_csum),
                                P<double>(c->rowsum), c->stream));
    if (c->timing) HIP_TRY(c, hipEventRecord(c->ev[10], c->stream));
    c->norm_timed = c->timing;
  }
  c->stage = 1;
  c->merged = 0;
  return SLH_OK;
}

int slh_lanczos(slh_ctx* c, int32_t n_it, double* ritz_out, int32_t* iters_out) {
  if (!c) return SLH_EINVAL;
  if (c->stage < 1) return fail(c, SLH_ESTATE, "slh_lanczos before slh_feature_map");
  const int64_t L = window_len(c);
  if (n_it < c->r || n_it > std::min<int64_t>(L, 256))
    return fail(c, SLH_EINVAL, "need r <= n_it <= min(L, 256) (n_it=%d, r=%d, L=%lld)", n_it,
                c->r, (long long)L);
  const int na = c->n_act;
  c->n_it = n_it;
  if (na > 0) {
    // start vectors of the spectral windows
    if (c->q1_L != L) {
      ENSURE(c, c->q1all, (size_t)c->N * sizeof(double));
      std::vector<double> q((size_t)c->N);
      for (int64_t w = 0; w < c->n_win; ++w) slh_gen_start(c->seed, w, L, q.data() + w * L);
      HIP_TRY(c, hipMemcpy(c->q1all.p, q.data(), q.size() * sizeof(double), hipMemcpyHostToDevice));
      c->q1_L = L;
    }
    const double* q1act = P<double>(c->q1all);
    if (na != c->n_win) {
      ENSURE(c, c->q1act, (size_t)na * L * sizeof(double));
      HIP_TRY(c, launch_gather_windows(P<double>(c->q1act), P<double>(c->q1all), P<int>(c->winlist),
                                       L, na, c->stream));
      q1act = P<double>(c->q1act);
    }
    if (c->short_win && local_supported((int)L, n_it, c->r)) {
      // short windows: Lanczos, Eigh and Ritz of each window in one wavefront
      ENSURE(c, c->Q, (size_t)na * (n_it + 1) * L * 8);
      ENSURE(c, c->alpha, (size_t)na * n_it * 8);
      ENSURE(c, c->beta, (size_t)na * n_it * 8);
      ENSURE(c, c->neff, (size_t)na * 4);
      ENSURE(c, c->theta, (size_t)na * c->r * 8);
      ENSURE(c, c->Z, (size_t)na * L * c->r * 8);
      if (c->timing) HIP_TRY(c, hipEventRecord(c->ev[2], c->stream));
      HIP_TRY(c, launch_local(P<float>(c->Phi), na, (int)c->m, (int)L, n_it, c->r, c->tol, q1act,
                              P<double>(c->Q), P<double>(c->alpha), P<double>(c->beta),
                              P<int>(c->neff), P<double>(c->theta), P<double>(c->Z), c->stream));
      if (c->timing) {
        HIP_TRY(c, hipEventRecord(c->ev[3], c->stream));
        HIP_TRY(c, hipEventRecord(c->ev[4], c->stream));
      }
      c->fused_timed = 0;
      c->passes_timed = 0;
      c->lz_w_valid = false;
      c->lz_res = false;
    } else {
      LanczosWS w;
      memset(&w, 0, sizeof w);      // the graph key compares the bytes
      w.n_act = na;
      w.L = (int)L;
      w.m = (int)c->m;
      w.n_it = n_it;
      w.ldq = n_it + 1;
      w.tol = c->tol;
      w.spin = c->wait_polls;
      // chunks of 16 rows per block of the pass: one chunk per block while the
      // blocks fit two per CU (all resident at once); beyond that, about one
      // block per CU, each streaming its chunks with the next in flight (the
      // current one staged in LDS, 16 m floats, so such a block runs alone on
      // its CU)
      {
        const int64_t chunks = (int64_t)na * ((L + 15) / 16);
        const int64_t ncu = std::max(1, c->n_cu);
        w.NCH = chunks <= 2 * ncu ? 1 : (int)((chunks + ncu - 1) / ncu);
        w.G3 = (int)((L + 16 * w.NCH - 1) / (16 * w.NCH));
      }
      const size_t hs = (size_t)w.ldq + 1;
      ENSURE(c, c->Q, (size_t)na * w.ldq * L * 8);
      ENSURE(c, c->T, (size_t)na * w.ldq * c->m * 8);
      // |t|^2 partials: m / 16 per window, or one per block of the resident kernel
      ENSURE(c, c->Apart, (size_t)na * std::max<int64_t>(c->m / 16, c->n_cu) * 8);
      ENSURE(c, c->Z1, (size_t)na * L * 8);
      ENSURE(c, c->Spart, (size_t)na * w.G3 * c->m * 8);
      ENSURE(c, c->Zs, (size_t)na * 2 * L * 8);
      ENSURE(c, c->H2part, (size_t)na * w.G3 * hs * 8);
      ENSURE(c, c->H2, (size_t)na * hs * 8);
      ENSURE(c, c->alpha, (size_t)na * n_it * 8);
      ENSURE(c, c->beta, (size_t)na * n_it * 8);
      ENSURE(c, c->neff, (size_t)na * 4);
      ENSURE(c, c->stop, (size_t)na * 4);
      ENSURE(c, c->amax, (size_t)na * 2 * 8);
      ENSURE(c, c->theta, (size_t)na * c->r * 8);
      ENSURE(c, c->Seig, (size_t)na * n_it * c->r * 8);
      ENSURE(c, c->Z, (size_t)na * L * c->r * 8);
      w.Phi = P<float>(c->Phi);
      w.Q = P<double>(c->Q);
      w.T = P<double>(c->T);
      w.Apart = P<double>(c->Apart);
      w.Z1 = P<double>(c->Z1);
      w.Spart = P<double>(c->Spart);
      w.Zs = P<double>(c->Zs);
      w.H2part = P<double>(c->H2part);
      w.H2 = P<double>(c->H2);
      w.alpha = P<double>(c->alpha);
      w.beta = P<double>(c->beta);
      w.neff = P<int>(c->neff);
      w.stop = P<int>(c->stop);
      w.amax = P<double>(c->amax);
      // one window whose Phi fits in the register files: the resident kernel
      const bool res = c->resident && lanczos_resident_ok(w, c->n_cu);
      (void)hipGetLastError();
      if (res) ENSURE(c, c->lz_bar, lanczos_resident_bar_words(c->n_cu) * sizeof(unsigned));
      if (c->timing) {
        // timing: launch the step sequence directly so that every pass over Phi
        // can be bracketed by events (events inside a captured graph cannot be timed)
        int rc_ev = make_events(c, n_it);
        if (rc_ev) return rc_ev;
        HIP_TRY(c, hipEventRecord(c->ev[2], c->stream));
        if (res)
          HIP_TRY(c, launch_lanczos_resident(w, q1act, P<unsigned>(c->lz_bar), c->n_cu, c->stream,
                                             c->ev_fb[0], c->ev_fa[0]));
        else
          HIP_TRY(c, launch_lanczos(w, q1act, c->stream, c->ev_fb.data(), c->ev_fa.data()));
        HIP_TRY(c, hipEventRecord(c->ev[3], c->stream));
        HIP_TRY(c, launch_eigh_ritz(w.alpha, w.beta, w.neff, na, n_it, c->r, P<double>(c->theta),
                                    P<double>(c->Seig), w.Q, (int)L, w.ldq, P<double>(c->Z),
                                    c->n_cu, c->stream));
        HIP_TRY(c, hipEventRecord(c->ev[4], c->stream));
      } else if (res) {
        // the resident path is four kernels, launched directly: the end of a
        // graph costs a gap before the stream's next kernel
        HIP_TRY(c, launch_lanczos_resident(w, q1act, P<unsigned>(c->lz_bar), c->n_cu, c->stream,
                                           nullptr, nullptr));
        HIP_TRY(c, launch_eigh_ritz(w.alpha, w.beta, w.neff, na, n_it, c->r, P<double>(c->theta),
                                    P<double>(c->Seig), w.Q, (int)L, w.ldq, P<double>(c->Z),
                                    c->n_cu, c->stream));
      } else {
        // The step sequence, Eigh(T) and the Ritz coordinates are captured once
        // per configuration and replayed as one graph.
        std::string key((const char*)&w, sizeof w);
        key.append((const char*)&q1act, sizeof q1act);
        key.append(res ? "r" : "s");
        const void* outs[3] = {c->theta.p, c->Seig.p, c->Z.p};   // the eigensolve's outputs
        key.append((const char*)outs, sizeof outs);
        if (!c->lz_exec || c->lz_key != key) {
          drop_graph(c);
          hipGraph_t g = nullptr;
          HIP_TRY(c, hipStreamBeginCapture(c->cap_stream, hipStreamCaptureModeThreadLocal));
          hipError_t le = launch_lanczos_graph_body(c, w, q1act, na, n_it, (int)L, res);
          hipError_t ee = hipStreamEndCapture(c->cap_stream, &g);
          if (le != hipSuccess || ee != hipSuccess) {
            if (g) (void)hipGraphDestroy(g);
            return fail(c, SLH_EHIP, "Lanczos graph capture: %s / %s", hipGetErrorString(le),
                        hipGetErrorString(ee));
          }
          hipError_t ie = hipGraphInstantiate(&c->lz_exec, g, nullptr, nullptr, 0);
          (void)hipGraphDestroy(g);
          if (ie != hipSuccess) {
            c->lz_exec = nullptr;
            return fail(c, SLH_EHIP, "hipGraphInstantiate: %s", hipGetErrorString(ie));
          }
          c->lz_key = key;
        }
        HIP_TRY(c, hipGraphLaunch(c->lz_exec, c->stream));
      }
      c->fused_timed = c->timing ? (res ? 1 : n_it) : 0;
      c->passes_timed = c->timing ? n_it : 0;
      c->lz_w = w;
      c->lz_w_valid = true;
      c->lz_res = res;
    }
  }
  if ((ritz_out || iters_out) && na > 0) {
    if (ritz_out)
      HIP_TRY(c, hipMemcpyAsync(ritz_out, c->theta.p, (size_t)na * c->r * 8, hipMemcpyDeviceToHost,
                                c->stream));
    if (iters_out)
      HIP_TRY(c, hipMemcpyAsync(iters_out, c->neff.p, (size_t)na * 4, hipMemcpyDeviceToHost,
                                c->stream));
    HIP_TRY(c, hipStreamSynchronize(c->stream));
    if (c->lz_res) {
      unsigned ew = 0;
      HIP_TRY(c, hipMemcpy(&ew, P<unsigned>(c->lz_bar) + LZ_BAR_ERR, 4, hipMemcpyDeviceToHost));
      if (ew) return fail(c, SLH_EHIP, "Lanczos: a wait between blocks of the resident kernel timed out");
    }
  }
  c->stage = 2;
  c->merged = 0;
  c->t_loaded = 0;
  return SLH_OK;
}

int slh_eigh_ritz(slh_ctx* c, int32_t n_it, double* ritz_out, int32_t* iters_out) {
  if (!c) return SLH_EINVAL;
  const bool loaded = c->t_loaded == 7;
  if (!loaded && c->stage < 2)
    return fail(c, SLH_ESTATE, "slh_eigh_ritz needs slh_lanczos or slh_load of alpha, beta and Q");
  if (n_it != c->n_it)
    return fail(c, SLH_EINVAL, "n_it %d differs from the tridiagonal's order %d", n_it, c->n_it);
  const int64_t L = window_len(c);
  const int na = c->n_act;
  if (na > 0) {
    ENSURE(c, c->theta, (size_t)na * c->r * 8);
    ENSURE(c, c->Seig, (size_t)na * n_it * c->r * 8);
    ENSURE(c, c->Z, (size_t)na * L * c->r * 8);
    HIP_TRY(c, launch_eigh_ritz(P<double>(c->alpha), P<double>(c->beta), P<int>(c->neff), na,
                                n_it, c->r, P<double>(c->theta), P<double>(c->Seig),
                                P<double>(c->Q), (int)L, n_it + 1, P<double>(c->Z), c->n_cu,
                                c->stream));
    if (ritz_out)
      HIP_TRY(c, hipMemcpyAsync(ritz_out, c->theta.p, (size_t)na * c->r * 8, hipMemcpyDeviceToHost,
                                c->stream));
    if (iters_out)
      HIP_TRY(c, hipMemcpyAsync(iters_out, c->neff.p, (size_t)na * 4, hipMemcpyDeviceToHost,
                                c->stream));
    if (ritz_out || iters_out) HIP_TRY(c, hipStreamSynchronize(c->stream));
  }
  c->lz_w_valid = false;            // the pass replay needs a Lanczos run
  c->stage = 2;
  c->merged = 0;
  return SLH_OK;
}

int slh_simhash(slh_ctx* c, uint32_t* codes_out) {
  if (!c) return SLH_EINVAL;
  if (c->stage < 2) return fail(c, SLH_ESTATE, "slh_simhash before slh_lanczos");
  const int64_t L = window_len(c);
  const int na = c->n_act;
  ENSURE(c, c->codes, (size_t)c->Ntot * 4);
  ENSURE(c, c->proj, (size_t)std::max(na, 1) * L * c->bits * 8);
  if (c->timing) HIP_TRY(c, hipEventRecord(c->ev[5], c->stream));
  if (na != c->n_win || c->keep_last)
    HIP_TRY(c, launch_fill_u32(P<uint32_t>(c->codes), c->Ntot, 0xFFFFFFFFu, c->stream));
  if (na > 0)
    HIP_TRY(c, launch_simhash(P<double>(c->Z), P<double>(c->R),
                              na == c->n_win ? nullptr : P<int>(c->winlist), na, (int)L, c->r,
                              c->bits, P<uint32_t>(c->codes), P<double>(c->proj), c->stream));
  if (c->timing) HIP_TRY(c, hipEventRecord(c->ev[6], c->stream));
  if (codes_out)
    HIP_TRY(c, hipMemcpyAsync(codes_out, c->codes.p, (size_t)c->Ntot * 4, hipMemcpyDeviceToDevice,
                              c->stream));
  c->stage = 3;
  c->merged = 0;
  return SLH_OK;
}

int slh_merge_async(slh_ctx* c, const void* X, int32_t dtype, int64_t ldx, float* emb_out,
                    int32_t* pos_out, int32_t* tok2macro_out, int64_t cap) {
  if (!c) return SLH_EINVAL;
  if (c->stage < 3) return fail(c, SLH_ESTATE, "slh_merge before slh_simhash");
  if (c->mq_head - c->mq_tail >= 2)
    return fail(c, SLH_ESTATE, "two merges outstanding: slh_merge_wait first");
  int rc = check_x(c, X, dtype, ldx);
  if (rc) return rc;
  if (!emb_out || !pos_out) return fail(c, SLH_EINVAL, "NULL output");
  const int64_t need = capacity(c);
  if (cap < need) return fail(c, SLH_EINVAL, "cap %lld < required %lld", (long long)cap, (long long)need);
  if (!norms_match(c, X, dtype, ldx))
    if ((rc = prep_norms(c, X, dtype, ldx))) return rc;
  const int64_t L = window_len(c);
  const int64_t N = c->N;
  const int CH = 16;
  const int nch = merge_nchunks(N, CH);
  ENSURE(c, c->keyA, N * 4);
  ENSURE(c, c->keyB, N * 4);
  ENSURE(c, c->valA, N * 4);
  ENSURE(c, c->valB, N * 4);
  ENSURE(c, c->tmpi, N * 4);
  ENSURE(c, c->segid, N * 4);
  ENSURE(c, c->segk, N * 4);
  ENSURE(c, c->sval, N * 4);
  ENSURE(c, c->sloc, N * 4);
  ENSURE(c, c->sseg, N * 4);
  ENSURE(c, c->mw, c->n_win * 4);
  ENSURE(c, c->wbase, (c->n_win + 1) * 4);
  ENSURE(c, c->Mtot, 4);
  ENSURE(c, c->part, (size_t)2 * nch * c->D * 4);
  ENSURE(c, c->part_seg, (size_t)2 * nch * 4);
  ENSURE(c, c->part_cnt, (size_t)2 * nch * 4);
  ENSURE(c, c->part_nsum, (size_t)2 * nch * 8);
  ENSURE(c, c->part_end, (size_t)2 * nch * 4);
  ENSURE(c, c->codes, (size_t)N * 4);
  if ((rc = ensure_routing(c))) return rc;
  MergeWS w;
  w.n_win = (int)c->n_win;
  w.L = (int)L;
  w.bits = c->bits;
  w.chunk_k = c->chunk_k;
  w.compact = c->compact;
  w.D = (int)c->D;
  w.N = N;
  w.route = P<uint8_t>(c->route);
  w.codes = P<uint32_t>(c->codes);
  w.nrm_x = P<double>(c->nrm_x);
  w.keyA = P<uint32_t>(c->keyA);
  w.keyB = P<uint32_t>(c->keyB);
  w.valA = P<int>(c->valA);
  w.valB = P<int>(c->valB);
  w.tmpi = P<int>(c->tmpi);
  w.segid = P<int>(c->segid);
  w.segk = P<int>(c->segk);
  w.sval = P<int>(c->sval);
  w.sloc = P<int>(c->sloc);
  w.mw = P<int>(c->mw);
  w.wbase = P<int>(c->wbase);
  w.sseg = P<int>(c->sseg);
  w.Mtot = P<int>(c->Mtot);
  w.part = P<float>(c->part);
  w.part_seg = P<int>(c->part_seg);
  w.part_cnt = P<int>(c->part_cnt);
  w.part_nsum = P<double>(c->part_nsum);
  w.part_end = P<int>(c->part_end);
  w.CH = CH;
  w.scheme = c->pos_scheme;
  w.posv = nullptr;
  w.pre = nullptr;
  w.tw = nullptr;
  w.tg = nullptr;
  if (c->target_len > 0) {
    if (c->pos_scheme) return fail(c, SLH_EINVAL, "TARGET_LEN needs max positions (POS_SCHEME 0)");
    if (!target_budgets(c, c->tw_h))
      return fail(c, SLH_EINVAL, "TARGET_LEN %lld is not reachable with this routing",
                  (long long)c->target_len);
    ENSURE(c, c->tg_tw, (size_t)c->n_win * 4);
    ENSURE(c, c->tg_scr, (size_t)N * 4);
    ENSURE(c, c->mg_pre, (size_t)N * 8);
    if (c->tg_tw.p != c->tw_dev_p || c->tw_h != c->tw_dev_h) {   // budgets changed
      HIP_TRY(c, hipMemcpyAsync(c->tg_tw.p, c->tw_h.data(), (size_t)c->n_win * 4,
                                hipMemcpyHostToDevice, c->stream));
      c->tw_dev_h = c->tw_h;
      c->tw_dev_p = c->tg_tw.p;
    }
    w.tw = P<int>(c->tg_tw);
    w.tg = P<int>(c->tg_scr);
    w.pre = P<long long>(c->mg_pre);
  }
  if (w.scheme) {
    ENSURE(c, c->posv, (size_t)N * 4);
    ENSURE(c, c->mg_pre, (size_t)N * 8);
    w.posv = P<int>(c->posv);
    w.pre = P<long long>(c->mg_pre);
  }
  if (c->timing) HIP_TRY(c, hipEventRecord(c->ev[7], c->stream));
  HIP_TRY(c, launch_merge(w, X, dtype == SLH_BF16 ? 0 : 1, ldx, emb_out, pos_out, tok2macro_out,
                          c->stream));
  HIP_TRY(c, launch_merge_tail(X, dtype == SLH_BF16 ? 0 : 1, ldx, (int)c->D, N, (int)c->keep_last,
                               P<int>(c->Mtot), c->compact, emb_out, pos_out, tok2macro_out,
                               c->stream));
  if (c->timing) HIP_TRY(c, hipEventRecord(c->ev[8], c->stream));
  const int sl = (int)(c->mq_head & 1);
  HIP_TRY(c, launch_merge_report(P<int>(c->Mtot), c->lz_res ? P<unsigned>(c->lz_bar) + LZ_BAR_ERR : nullptr,
                                 c->mq_pin + 2 * sl, c->stream));
  HIP_TRY(c, hipEventRecord(c->mq_ev[sl], c->stream));
  c->mq_res[sl] = c->lz_res;
  c->mq_keep[sl] = (int)c->keep_last;
  ++c->mq_head;
  c->merged = 1;
  forget_norms(c);                  // the next prompt may reuse this buffer
  return SLH_OK;
}

int slh_merge_wait(slh_ctx* c, int64_t* M_out) {
  if (!c || !M_out) return SLH_EINVAL;
  if (c->mq_tail == c->mq_head) return fail(c, SLH_ESTATE, "slh_merge_wait with no merge outstanding");
  const int sl = (int)(c->mq_tail & 1);
  hipError_t e;
  while ((e = hipEventQuery(c->mq_ev[sl])) == hipErrorNotReady) {
  }
  ++c->mq_tail;
  if (e != hipSuccess) return fail(c, SLH_EHIP, "hipEventQuery: %s", hipGetErrorString(e));
  if (c->mq_res[sl] && c->mq_pin[2 * sl + 1] != 0)
    return fail(c, SLH_EHIP, "Lanczos: a wait between blocks of the resident kernel timed out");
  *M_out = (int64_t)(int)c->mq_pin[2 * sl] + c->mq_keep[sl];
  return SLH_OK;
}

int slh_merge(slh_ctx* c, const void* X, int32_t dtype, int64_t ldx, float* emb_out,
              int32_t* pos_out, int32_t* tok2macro_out, int64_t cap, int64_t* M_out) {
  if (!c) return SLH_EINVAL;
  if (!M_out) return fail(c, SLH_EINVAL, "NULL output");
  if (c->mq_head != c->mq_tail)
    return fail(c, SLH_ESTATE, "slh_merge while a merge from slh_merge_async is outstanding");
  const int rc = slh_merge_async(c, X, dtype, ldx, emb_out, pos_out, tok2macro_out, cap);
  if (rc) return rc;
  return slh_merge_wait(c, M_out);
}

int slh_spectral_energy(slh_ctx* c, double* out) {
  if (!c || !out) return SLH_EINVAL;
  if (c->stage < 2) return fail(c, SLH_ESTATE, "slh_spectral_energy before slh_lanczos");
  const int64_t L = window_len(c);
  const int na = c->n_act;
  if (na == 0) return SLH_OK;
  ENSURE(c, c->dg_rowsq, (size_t)na * L * 8);
  ENSURE(c, c->dg_energy, (size_t)na * 8);
  HIP_TRY(c, launch_energy(P<float>(c->Phi), P<double>(c->theta), na, (int)L, (int)c->m, c->r,
                           P<double>(c->dg_rowsq), P<double>(c->dg_energy), c->stream));
  HIP_TRY(c, hipMemcpyAsync(out, c->dg_energy.p, (size_t)na * 8, hipMemcpyDeviceToHost, c->stream));
  HIP_TRY(c, hipStreamSynchronize(c->stream));
  return SLH_OK;
}

int slh_bucket_purity(slh_ctx* c, const void* X, int32_t dtype, int64_t ldx, double thresh,
                      int64_t* counts_out) {
  if (!c || !counts_out) return SLH_EINVAL;
  if (!c->merged) return fail(c, SLH_ESTATE, "slh_bucket_purity before slh_merge");
  int rc = check_x(c, X, dtype, ldx);
  if (rc) return rc;
  if (!(thresh >= -1.0 && thresh <= 1.0)) return fail(c, SLH_EINVAL, "thresh must be in [-1, 1]");
  if ((rc = prep_norms(c, X, dtype, ldx))) return rc;
  forget_norms(c);
  const int64_t N = c->N, L = window_len(c);
  // tiles of 64 x 64 sorted positions that hold same-bucket pairs (spectral windows)
  std::vector<int> seg((size_t)N);
  HIP_TRY(c, hipStreamSynchronize(c->stream));
  HIP_TRY(c, hipMemcpy(seg.data(), c->sseg.p, (size_t)N * 4, hipMemcpyDeviceToHost));
  const int64_t nb = (N + 63) / 64;
  std::vector<uint8_t> mark;
  std::vector<int> tiles;
  auto add = [&](int64_t A, int64_t B) {
    const int64_t key = A * nb + B;
    if (key >= (int64_t)mark.size() * 8) mark.resize((size_t)(key / 8 + 1 + nb), 0);
    if (mark[(size_t)(key >> 3)] & (1u << (key & 7))) return;
    mark[(size_t)(key >> 3)] |= (uint8_t)(1u << (key & 7));
    tiles.push_back((int)A);
    tiles.push_back((int)B);
  };
  for (int64_t s0 = 0; s0 < N;) {
    int64_t s1 = s0 + 1;
    while (s1 < N && seg[(size_t)s1] == seg[(size_t)s0]) ++s1;
    if (s1 - s0 >= 2 && c->route_h[(size_t)(s0 / L)]) {
      const int64_t fa = s0 / 64, fb = (s1 - 1) / 64;
      for (int64_t A = fa; A <= fb; ++A)
        for (int64_t B = A; B <= fb; ++B) add(A, B);
    }
    s0 = s1;
  }
  const int ntiles = (int)(tiles.size() / 2);
  ENSURE(c, c->dg_counts, 16);
  HIP_TRY(c, hipMemsetAsync(c->dg_counts.p, 0, 16, c->stream));
  if (ntiles > 0) {
    ENSURE(c, c->dg_tiles, tiles.size() * 4);
    HIP_TRY(c, hipMemcpyAsync(c->dg_tiles.p, tiles.data(), tiles.size() * 4, hipMemcpyHostToDevice,
                              c->stream));
    HIP_TRY(c, launch_purity(X, dtype == SLH_BF16 ? 0 : 1, ldx, (int)c->D, P<int>(c->sval),
                             P<int>(c->sseg), P<double>(c->nrm_x), N, P<int>(c->dg_tiles), ntiles,
                             thresh, P<unsigned long long>(c->dg_counts), c->stream));
  }
  unsigned long long cnt[2] = {0, 0};
  HIP_TRY(c, hipMemcpyAsync(cnt, c->dg_counts.p, 16, hipMemcpyDeviceToHost, c->stream));
  HIP_TRY(c, hipStreamSynchronize(c->stream));
  counts_out[0] = (int64_t)cnt[0];
  counts_out[1] = (int64_t)cnt[1];
  return SLH_OK;
}

int slh_stage_times(slh_ctx* c, double* out, int32_t n) {
  if (!c || !out || n < 0) return SLH_EINVAL;
  if (!c->timing || !c->ev_made) return fail(c, SLH_ESTATE, "SLH_OPT_TIMING is off");
  HIP_TRY(c, hipStreamSynchronize(c->stream));
  double v[9] = {0, 0, 0, 0, 0, 0, 0, 0, 0};
  float ms = 0.f;
  auto el = [&](hipEvent_t a, hipEvent_t b) -> double {
    float t = 0.f;
    return hipEventElapsedTime(&t, a, b) == hipSuccess ? (double)t : -1.0;
  };
  v[0] = el(c->ev[0], c->ev[1]);
  v[1] = el(c->ev[2], c->ev[3]);
  for (int j = 0; j < c->fused_timed; ++j) {
    ms = (float)el(c->ev_fb[(size_t)j], c->ev_fa[(size_t)j]);
    v[2] += ms;
  }
  v[3] = c->passes_timed;
  v[4] = el(c->ev[3], c->ev[4]);
  v[5] = el(c->ev[5], c->ev[6]);
  v[6] = el(c->ev[7], c->ev[8]);
  v[7] = c->norm_timed ? el(c->ev[9], c->ev[10]) : 0.0;
  v[8] = c->lz_res ? 1.0 : 0.0;
  for (int i = 0; i < n && i < 9; ++i) out[i] = v[i];
  (void)hipGetLastError();   // a stage that did not run leaves unrecorded events
  return SLH_OK;
}

int slh_time_passes(slh_ctx* c, int32_t reps, double* us_out) {
  if (!c || !us_out) return SLH_EINVAL;
  if (reps < 1 || reps > 4096) return fail(c, SLH_EINVAL, "reps must be in [1, 4096]");
  if (c->stage < 2 || !c->lz_w_valid)
    return fail(c, SLH_ESTATE, "slh_time_passes needs a preceding full-size slh_lanczos");
  const LanczosWS& w = c->lz_w;
  hipGraph_t g = nullptr;
  hipGraphExec_t ge = nullptr;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  if (c->lz_res) {
    // the resident kernel: reps whole runs, each kernel between two events
    // (its preparation kernel outside them); us per Lanczos step
    const double* q1act = (c->n_act != c->n_win) ? P<double>(c->q1act) : P<double>(c->q1all);
    hipEvent_t r0 = nullptr, r1 = nullptr;
    hipError_t e = hipEventCreate(&r0);
    if (e == hipSuccess) e = hipEventCreate(&r1);
    double tot = 0.0;
    for (int q = 0; q < reps && e == hipSuccess; ++q) {
      e = launch_lanczos_resident(w, q1act, P<unsigned>(c->lz_bar), c->n_cu, c->stream, r0, r1);
      if (e == hipSuccess) e = hipEventSynchronize(r1);
      float ms = 0.f;
      if (e == hipSuccess) e = hipEventElapsedTime(&ms, r0, r1);
      if (q > 0 || reps == 1) tot += ms;   // the first run warms up
    }
    if (r0) (void)hipEventDestroy(r0);
    if (r1) (void)hipEventDestroy(r1);
    if (e != hipSuccess) return fail(c, SLH_EHIP, "slh_time_passes: %s", hipGetErrorString(e));
    unsigned ew = 0;
    HIP_TRY(c, hipMemcpy(&ew, P<unsigned>(c->lz_bar) + LZ_BAR_ERR, 4, hipMemcpyDeviceToHost));
    if (ew) return fail(c, SLH_EHIP, "Lanczos: a wait between blocks of the resident kernel timed out");
    *us_out = 1000.0 * tot / (reps > 1 ? reps - 1 : 1) / w.n_it;
    return SLH_OK;
  }
  HIP_TRY(c, hipStreamBeginCapture(c->cap_stream, hipStreamCaptureModeThreadLocal));
  const hipError_t le = launch_lanczos_passes(w, w.n_it - 1, reps, c->cap_stream);
  const hipError_t ce = hipStreamEndCapture(c->cap_stream, &g);
  if (le != hipSuccess || ce != hipSuccess) {
    if (g) (void)hipGraphDestroy(g);
    return fail(c, SLH_EHIP, "pass graph capture: %s / %s", hipGetErrorString(le),
                hipGetErrorString(ce));
  }
  hipError_t e = hipGraphInstantiate(&ge, g, nullptr, nullptr, 0);
  (void)hipGraphDestroy(g);
  if (e == hipSuccess) e = hipEventCreate(&e0);
  if (e == hipSuccess) e = hipEventCreate(&e1);
  if (e == hipSuccess) e = hipGraphLaunch(ge, c->stream);          // warm-up replay
  if (e == hipSuccess) e = hipEventRecord(e0, c->stream);
  if (e == hipSuccess) e = hipGraphLaunch(ge, c->stream);
  if (e == hipSuccess) e = hipEventRecord(e1, c->stream);
  if (e == hipSuccess) e = hipEventSynchronize(e1);
  float ms = 0.f;
  if (e == hipSuccess) e = hipEventElapsedTime(&ms, e0, e1);
  if (ge) (void)hipGraphExecDestroy(ge);
  if (e0) (void)hipEventDestroy(e0);
  if (e1) (void)hipEventDestroy(e1);
  if (e != hipSuccess) return fail(c, SLH_EHIP, "slh_time_passes: %s", hipGetErrorString(e));
  *us_out = 1000.0 * (double)ms / reps;
  return SLH_OK;
}

int slh_load(slh_ctx* c, int32_t which, const void* src, int64_t bytes) {
  if (!c || !src) return SLH_EINVAL;
  forget_norms(c);
  const int64_t L = window_len(c);
  const int64_t na = c->n_act;
  int rc = ensure_routing(c);
  if (rc) return rc;
  if (which == SLH_OUT_PHI) {
    const int64_t want = na * L * c->m * 4;
    if (bytes != want) return fail(c, SLH_EINVAL, "bytes must be %lld", (long long)want);
    ENSURE(c, c->Phi, (size_t)std::max<int64_t>(want, 4));
    if (want) HIP_TRY(c, hipMemcpyAsync(c->Phi.p, src, (size_t)want, hipMemcpyDeviceToDevice, c->stream));
    c->stage = 1;
    c->merged = 0;
    return SLH_OK;
  }
  if (which == SLH_OUT_CODES) {
    const int64_t want = c->Ntot * 4;
    if (bytes != want) return fail(c, SLH_EINVAL, "bytes must be %lld", (long long)want);
    ENSURE(c, c->codes, (size_t)want);
    HIP_TRY(c, hipMemcpyAsync(c->codes.p, src, (size_t)want, hipMemcpyDeviceToDevice, c->stream));
    c->stage = 3;
    c->merged = 0;
    return SLH_OK;
  }
  if (which == SLH_OUT_ALPHA) {
    // alpha of every spectral window: n_act x n_it doubles; sets n_it and
    // n_eff = n_it (and clears beta)
    if (na < 1 || bytes <= 0 || bytes % (na * 8) != 0)
      return fail(c, SLH_EINVAL, "bytes must be a positive multiple of n_act * 8");
    const int64_t n_it = bytes / (na * 8);
    if (n_it < c->r || n_it > std::min<int64_t>(L, 256))
      return fail(c, SLH_EINVAL, "need r <= n_it <= min(L, 256) (n_it=%lld)", (long long)n_it);
    ENSURE(c, c->alpha, (size_t)bytes);
    ENSURE(c, c->beta, (size_t)bytes);
    ENSURE(c, c->neff, (size_t)na * 4);
    ENSURE(c, c->Q, (size_t)na * (n_it + 1) * L * 8);
    HIP_TRY(c, hipMemcpyAsync(c->alpha.p, src, (size_t)bytes, hipMemcpyDeviceToDevice, c->stream));
    HIP_TRY(c, hipMemsetAsync(c->beta.p, 0, (size_t)bytes, c->stream));
    std::vector<int> ne((size_t)na, (int)n_it);
    HIP_TRY(c, hipMemcpyAsync(c->neff.p, ne.data(), ne.size() * 4, hipMemcpyHostToDevice, c->stream));
    HIP_TRY(c, hipStreamSynchronize(c->stream));     // ne leaves scope
    c->n_it = (int)n_it;
    c->t_loaded = 1;
    c->lz_w_valid = false;
    c->lz_res = false;
    c->stage = 1;
    c->merged = 0;
    return SLH_OK;
  }
  if (which == SLH_OUT_BETA || which == SLH_OUT_Q) {
    if (!(c->t_loaded & 1)) return fail(c, SLH_ESTATE, "load SLH_OUT_ALPHA first");
    const int64_t want = which == SLH_OUT_BETA ? na * c->n_it * 8 : na * (c->n_it + 1) * L * 8;
    if (bytes != want) return fail(c, SLH_EINVAL, "bytes must be %lld", (long long)want);
    DevBuf& b = which == SLH_OUT_BETA ? c->beta : c->Q;
    HIP_TRY(c, hipMemcpyAsync(b.p, src, (size_t)want, hipMemcpyDeviceToDevice, c->stream));
    c->t_loaded |= which == SLH_OUT_BETA ? 2 : 4;
    return SLH_OK;
  }
  return fail(c, SLH_EINVAL, "slh_load supports SLH_OUT_PHI, ALPHA, BETA, Q and CODES");
}

int slh_copy_out(slh_ctx* c, int32_t which, void* dst, int64_t bytes) {
  if (!c || !dst) return SLH_EINVAL;
  const int64_t L = window_len(c);
  const int64_t na = c->n_act;
  const DevBuf* b = nullptr;
  int64_t want = 0;
  switch (which) {
    case SLH_OUT_PHI: b = &c->Phi; want = na * L * c->m * 4; break;
    case SLH_OUT_ALPHA: b = &c->alpha; want = na * c->n_it * 8; break;
    case SLH_OUT_BETA: b = &c->beta; want = na * c->n_it * 8; break;
    case SLH_OUT_Z: b = &c->Z; want = na * L * c->r * 8; break;
    case SLH_OUT_PROJ: b = &c->proj; want = na * L * c->bits * 8; break;
    case SLH_OUT_CODES: b = &c->codes; want = c->Ntot * 4; break;
    case SLH_OUT_THETA: b = &c->theta; want = na * c->r * 8; break;
    case SLH_OUT_Q: b = &c->Q; want = na * (c->n_it + 1) * L * 8; break;
    case SLH_OUT_ROWSUM: b = &c->rowsum; want = na * L * 8; break;
    case SLH_OUT_WINDOWS:
      if (bytes != na * 4) return fail(c, SLH_EINVAL, "bytes must be %lld", (long long)(na * 4));
      if (na) std::memcpy(dst, c->winlist_h.data(), (size_t)na * 4);
      return SLH_OK;
    default: return fail(c, SLH_EINVAL, "unknown output %d", which);
  }
  if (bytes != want) return fail(c, SLH_EINVAL, "bytes must be %lld", (long long)want);
  if (want == 0) return SLH_OK;
  if (!b->p || (int64_t)b->bytes < want) return fail(c, SLH_ESTATE, "output %d not computed", which);
  HIP_TRY(c, hipStreamSynchronize(c->stream));
  HIP_TRY(c, hipMemcpy(dst, b->p, (size_t)want, hipMemcpyDeviceToHost));
  return SLH_OK;
}

}  // extern "C"
