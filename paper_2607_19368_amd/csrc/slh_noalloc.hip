// The merge of slh_merge (Eq. 7, section 3.4 max positions, section 3.6
// order) for callers that cannot allocate device memory: every workspace lives
// in one file-scope device array of fixed size instead of memory the call
// allocates.  The array is not a device address in host code; its address on
// each device is taken once with hipGetSymbolAddress (with that device current)
// and only that address is handed to kernels.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <mutex>

#include "slh.h"
#include "slh_internal.h"

namespace {

constexpr int64_t NA_NMAX = 8192;           // tokens
constexpr int64_t NA_DMAX = 4096;           // embedding width
constexpr int NA_CH = 16;                   // sorted positions per reduction chunk (as slh_merge)
constexpr int64_t NA_NCH = (NA_NMAX + NA_CH - 1) / NA_CH;

// byte offsets of the workspaces inside the array (each 256-byte aligned)
constexpr int64_t na_al(int64_t b) { return (b + 255) & ~(int64_t)255; }
constexpr int64_t NA_INTS = 0;                                   // 10 int arrays of NMAX
constexpr int64_t NA_NRM = NA_INTS + na_al(10 * NA_NMAX * 4);    // nrm2_fm, nrm_x, inv_x (double)
constexpr int64_t NA_RSC = NA_NRM + na_al(3 * NA_NMAX * 8);      // rowscale (float)
constexpr int64_t NA_SMALL = NA_RSC + na_al(NA_NMAX * 4);        // mw, wbase[2], Mtot, route
constexpr int64_t NA_PSEG = NA_SMALL + 256;                      // part_seg, part_cnt, part_end
constexpr int64_t NA_PNS = NA_PSEG + na_al(3 * 2 * NA_NCH * 4);  // part_nsum (double)
constexpr int64_t NA_PART = NA_PNS + na_al(2 * NA_NCH * 8);      // part (float, 2 NCH x DMAX)
constexpr int64_t NA_BYTES = NA_PART + na_al(2 * NA_NCH * NA_DMAX * 4);
static_assert(NA_BYTES == SLH_NOALLOC_BYTES, "SLH_NOALLOC_BYTES in slh.h must match the layout");

// The workspace array: one copy per device, held until the process ends.
static __device__ __align__(256) unsigned char scratch[NA_BYTES];

constexpr int NA_MAXDEV = 64;
std::mutex na_mu;
void* na_ptr[NA_MAXDEV] = {};               // device address of `scratch` per device

// Device address of the array on the current device (taken on the first call
// on that device).
hipError_t scratch_address(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= NA_MAXDEV) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(na_mu);
  if (!na_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    na_ptr[dev] = p;
  }
  *out = na_ptr[dev];
  return hipSuccess;
}

}  // namespace

extern "C" int slh_merge_noalloc(const void* X, int32_t dtype, int64_t ldx, int64_t N, int64_t D,
                                 const uint32_t* codes, int32_t bits, float* emb_out,
                                 int32_t* pos_out, int32_t* tok2macro_out, int64_t cap,
                                 int64_t* M_out, void* stream) {
  using namespace slh;
  if (!X || !codes || !emb_out || !pos_out || !M_out) return SLH_EINVAL;
  if (dtype != SLH_BF16 && dtype != SLH_F32) return SLH_EINVAL;
  if (N < 2 || N > NA_NMAX || D < 8 || D > NA_DMAX || D % 8 != 0) return SLH_EINVAL;
  if (ldx < D || ldx % 8 != 0 || ((uintptr_t)X) % 16 != 0) return SLH_EINVAL;
  if (bits < 1 || bits > 16) return SLH_EINVAL;
  if (cap < std::min<int64_t>(N, (int64_t)1 << bits)) return SLH_EINVAL;
  void* base = nullptr;
  if (scratch_address(&base) != hipSuccess) return SLH_EHIP;
  unsigned char* b = (unsigned char*)base;
  hipStream_t s = (hipStream_t)stream;
  int* ints = (int*)(b + NA_INTS);
  double* nrm = (double*)(b + NA_NRM);
  int* small = (int*)(b + NA_SMALL);
  int* pseg = (int*)(b + NA_PSEG);
  MergeWS w;
  w.n_win = 1;
  w.L = (int)N;
  w.bits = bits;
  w.chunk_k = 1;
  w.compact = 0;
  w.D = (int)D;
  w.N = N;
  w.route = (const uint8_t*)(small + 4);
  w.codes = codes;
  w.nrm_x = nrm + NA_NMAX;
  w.keyA = (uint32_t*)(ints + 0 * NA_NMAX);
  w.keyB = (uint32_t*)(ints + 1 * NA_NMAX);
  w.valA = ints + 2 * NA_NMAX;
  w.valB = ints + 3 * NA_NMAX;
  w.tmpi = ints + 4 * NA_NMAX;
  w.segid = ints + 5 * NA_NMAX;
  w.segk = ints + 6 * NA_NMAX;
  w.sval = ints + 7 * NA_NMAX;
  w.sloc = ints + 8 * NA_NMAX;
  w.sseg = ints + 9 * NA_NMAX;
  w.mw = small + 0;
  w.wbase = small + 1;                      // 2 entries
  w.Mtot = small + 3;
  w.part = (float*)(b + NA_PART);
  w.part_seg = pseg;
  w.part_cnt = pseg + 2 * NA_NCH;
  w.part_end = pseg + 4 * NA_NCH;
  w.part_nsum = (double*)(b + NA_PNS);
  w.CH = NA_CH;
  w.scheme = 0;
  w.posv = nullptr;
  w.pre = nullptr;
  w.tw = nullptr;
  w.tg = nullptr;
  // the window's route flag (spectral: every byte 1) by a fill kernel, not a
  // memset, so that the call may be captured into a graph
  if (launch_fill_u32((uint32_t*)(small + 4), 1, 0x01010101u, s) != hipSuccess) return SLH_EHIP;
  if (launch_rownorm(X, dtype == SLH_BF16 ? 0 : 1, ldx, N, (int)D, 256, 0, nrm, nrm + NA_NMAX,
                     nrm + 2 * NA_NMAX, (float*)(b + NA_RSC), nullptr, s) != hipSuccess)
    return SLH_EHIP;
  if (launch_merge(w, X, dtype == SLH_BF16 ? 0 : 1, ldx, emb_out, pos_out, tok2macro_out, s) !=
      hipSuccess)
    return SLH_EHIP;
  int M = 0;
  if (hipMemcpyAsync(&M, w.Mtot, 4, hipMemcpyDeviceToHost, s) != hipSuccess) return SLH_EHIP;
  if (hipStreamSynchronize(s) != hipSuccess) return SLH_EHIP;
  *M_out = M;
  return SLH_OK;
}
