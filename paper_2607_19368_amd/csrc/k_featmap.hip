// Random-feature map (section 3.2, Eq. 3; first line of Algorithm 1):
//   Phi[i, j] = rowscale_i * cos( sum_k bf16(X)[i, k] W[k, j] + psi_j )
// with rowscale_i = s(x_i) sqrt(2/m).  The contraction is a dense
// (n_rows x D) . (D x m) GEMM on bf16 MFMA (v_mfma_f32_32x32x16_bf16) with fp32
// accumulation; the cos/scale epilogue is fused and Phi is stored fp32.
//
// Tiling: a workgroup of WGM x WGN waves owns a BM x BN output tile (256 x 256
// with 2 x 4 waves, two waves per SIMD so that one issues MFMAs while the other
// waits on memory; 128 x 128 with 2 x 2 waves for small problems); each wave
// owns (BM/WGM) x (BN/WGN) as 32x32 MFMA tiles.  K advances 64 at a time through two LDS stages (register-staged
// prefetch of the next stage while the current one feeds the MFMAs).  LDS rows
// are 128 bytes (64 bf16); their eight 16-byte chunks are XOR-swizzled by the
// row index so that the MFMA operand reads of 8 consecutive rows hit distinct
// banks.  Rows beyond n_rows read zeros and are not stored; K beyond D is
// zero-filled (D % 8 == 0).  The epilogue stages the accumulators through LDS
// so the cos/scale work runs on contiguous rows and Phi leaves in 16-byte
// stores.
#include "slh_device.h"
#include "slh_internal.h"

#include <hip/hip_ext.h>

namespace slh {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

#define FM_BK 64

__device__ __forceinline__ int fm_global_row(int ar, const int* winlist, int L) {
  if (!winlist) return ar;
  const int w = ar / L;
  return winlist[w] * L + (ar - w * L);
}

template <int BM, int BN, int WGM, int WGN>
__global__ __launch_bounds__(64 * WGM * WGN) void k_featmap(FeatmapArgs a) {
  constexpr int NT = 64 * WGM * WGN;                 // threads
  constexpr int WM = BM / WGM, WN = BN / WGN;        // wave tile
  constexpr int TM = WM / 32, TN = WN / 32;          // MFMA tiles per wave
  constexpr int RS = NT / 8;                         // rows loaded per pass (8 chunks per row)
  constexpr int AR = BM / RS, BR = BN / RS;          // 16-byte chunks per thread per stage
  constexpr int STAGE_A = BM * FM_BK, STAGE_B = BN * FM_BK;   // bf16 elements
  // two K stages of A and B; reused after the main loop to stage the output
  __shared__ __attribute__((aligned(16))) uint16_t smem[2 * (STAGE_A + STAGE_B)];
  uint16_t* sA = smem;                        // [2][BM * 64]
  uint16_t* sB = smem + 2 * STAGE_A;          // [2][BN * 64]

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WGN, wn = wave % WGN;
  const int n_ntiles = a.m / BN;
  const int tile = blockIdx.x;
  const int m0 = (tile / n_ntiles) * BM;
  const int n0 = (tile % n_ntiles) * BN;
  const int n_rows = (int)a.n_rows;

  // loader: thread covers 16-byte chunk lc of rows lr + RS*i
  const int lc = tid & 7, lr = tid >> 3;
  const uint16_t* arow[AR];
  bool avalid[AR];
#pragma unroll
  for (int i = 0; i < AR; ++i) {
    const int ar = m0 + lr + RS * i;
    avalid[i] = ar < n_rows;
    arow[i] = a.X + (int64_t)fm_global_row(avalid[i] ? ar : 0, a.winlist, (int)a.L) * a.ldx;
  }
  const uint16_t* brow[BR];
#pragma unroll
  for (int i = 0; i < BR; ++i) brow[i] = a.Wt + (int64_t)(n0 + lr + RS * i) * a.D;

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;

  const int nk = (a.D + FM_BK - 1) / FM_BK;
  uint4 ra[AR], rb[BR];
  {
    const int kc = lc * 8;
    const bool kin = kc < a.D;
    const int kcc = min(kc, a.D - 8);
#pragma unroll
    for (int i = 0; i < AR; ++i) {
      const uint4 v = *(const uint4*)(arow[i] + kcc);
      ra[i] = (kin && avalid[i]) ? v : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < BR; ++i) {
      const uint4 v = *(const uint4*)(brow[i] + kcc);
      rb[i] = kin ? v : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < AR; ++i) {
      const int r = lr + RS * i;
      *(uint4*)(&sA[r * FM_BK + ((lc ^ (r & 7)) * 8)]) = ra[i];
    }
#pragma unroll
    for (int i = 0; i < BR; ++i) {
      const int r = lr + RS * i;
      *(uint4*)(&sB[r * FM_BK + ((lc ^ (r & 7)) * 8)]) = rb[i];
    }
  }
  __syncthreads();

  const int fr = lane & 31, fk = lane >> 5;   // fragment row/col within a 32-tile, k half
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    const bool more = kt + 1 < nk;
    if (more) {                                // prefetch the next K stage into registers
      const int kc = (kt + 1) * FM_BK + lc * 8;
      const bool kin = kc < a.D;
      const int kcc = min(kc, a.D - 8);
#pragma unroll
      for (int i = 0; i < AR; ++i) {
        const uint4 v = *(const uint4*)(arow[i] + kcc);
        ra[i] = (kin && avalid[i]) ? v : make_uint4(0, 0, 0, 0);
      }
#pragma unroll
      for (int i = 0; i < BR; ++i) {
        const uint4 v = *(const uint4*)(brow[i] + kcc);
        rb[i] = kin ? v : make_uint4(0, 0, 0, 0);
      }
    }
    const uint16_t* cA = sA + cur * STAGE_A;
    const uint16_t* cB = sB + cur * STAGE_B;
#pragma unroll
    for (int kk = 0; kk < FM_BK / 16; ++kk) {
      const int ch = 2 * kk + fk;
      bf16x8 fa[TM], fb[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int r = wm * WM + 32 * i + fr;
        fa[i] = *(const bf16x8*)(&cA[r * FM_BK + ((ch ^ (r & 7)) * 8)]);
      }
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int r = wn * WN + 32 * j + fr;
        fb[j] = *(const bf16x8*)(&cB[r * FM_BK + ((ch ^ (r & 7)) * 8)]);
      }
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[i], fb[j], acc[i][j], 0, 0, 0);
    }
    if (more) {
      uint16_t* nA = sA + (cur ^ 1) * STAGE_A;
      uint16_t* nB = sB + (cur ^ 1) * STAGE_B;
#pragma unroll
      for (int i = 0; i < AR; ++i) {
        const int r = lr + RS * i;
        *(uint4*)(&nA[r * FM_BK + ((lc ^ (r & 7)) * 8)]) = ra[i];
      }
#pragma unroll
      for (int i = 0; i < BR; ++i) {
        const int r = lr + RS * i;
        *(uint4*)(&nB[r * FM_BK + ((lc ^ (r & 7)) * 8)]) = rb[i];
      }
    }
    __syncthreads();
  }

  // epilogue, 32 rows of each wave at a time: stage the accumulators in LDS
  // (static register indices only), then apply cos(. + psi) * rowscale while
  // streaming rows out with 16-byte stores.  Accumulator layout: lane holds
  // column (lane & 31) of each 32x32 tile, rows 8*(v/4) + 4*(lane/32) + (v%4).
  constexpr int HM = 1;                              // MFMA row tiles staged per pass
  constexpr int SROWS = HM * 32, SCOLS = WN + 4;     // staged rows x (cols + pad)
  static_assert(WGM * WGN * SROWS * SCOLS * 4 <= 2 * (STAGE_A + STAGE_B) * 2, "staging exceeds LDS");
  float* stage = (float*)smem + wave * (SROWS * SCOLS);
#pragma unroll
  for (int h = 0; h < TM / HM; ++h) {
#pragma unroll
    for (int ii = 0; ii < HM; ++ii) {
#pragma unroll
      for (int j = 0; j < TN; ++j) {
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int r = 32 * ii + 8 * (v >> 2) + 4 * fk + (v & 3);
          stage[r * SCOLS + 32 * j + fr] = acc[h * HM + ii][j][v];
        }
      }
    }
    __syncthreads();
    // lane handles float4 column chunk (lane % (WN/4)) of rows lane / (WN/4) + k * (256/WN)
    constexpr int CPR = WN / 4;                      // float4 chunks per row
    constexpr int RPI = 64 / CPR;                    // rows per pass
    const int cc = lane % CPR, rr = lane / CPR;
    const int col = n0 + wn * WN + 4 * cc;
    const float4 ps = *(const float4*)(a.psi + col);
    for (int r = rr; r < SROWS; r += RPI) {
      const int row = m0 + wm * WM + h * SROWS + r;
      if (row < n_rows) {
        const float sc = a.rowscale[fm_global_row(row, a.winlist, (int)a.L)];
        const float4 v = *(const float4*)(&stage[r * SCOLS + 4 * cc]);
        float4 o;
        o.x = cosf(v.x + ps.x) * sc;
        o.y = cosf(v.y + ps.y) * sc;
        o.z = cosf(v.z + ps.z) * sc;
        o.w = cosf(v.w + ps.w) * sc;
        *(float4*)(a.Phi + (int64_t)row * a.m + col) = o;
      }
    }
    __syncthreads();
  }
}

hipError_t launch_featmap(const FeatmapArgs& a, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  (void)hipGetLastError();
  if (a.n_rows <= 0) return hipSuccess;
  // 256 x 256 tiles when that still gives at least one tile per CU, else 128 x 128
  int64_t t256 = ((a.n_rows + 255) / 256) * (a.m / 256);
  if (a.m % 256 == 0 && t256 >= 256) {
    auto k = k_featmap<256, 256, 2, 4>;
    if (e0) hipExtLaunchKernelGGL(k, dim3((unsigned)t256), dim3(512), 0, s, e0, e1, 0, a);
    else hipLaunchKernelGGL(k, dim3((unsigned)t256), dim3(512), 0, s, a);
  } else {
    int64_t t128 = ((a.n_rows + 127) / 128) * (a.m / 128);
    auto k = k_featmap<128, 128, 2, 2>;
    if (e0) hipExtLaunchKernelGGL(k, dim3((unsigned)t128), dim3(256), 0, s, e0, e1, 0, a);
    else hipLaunchKernelGGL(k, dim3((unsigned)t128), dim3(256), 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace slh
