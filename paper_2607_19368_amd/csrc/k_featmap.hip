// Random-feature map (section 3.2, Eq. 3; first line of Algorithm 1):
//   Phi[i, j] = rowscale_i * cos( sum_k bf16(X)[i, k] W[k, j] + psi_j )
// with rowscale_i = s(x_i) sqrt(2/m).  The contraction is a dense
// (n_rows x D) . (D x m) GEMM on bf16 MFMA (v_mfma_f32_32x32x16_bf16) with fp32
// accumulation; the cos/scale epilogue is fused and Phi is stored fp32.
//
// Tiling: a workgroup of WGM x WGN waves owns a BM x BN output tile (256 x 256
// with 2 x 4 waves, two waves per SIMD so that one issues MFMAs while the other
// waits on memory; 128 x 128 with 2 x 2 waves for small problems); each wave
// owns (BM/WGM) x (BN/WGN) as 32x32 MFMA tiles.  K advances FM_BK at a time
// through FM_NS LDS stages filled by direct global-to-LDS loads issued
// FM_NS - 1 stages ahead of the MFMAs that consume them (no register staging);
// within a stage the operands of the next k16 step are read while the current
// step's MFMAs run.  The 16-byte chunks of each LDS row are XOR-swizzled by the
// row index so that the MFMA operand reads of 16 consecutive rows hit distinct
// banks (see fm_swz).  Rows beyond n_rows re-read the last row and are not stored; K
// beyond D is zero-filled in W (D % 8 == 0).  The epilogue stages the accumulators through LDS
// so the cos/scale work runs on contiguous rows and Phi leaves in 16-byte
// stores.
#include "slh_device.h"
#include "slh_internal.h"

#include <hip/hip_ext.h>

namespace slh {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

#ifndef FM_BK
#define FM_BK 64                 // K per LDS stage (32 or 64)
#endif
#ifndef FM_NS
#define FM_NS 2                  // LDS stages (loads run FM_NS - 1 stages ahead)
#endif
#ifndef FM_DB
#define FM_DB 1                  // read the next k16 step's operands during this step's MFMAs
#endif
#ifndef FM_IL
#define FM_IL 1                  // pin an MFMA / LDS-read interleave (with FM_DB)
#endif
#ifndef FM_EPI
#define FM_EPI 1                 // epilogue staging sync: 0 block barriers, 1 per wave
#endif
#ifndef FM_BIG_BN
#define FM_BIG_BN 256            // N extent of the large tile (256 x FM_BIG_BN)
#endif
#ifndef FM_SROWS
#define FM_SROWS 32              // epilogue rows staged per pass (16 or 32)
#endif
#ifndef FM_BIG_WGM
#define FM_BIG_WGM 2             // waves along M in the large tile
#endif
#ifndef FM_BIG_WGN
#define FM_BIG_WGN 4             // waves along N in the 256 x 256 tile (2 x FM_BIG_WGN waves)
#endif
constexpr int FM_CPR = FM_BK / 8;        // 16-byte chunks per LDS row
constexpr int FM_RPL = 64 / FM_CPR;      // rows filled by one 1 KB direct-to-LDS load

// Physical 16-byte chunk of logical chunk c in LDS row r is c ^ fm_swz(r).  The
// LDS serves 16 lanes' 16-byte reads per clock over 256 bytes, so the 16
// consecutive rows read at one logical chunk must land in 16 distinct 16-byte
// bank groups.  64-byte rows (4 chunks): row r sits at group 4 (r & 3) + chunk,
// so the chunk must differ across r >> 2.  128-byte rows (8 chunks): group
// 8 (r & 1) + chunk, so the chunk must differ across the even (odd) rows; the
// r & 7 term also keeps any 8 consecutive rows distinct.
__device__ __forceinline__ int fm_swz(int r) {
  if constexpr (FM_CPR == 4) return (r >> 2) & 3;
  else return (r & 7) ^ ((r >> 3) & 1);
}

// s_waitcnt vmcnt(N) for the counts the pipeline uses
template <int N>
__device__ __forceinline__ void fm_wait_vm() {
  static_assert(N == 0 || N == 4 || N == 6 || N == 8 || N == 12 || N == 16, "unsupported count");
  if constexpr (N == 0) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  else if constexpr (N == 4) asm volatile("s_waitcnt vmcnt(4)" ::: "memory");
  else if constexpr (N == 6) asm volatile("s_waitcnt vmcnt(6)" ::: "memory");
  else if constexpr (N == 8) asm volatile("s_waitcnt vmcnt(8)" ::: "memory");
  else if constexpr (N == 12) asm volatile("s_waitcnt vmcnt(12)" ::: "memory");
  else asm volatile("s_waitcnt vmcnt(16)" ::: "memory");
}

__device__ __forceinline__ int fm_global_row(int ar, const int* winlist, int L) {
  if (!winlist) return ar;
  const int w = ar / L;
  return winlist[w] * L + (ar - w * L);
}

// Workgroups are dealt round-robin to the 8 XCDs (each with its own L2); give
// XCD x a contiguous range of tile ids, i.e. a band of output rows, so that each
// XCD streams only its share of X (W is small and shared).  A bijection on
// [0, T) for any T.
__device__ __forceinline__ int xcd_tile(int w, int T) {
  const int x = w & 7, idx = w >> 3;
  const int per = T >> 3, rem = T & 7;
  return (x < rem) ? x * (per + 1) + idx : rem * (per + 1) + (x - rem) * per + idx;
}

typedef __attribute__((address_space(1))) const void* fm_gptr;
typedef __attribute__((address_space(3))) void* fm_lptr;

template <int BM, int BN, int WGM, int WGN>
__global__ __launch_bounds__(64 * WGM * WGN) void k_featmap(FeatmapArgs a) {
  constexpr int NW = WGM * WGN;                      // waves
  constexpr int WM = BM / WGM, WN = BN / WGN;        // wave tile
  constexpr int TM = WM / 32, TN = WN / 32;          // MFMA tiles per wave
  constexpr int STAGE_A = BM * FM_BK, STAGE_B = BN * FM_BK;   // bf16 elements
  // a stage is loaded in groups of FM_RPL rows (1 KB, one direct-to-LDS load per wave)
  constexpr int LA = BM / FM_RPL / NW, LB = BN / FM_RPL / NW;  // loads per wave per stage
  static_assert(LA * FM_RPL * NW == BM && LB * FM_RPL * NW == BN, "row groups must split over the waves");
  constexpr int AHEAD = (FM_NS - 2) * (LA + LB);     // loads allowed in flight at a stage wait
  // FM_NS K stages of A and B; reused after the main loop to stage the output
  __shared__ __attribute__((aligned(16))) uint16_t smem[FM_NS * (STAGE_A + STAGE_B)];
  uint16_t* sA = smem;                        // [FM_NS][BM * FM_BK]
  uint16_t* sB = smem + FM_NS * STAGE_A;      // [FM_NS][BN * FM_BK]

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WGN, wn = wave % WGN;
  const int n_ntiles = a.m / BN;
  const int tile = xcd_tile(blockIdx.x, gridDim.x);
  const int m0 = (tile / n_ntiles) * BM;
  const int n0 = (tile % n_ntiles) * BN;
  const int n_rows = (int)a.n_rows;

  // Direct-to-LDS loader: load q of this wave fills stage rows FM_RPL g ..
  // FM_RPL (g + 1) - 1, g = q * NW + wave; lane l lands at row FM_RPL g + l /
  // FM_CPR, physical chunk l % FM_CPR, so it fetches logical chunk
  // (l % FM_CPR) ^ fm_swz(row).  Every load is unconditional:
  // A rows past n_rows re-read the last row (their outputs are never stored); A's
  // K index is clamped to the last chunk while W (zero for k >= D, row stride
  // ldw) supplies the zeros that cancel it.
  const int lrow = lane / FM_CPR, lchk = lane % FM_CPR;
  const uint16_t* arow[LA];
  int achk[LA];
#pragma unroll
  for (int q = 0; q < LA; ++q) {
    const int r = FM_RPL * (q * NW + wave) + lrow;
    const int ar = min(m0 + r, n_rows - 1);
    arow[q] = a.X + (int64_t)fm_global_row(ar, a.winlist, (int)a.L) * a.ldx;
    achk[q] = 8 * (lchk ^ fm_swz(r));
  }
  const uint16_t* bsrc[LB];
#pragma unroll
  for (int q = 0; q < LB; ++q) {
    const int r = FM_RPL * (q * NW + wave) + lrow;
    bsrc[q] = a.Wt + (int64_t)(n0 + r) * a.ldw + 8 * (lchk ^ fm_swz(r));
  }
  auto load_stage = [&](int kt, int buf) {
    const int k0 = kt * FM_BK;
    uint16_t* dA = sA + buf * STAGE_A;
    uint16_t* dB = sB + buf * STAGE_B;
#pragma unroll
    for (int q = 0; q < LA; ++q)
      __builtin_amdgcn_global_load_lds((fm_gptr)(arow[q] + min(k0 + achk[q], a.D - 8)),
                                       (fm_lptr)(dA + (q * NW + wave) * 512), 16, 0, 0);
#pragma unroll
    for (int q = 0; q < LB; ++q)
      __builtin_amdgcn_global_load_lds((fm_gptr)(bsrc[q] + k0),
                                       (fm_lptr)(dB + (q * NW + wave) * 512), 16, 0, 0);
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;

  const int nk = a.ldw / FM_BK;
#pragma unroll
  for (int p = 0; p < FM_NS - 1; ++p) load_stage(min(p, nk - 1), p);
  fm_wait_vm<AHEAD>();                               // stage 0 landed (this wave's part)
  __syncthreads();

  const int fr = lane & 31, fk = lane >> 5;   // fragment row/col within a 32-tile, k half
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & (FM_NS - 1);
    // stage kt + FM_NS - 1 streams into the buffer freed by the previous iteration
    // while this one feeds the MFMAs (past the end the last stage is re-read,
    // keeping the body branch-free and the per-stage load count fixed)
    load_stage(min(kt + FM_NS - 1, nk - 1), (kt + FM_NS - 1) & (FM_NS - 1));
    __builtin_amdgcn_sched_barrier(0);
    const uint16_t* cA = sA + cur * STAGE_A;
    const uint16_t* cB = sB + cur * STAGE_B;
    // operands of k16 step kk + 1 are read while step kk's MFMAs run
    bf16x8 fa[2][TM], fb[2][TN];
    auto read_ops = [&](int kk, int p) {
      const int ch = 2 * kk + fk;
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int r = wm * WM + 32 * i + fr;
        fa[p][i] = *(const bf16x8*)(&cA[r * FM_BK + ((ch ^ fm_swz(r)) * 8)]);
      }
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int r = wn * WN + 32 * j + fr;
        fb[p][j] = *(const bf16x8*)(&cB[r * FM_BK + ((ch ^ fm_swz(r)) * 8)]);
      }
    };
#if FM_DB
    read_ops(0, 0);
#pragma unroll
    for (int kk = 0; kk < FM_BK / 16; ++kk) {
      const int p = kk & 1;
      if (kk + 1 < FM_BK / 16) read_ops(kk + 1, p ^ 1);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[p][i], fb[p][j], acc[i][j], 0, 0, 0);
#if FM_IL
      // interleave: one MFMA, then one LDS read of the next step, ...
#pragma unroll
      for (int e = 0; e < TM + TN; ++e) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      }
      __builtin_amdgcn_sched_group_barrier(0x008, TM * TN - TM - TN, 0);
#endif
    }
#else
#pragma unroll
    for (int kk = 0; kk < FM_BK / 16; ++kk) {
      read_ops(kk, 0);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[0][i], fb[0][j], acc[i][j], 0, 0, 0);
    }
#endif
    fm_wait_vm<AHEAD>();                              // stage kt + 1 landed
    __syncthreads();
  }
  fm_wait_vm<0>();                                   // nothing in flight into smem
  __syncthreads();

  // epilogue, 32 rows of each wave at a time: stage the accumulators in the
  // wave's own LDS region (static register indices only), then apply
  // cos(. + psi) * rowscale while streaming rows out with 16-byte stores.
  // Accumulator layout: lane holds column (lane & 31) of each 32x32 tile, rows
  // 8*(v/4) + 4*(lane/32) + (v%4).
  // pad 8 floats: rows 4 apart (the two half-waves of a store) start 32 banks apart
  constexpr int SROWS = FM_SROWS, SCOLS = WN + 8;    // staged rows x (cols + pad)
  constexpr int NV = SROWS / 2;                      // accumulator values per lane per pass
  static_assert(SROWS == 16 || SROWS == 32, "stage 16 or 32 rows at a time");
  static_assert(WGM * WGN * SROWS * SCOLS * 4 <= FM_NS * (STAGE_A + STAGE_B) * 2, "staging exceeds LDS");
  float* stage = (float*)smem + wave * (SROWS * SCOLS);
#pragma unroll
  for (int h = 0; h < TM; ++h) {
#pragma unroll
    for (int hf = 0; hf < 32 / SROWS; ++hf) {
#pragma unroll
      for (int j = 0; j < TN; ++j) {
#pragma unroll
        for (int vv = 0; vv < NV; ++vv) {
          const int v = hf * NV + vv;
          const int r = 8 * (v >> 2) + 4 * fk + (v & 3) - hf * SROWS;
          stage[r * SCOLS + 32 * j + fr] = acc[h][j][v];
        }
      }
#if FM_EPI == 1
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#else
      __syncthreads();
#endif
      // lane handles float4 column chunk (lane % (WN/4)) of rows lane / (WN/4) + k * (256/WN)
      constexpr int CPR = WN / 4;                    // float4 chunks per row
      constexpr int RPI = 64 / CPR;                  // rows per pass
      const int cc = lane % CPR, rr = lane / CPR;
      const int col = n0 + wn * WN + 4 * cc;
      const float4 ps = *(const float4*)(a.psi + col);
      for (int r = rr; r < SROWS; r += RPI) {
        const int row = m0 + wm * WM + h * 32 + hf * SROWS + r;
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
#if FM_EPI == 1
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#else
      __syncthreads();
#endif
    }
  }
}



hipError_t launch_featmap(const FeatmapArgs& a, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  (void)hipGetLastError();
  if (a.n_rows <= 0) return hipSuccess;
  // 256 x 256 tiles when that still gives at least one tile per CU, else 128 x 128
  int64_t t256 = ((a.n_rows + 255) / 256) * (a.m / FM_BIG_BN);
  if (a.m % FM_BIG_BN == 0 && t256 >= 256) {
    auto k = k_featmap<256, FM_BIG_BN, FM_BIG_WGM, FM_BIG_WGN>;
    const dim3 blk(64 * FM_BIG_WGM * FM_BIG_WGN);
    if (e0) hipExtLaunchKernelGGL(k, dim3((unsigned)t256), blk, 0, s, e0, e1, 0, a);
    else hipLaunchKernelGGL(k, dim3((unsigned)t256), blk, 0, s, a);
  } else {
    int64_t t128 = ((a.n_rows + 127) / 128) * (a.m / 128);
    auto k = k_featmap<128, 128, 2, 2>;
    if (e0) hipExtLaunchKernelGGL(k, dim3((unsigned)t128), dim3(256), 0, s, e0, e1, 0, a);
    else hipLaunchKernelGGL(k, dim3((unsigned)t128), dim3(256), 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace slh
