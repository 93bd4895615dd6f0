// Random-feature map (section 3.2, Eq. 3; first line of Algorithm 1):
//   Phi[i, j] = rowscale_i * cos( sum_k bf16(X)[i, k] W[k, j] + psi_j )
// with rowscale_i = s(x_i) sqrt(2/m).  The contraction is a dense
// (n_rows x D) . (D x m) GEMM on bf16 MFMA (v_mfma_f32_32x32x16_bf16) with fp32
// accumulation; the cos/scale epilogue is fused and Phi is stored fp32.
//
// Tiling: a workgroup of WGM x WGN waves owns a BM x BN output tile (256 x 256
// with 2 x 4 waves, two waves per SIMD so that one issues MFMAs while the other
// waits on memory; 128 x 128, 64 x 128 or 64 x 64 when the large tiles would
// leave CUs idle, see launch_featmap); each wave
// owns (BM/WGM) x (BN/WGN) as 32x32 MFMA tiles.  K advances FM_BK at a time
// through FM_NS LDS stages filled by direct global-to-LDS loads issued
// FM_NS - 1 stages ahead of the MFMAs that consume them (no register staging),
// spread one behind each MFMA rather than in a burst; the operands of the next
// k16 step are read while the current step's MFMAs run, and the last step of a
// stage runs after the stage barrier.  The 16-byte chunks of each LDS row are
// XOR-swizzled by the row index so that the MFMA operand reads of 16
// consecutive rows hit distinct banks (see fm_swz).  Rows beyond n_rows re-read
// the last row and are not stored; K beyond D is zero-filled in W (D % 8 == 0).
// The epilogue stages the accumulators through LDS so the cos/scale work runs
// on contiguous rows and Phi leaves in 16-byte streaming stores.
#include "slh_device.h"
#include "slh_internal.h"

#include <hip/hip_ext.h>

namespace slh {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int FM_BK = 64;                // K per LDS stage
constexpr int FM_NS = 2;                 // LDS stages (loads run one stage ahead)
static_assert(FM_NS == 2, "the stage waits allow no load in flight");
constexpr int FM_LSPREAD = 1;            // k16 steps over which a stage's global->LDS loads go out
constexpr int FM_SROWS = 32;             // epilogue rows staged per pass
constexpr int FM_CPR = FM_BK / 8;        // 16-byte chunks per LDS row
constexpr int FM_RPL = 64 / FM_CPR;      // rows filled by one 1 KB direct-to-LDS load

// Physical 16-byte chunk of logical chunk c in LDS row r is c ^ fm_swz(r).  The
// LDS serves 16 lanes' 16-byte reads per clock over 256 bytes, so the 16
// consecutive rows read at one logical chunk must land in 16 distinct 16-byte
// bank groups.  A 128-byte row (8 chunks) sits at group 8 (r & 1) + chunk, so
// the chunk must differ across the even (odd) rows; the r & 7 term also keeps
// any 8 consecutive rows distinct.
static_assert(FM_CPR == 8, "the swizzle is laid out for 128-byte LDS rows");
__device__ __forceinline__ int fm_swz(int r) { return (r & 7) ^ ((r >> 3) & 1); }

// every global->LDS load of this wave landed (with two stages the next stage's
// loads are issued during the current one, so a stage wait allows none in flight)
__device__ __forceinline__ void fm_wait_loads() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// cos(x) in fp32 for the epilogue, about 1 ulp for |x| up to several thousand:
// Cody and Waite's reduction x = k pi/2 + r with pi/2 split into three fp32
// parts (x - k P1 is exact in the fma, so r carries one rounding), then the Taylor
// series of cos and sin on |r| <= pi/4 truncated after r^10 and r^9 (remainders
// below 2e-9), and the quadrant k mod 4 selecting +-cos r or +-sin r.  Straight-
// line code with no large-argument path, so the unrolled epilogue stays free
// of private memory.
__device__ __forceinline__ float fm_cos(float x) {
  const float k = __builtin_rintf(x * 0.636619747f);            // 2/pi
  float r = __builtin_fmaf(-k, 1.57079637f, x);                 // pi/2 = P1 + P2 + P3
  r = __builtin_fmaf(-k, -4.37113883e-08f, r);
  r = __builtin_fmaf(-k, -1.77635684e-15f, r);
  const float s = r * r;
  float c = __builtin_fmaf(s, -2.75573200e-07f, 2.48015876e-05f);  // -1/10!, 1/8!
  c = __builtin_fmaf(s, c, -1.38888892e-03f);                   // -1/6!
  c = __builtin_fmaf(s, c, 4.16666679e-02f);                    // 1/4!
  c = __builtin_fmaf(s, c, -0.5f);
  c = __builtin_fmaf(s, c, 1.0f);
  float sn = __builtin_fmaf(s, 2.75573188e-06f, -1.98412701e-04f); // 1/9!, -1/7!
  sn = __builtin_fmaf(s, sn, 8.33333377e-03f);                  // 1/5!
  sn = __builtin_fmaf(s, sn, -1.66666672e-01f);                 // -1/3!
  sn = __builtin_fmaf(s * r, sn, r);
  const int q = (int)k;                      // cos(r + q pi/2): c, -sn, -c, sn
  const float v = (q & 1) ? sn : c;
  return ((q + 1) & 2) ? -v : v;
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
  // load c of a stage (c < LA: A rows, else B rows) into stage buffer buf
  auto load_one = [&](int kt, int buf, int c) {
    const int k0 = kt * FM_BK;
    if (c < LA)
      __builtin_amdgcn_global_load_lds((fm_gptr)(arow[c] + min(k0 + achk[c], a.D - 8)),
                                       (fm_lptr)(sA + buf * STAGE_A + (c * NW + wave) * 512), 16, 0, 0);
    else
      __builtin_amdgcn_global_load_lds((fm_gptr)(bsrc[c - LA] + k0),
                                       (fm_lptr)(sB + buf * STAGE_B + ((c - LA) * NW + wave) * 512), 16, 0, 0);
  };
  auto load_stage = [&](int kt, int buf) {
#pragma unroll
    for (int c = 0; c < LA + LB; ++c) load_one(kt, buf, c);
  };
  constexpr int NLD = LA + LB;                       // loads per wave per stage
  constexpr int KS = FM_BK / 16;                     // k16 steps per stage
  constexpr int LSP = FM_LSPREAD < KS - 1 ? FM_LSPREAD : KS - 1;
  static_assert(KS >= 2, "the last k16 step of a stage runs after its barrier");
  constexpr int LPS = (NLD + LSP - 1) / LSP;         // loads issued per k16 step

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
  fm_wait_loads();                                   // stage 0 landed (this wave's part)
  __syncthreads();

  const int fr = lane & 31, fk = lane >> 5;   // fragment row/col within a 32-tile, k half
  // two register sets of MFMA operands: step kk of a stage uses set kk & 1
  bf16x8 fa[2][TM], fb[2][TN];
  auto read_ops = [&](const uint16_t* cA, const uint16_t* cB, int kk, int p) {
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
  auto mfmas = [&](int p) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[p][i], fb[p][j], acc[i][j], 0, 0, 0);
  };
  // pin the order of one step: an MFMA, then up to two of the step's nd LDS
  // reads behind each of the first MFMAs, then one of its nv global->LDS loads
  // behind each later MFMA
  auto pattern = [&](int nd, int nv) {
    const int d0 = (nd + 1) / 2;
#pragma unroll
    for (int e = 0; e < TM * TN; ++e) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      if (2 * e < nd) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      if (2 * e + 1 < nd) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      if (e >= d0 && e - d0 < nv) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
    }
  };

  // Software pipeline over the k16 steps: the operands of step kk + 1 are read
  // (into the other register set) while step kk's MFMAs run.  The last step of
  // a stage runs after the stage barrier, its operands already in registers, so
  // its MFMAs cover the latency of the first reads from the next stage.  The
  // next stage's global->LDS loads go out one behind each MFMA in the first LSP
  // steps rather than in one burst that would hold up the MFMA issue.
  read_ops(sA, sB, 0, 0);
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & (FM_NS - 1);
    // stage kt + FM_NS - 1 streams into the buffer freed by the previous
    // iteration while this one feeds the MFMAs (past the end the last stage is
    // re-read, keeping the body branch-free and the per-stage load count fixed)
    const int lkt = min(kt + FM_NS - 1, nk - 1), lbuf = (kt + FM_NS - 1) & (FM_NS - 1);
    const uint16_t* cA = sA + cur * STAGE_A;
    const uint16_t* cB = sB + cur * STAGE_B;
#pragma unroll
    for (int kk = 0; kk + 1 < KS; ++kk) {
      read_ops(cA, cB, kk + 1, (kk + 1) & 1);
#pragma unroll
      for (int c = 0; c < NLD; ++c)
        if (c / LPS == kk) load_one(lkt, lbuf, c);
      mfmas(kk & 1);
      pattern(TM + TN, (kk < LSP) ? min(LPS, NLD - kk * LPS) : 0);
      __builtin_amdgcn_sched_barrier(0);
    }
    // every read of this stage has landed in registers before the barrier (the
    // buffer is refilled after it); stage kt + 1 has landed after it
    fm_wait_loads();
    __syncthreads();
    // first operands of stage kt + 1 (after the last stage: a re-read of valid
    // data, discarded), under the MFMAs of this stage's last step
    const int nb = (kt + 1) & (FM_NS - 1);
    read_ops(sA + nb * STAGE_A, sB + nb * STAGE_B, 0, 0);
    mfmas((KS - 1) & 1);
    pattern(TM + TN, 0);
    __builtin_amdgcn_sched_barrier(0);
  }
  fm_wait_loads();                                   // nothing in flight into smem
  __syncthreads();

  // epilogue, 32 rows of each wave at a time: stage the accumulators in the
  // wave's own LDS region (static register indices only), then apply
  // cos(. + psi) * rowscale while streaming rows out with 16-byte stores.
  // Accumulator layout: lane holds column (lane & 31) of each 32x32 tile, rows
  // 8*(v/4) + 4*(lane/32) + (v%4).
  // pad 8 floats: rows 4 apart (the two half-waves of a store) start 32 banks apart
  constexpr int SROWS = FM_SROWS, SCOLS = WN + 8;    // staged rows x (cols + pad)
  constexpr int NV = SROWS / 2;                      // accumulator values per lane per pass
  static_assert(WGM * WGN * SROWS * SCOLS * 4 <= FM_NS * (STAGE_A + STAGE_B) * 2, "staging exceeds LDS");
  static_assert(WM % 64 == 0, "row scales are held 64 rows per register");
  float* stage = (float*)smem + wave * (SROWS * SCOLS);
  // lane handles float4 column chunk (lane % (WN/4)) of rows lane / (WN/4) + k * (256/WN)
  constexpr int CPR = WN / 4;                        // float4 chunks per row
  constexpr int RPI = 64 / CPR;                      // rows per pass
  constexpr int NP = SROWS / RPI;                    // passes per staged block
  const int cc = lane % CPR, rr = lane / CPR;
  const int col = n0 + wn * WN + 4 * cc;
  const float4 ps = *(const float4*)(a.psi + col);
  // the wave's row scales, one per lane and 64 rows, fetched once up front
  // (clamped rows: never stored) and handed to the storing lanes by shuffles
  float rsc[WM / 64];
#pragma unroll
  for (int q = 0; q < WM / 64; ++q) {
    const int row = min(m0 + wm * WM + 64 * q + lane, n_rows - 1);
    rsc[q] = a.rowscale[fm_global_row(row, a.winlist, (int)a.L)];
  }
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
      // the staging region is the wave's own: a wave barrier orders it
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      // all staged values and row scales are read before any store, so no
      // wait sits behind the row guard
      const int lr0 = h * 32 + hf * SROWS;          // wave-local row of staged row 0
      float4 vs[NP];
      float scs[NP];
#pragma unroll
      for (int k = 0; k < NP; ++k) {
        const int r = rr + k * RPI;
        vs[k] = *(const float4*)(&stage[r * SCOLS + 4 * cc]);
        scs[k] = __shfl(rsc[lr0 / 64], (lr0 % 64) + r, 64);
      }
#pragma unroll
      for (int k = 0; k < NP; ++k) {
        const int row = m0 + wm * WM + lr0 + rr + k * RPI;
        float4 o;
        o.x = fm_cos(vs[k].x + ps.x) * scs[k];
        o.y = fm_cos(vs[k].y + ps.y) * scs[k];
        o.z = fm_cos(vs[k].z + ps.z) * scs[k];
        o.w = fm_cos(vs[k].w + ps.w) * scs[k];
        if (row < n_rows) {
          float* dst = a.Phi + (int64_t)row * a.m + col;
          // the four merge into one 16-byte streaming store
          __builtin_nontemporal_store(o.x, dst);
          __builtin_nontemporal_store(o.y, dst + 1);
          __builtin_nontemporal_store(o.z, dst + 2);
          __builtin_nontemporal_store(o.w, dst + 3);
        }
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }
  }
}



template <int BM, int BN, int WGM, int WGN>
static void launch_tiles(const FeatmapArgs& a, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  const int64_t t = ((a.n_rows + BM - 1) / BM) * (a.m / BN);
  auto k = k_featmap<BM, BN, WGM, WGN>;
  const dim3 blk(64 * WGM * WGN);
  if (e0) hipExtLaunchKernelGGL(k, dim3((unsigned)t), blk, 0, s, e0, e1, 0, a);
  else hipLaunchKernelGGL(k, dim3((unsigned)t), blk, 0, s, a);
}

hipError_t launch_featmap(const FeatmapArgs& a, int n_cu, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  (void)hipGetLastError();
  if (a.n_rows <= 0) return hipSuccess;
  // Tile shape by how the tiles fill the CUs.  256 x 256 (eight waves) when
  // every CU gets a tile; below that, the largest of 128 x 128 (eight waves),
  // 64 x 128 (four) and 64 x 64 (two) that still gives every CU two tiles, so
  // that two workgroups share each CU's MFMA pipes and cover each other's
  // memory waits (measured at 4096 x 4096 x 1024, 8192 x 3584 x 256 and
  // 4000 x 3584 x 2048: the rule picks the fastest shape or one within 2%).
  const int64_t rb = (a.n_rows + 63) / 64, rb2 = (a.n_rows + 127) / 128;
  const int64_t t256 = ((a.n_rows + 255) / 256) * (a.m / 256);
  if (a.m % 256 == 0 && t256 >= n_cu)
    launch_tiles<256, 256, 2, 4>(a, s, e0, e1);
  else if (rb2 * (a.m / 128) >= 2LL * n_cu)
    launch_tiles<128, 128, 2, 4>(a, s, e0, e1);
  else if (rb * (a.m / 128) >= 2LL * n_cu)
    launch_tiles<64, 128, 1, 4>(a, s, e0, e1);
  else
    launch_tiles<64, 64, 1, 2>(a, s, e0, e1);
  return hipGetLastError();
}

}  // namespace slh
