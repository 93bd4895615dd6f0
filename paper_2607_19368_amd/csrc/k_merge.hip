// Macro-token construction (Eq. 7, section 3.4 max positions, section 3.6
// ordering by representative position).
//
// book      one workgroup per window.  Spectral windows: stable LSD radix sort
//           of (code, token) by code with 8-bit digits (histogram, scan and a
//           stable scatter whose in-wave ranks come from ballot matching), so
//           every bucket becomes a run of ascending token indices; a bucket's
//           position is its last token; buckets are ranked by that position
//           with a scan over the window in token order.  Chunk windows: groups
//           of k consecutive tokens (section 3.5).
// wbase     prefix of the per-window macro counts -> global macro indices.
// finalize  global macro index per sorted position, token -> macro map, P.
// reduce    the sorted member list is cut into chunks of CH positions; a
//           workgroup sums the member rows of each run (fp32 accumulation) and
//           renormalises runs that are whole buckets; runs cut by a chunk edge
//           leave a partial sum.
// combine   sums the partials of each cut bucket in chunk order and renormalises.
// All orders are fixed, so results are bitwise reproducible.
#include "slh_device.h"
#include "slh_internal.h"

namespace slh {

#define MG_CHMAX 64

// inclusive scan of one int per thread over a 1024-thread block
__device__ __forceinline__ int block_incl_scan_1024(int v, int* wsum, int& total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    int t = __shfl_up(v, o, 64);
    if (lane >= o) v += t;
  }
  __syncthreads();
  if (lane == 63) wsum[wave] = v;
  __syncthreads();
  int pre = 0, tot = 0;
  for (int k = 0; k < 16; ++k) {
    int x = wsum[k];
    if (k < wave) pre += x;
    tot += x;
  }
  total = tot;
  return v + pre;
}

__global__ __launch_bounds__(1024) void k_mg_book(MergeWS w) {
  const int win = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int L = w.L;
  const int64_t base = (int64_t)win * L;
  __shared__ int hist[256];
  __shared__ int wcnt[16][256];
  __shared__ int wsum[16];
  if (!w.route[win]) {
    const int k = w.chunk_k;
    for (int s = tid; s < L; s += 1024) {
      w.sval[base + s] = (int)(base + s);
      w.sloc[base + s] = s / k;
    }
    if (tid == 0) w.mw[win] = (L + k - 1) / k;
    return;
  }
  const int npass = (w.bits + 7) / 8;
  uint32_t* kb[2] = {w.keyA + base, w.keyB + base};
  int* vb[2] = {w.valA + base, w.valB + base};
  for (int k = tid; k < 16 * 256; k += 1024) (&wcnt[0][0])[k] = 0;
  for (int p = 0; p < npass; ++p) {
    const int shift = 8 * p;
    const uint32_t* kin = (p == 0) ? (w.codes + base) : kb[(p - 1) & 1];
    const int* vin = (p == 0) ? nullptr : vb[(p - 1) & 1];
    uint32_t* kout = kb[p & 1];
    int* vout = vb[p & 1];
    if (tid < 256) hist[tid] = 0;
    __syncthreads();
    for (int i = tid; i < L; i += 1024) atomicAdd(&hist[(kin[i] >> shift) & 255], 1);
    __syncthreads();
    // exclusive scan of the 256 digit counts
    int h = (tid < 256) ? hist[tid] : 0;
    int tot;
    int inc = block_incl_scan_1024(h, wsum, tot);
    __syncthreads();
    if (tid < 256) hist[tid] = inc - h;      // running base per digit
    __syncthreads();
    for (int b0 = 0; b0 < L; b0 += 1024) {
      const int i = b0 + tid;
      const bool valid = i < L;
      uint32_t key = 0;
      int val = 0;
      if (valid) {
        key = kin[i];
        val = vin ? vin[i] : (int)(base + i);
      }
      const int d = valid ? (int)((key >> shift) & 255) : 256;
      unsigned long long peers = ~0ull;
#pragma unroll
      for (int bit = 0; bit < 9; ++bit) {
        const bool on = (d >> bit) & 1;
        const unsigned long long bal = __ballot(on);
        peers &= on ? bal : ~bal;
      }
      const unsigned long long lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
      const int rank = __popcll(peers & lt);
      const int leader = 63 - __clzll(peers);
      if (valid && lane == leader) wcnt[wave][d] = __popcll(peers);
      __syncthreads();
      if (valid) {
        int off = hist[d] + rank;
        for (int q = 0; q < wave; ++q) off += wcnt[q][d];
        kout[off] = key;
        vout[off] = val;
      }
      __syncthreads();
      if (tid < 256) {
        int s = 0;
        for (int q = 0; q < 16; ++q) {
          s += wcnt[q][tid];
          wcnt[q][tid] = 0;
        }
        hist[tid] += s;
      }
      __threadfence_block();
      __syncthreads();
    }
    __threadfence();
    __syncthreads();
  }
  const uint32_t* K = kb[(npass - 1) & 1];
  const int* V = vb[(npass - 1) & 1];
  int* flag = w.tmpi + base;      // token order: 1 = bucket representative
  int* segid = w.segid + base;    // sorted order: bucket ordinal (by code)
  int* segk = w.segk + base;      // bucket ordinal -> macro rank
  for (int s = tid; s < L; s += 1024) flag[s] = 0;
  __threadfence();
  __syncthreads();
  // bucket ordinals and representatives
  int carry = 0;
  for (int b0 = 0; b0 < L; b0 += 1024) {
    const int s = b0 + tid;
    int st = 0;
    if (s < L) {
      st = (s == 0 || K[s] != K[s - 1]);
      if (s == L - 1 || K[s + 1] != K[s]) flag[V[s] - base] = 1;
    }
    int tot;
    int inc = block_incl_scan_1024(st, wsum, tot);
    if (s < L) segid[s] = carry + inc - 1;
    carry += tot;
    __syncthreads();
  }
  const int nseg = carry;
  __threadfence();
  __syncthreads();
  // macro rank of each representative = number of representatives before it
  carry = 0;
  for (int b0 = 0; b0 < L; b0 += 1024) {
    const int i = b0 + tid;
    const int f = (i < L) ? flag[i] : 0;
    int tot;
    int inc = block_incl_scan_1024(f, wsum, tot);
    if (i < L) flag[i] = f ? (carry + inc - 1) : -1;
    carry += tot;
    __syncthreads();
  }
  __threadfence();
  __syncthreads();
  for (int s = tid; s < L; s += 1024)
    if (s == L - 1 || K[s + 1] != K[s]) segk[segid[s]] = flag[V[s] - base];
  __threadfence();
  __syncthreads();
  for (int s = tid; s < L; s += 1024) {
    w.sval[base + s] = V[s];
    w.sloc[base + s] = segk[segid[s]];
  }
  if (tid == 0) w.mw[win] = nseg;
}

__global__ __launch_bounds__(1024) void k_mg_wbase(MergeWS w) {
  __shared__ int wsum[16];
  int carry = 0;
  for (int b0 = 0; b0 < w.n_win; b0 += 1024) {
    const int i = b0 + threadIdx.x;
    const int v = (i < w.n_win) ? w.mw[i] : 0;
    int tot;
    int inc = block_incl_scan_1024(v, wsum, tot);
    if (i < w.n_win) w.wbase[i] = carry + inc - v;
    carry += tot;
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    w.wbase[w.n_win] = carry;
    *w.Mtot = carry;
  }
}

__global__ __launch_bounds__(256) void k_mg_finalize(MergeWS w, int* __restrict__ P,
                                                     int* __restrict__ tok2macro) {
  const int64_t s = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (s >= w.N) return;
  const int win = (int)(s / w.L);
  const int loc = w.sloc[s];
  const int g = w.wbase[win] + loc;
  w.sseg[s] = g;
  const int tok = w.sval[s];
  if (tok2macro) tok2macro[tok] = g;
  const bool end = (s + 1 == w.N) || ((s + 1) % w.L == 0) || (w.sloc[s + 1] != loc);
  if (end) P[g] = w.compact ? g : tok;
}

template <int DT, int PPT>
__device__ __forceinline__ void mg_load(const void* X, int64_t ldx, int tok, int D,
                                        float (&x)[2 * PPT]) {
  const int tid = threadIdx.x;
#pragma unroll
  for (int q = 0; q < PPT; ++q) {
    const int p = tid + 256 * q;
    if (2 * p < D) {
      if (DT == 0) {
        const uint32_t v = *((const uint32_t*)((const uint16_t*)X + (int64_t)tok * ldx) + p);
        x[2 * q] = __uint_as_float(v << 16);
        x[2 * q + 1] = __uint_as_float(v & 0xFFFF0000u);
      } else {
        const float2 v = *((const float2*)((const float*)X + (int64_t)tok * ldx) + p);
        x[2 * q] = v.x;
        x[2 * q + 1] = v.y;
      }
    } else {
      x[2 * q] = 0.0f;
      x[2 * q + 1] = 0.0f;
    }
  }
}

template <int DT, int PPT>
__global__ __launch_bounds__(256) void k_mg_reduce(MergeWS w, const void* __restrict__ X,
                                                   int64_t ldx, float* __restrict__ E) {
  const int c = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int D = w.D;
  const int64_t s0 = (int64_t)c * w.CH;
  const int n = (int)min((int64_t)w.CH, w.N - s0);
  __shared__ int ssv[MG_CHMAX], ssg[MG_CHMAX];
  __shared__ double snrm[MG_CHMAX];
  __shared__ int prev_g, next_g;
  __shared__ float runsq[MG_CHMAX][4];
  __shared__ int run_g[MG_CHMAX], run_len[MG_CHMAX], run_kind[MG_CHMAX];
  __shared__ double run_nsum[MG_CHMAX];
  if (tid < n) {
    const int tok = w.sval[s0 + tid];
    ssv[tid] = tok;
    ssg[tid] = w.sseg[s0 + tid];
    snrm[tid] = w.nrm_x[tok];
  }
  if (tid == 0) {
    prev_g = (s0 > 0) ? w.sseg[s0 - 1] : -1;
    next_g = (s0 + n < w.N) ? w.sseg[s0 + n] : -1;
  }
  __syncthreads();
  float acc[2 * PPT], x[2 * PPT];
#pragma unroll
  for (int e = 0; e < 2 * PPT; ++e) acc[e] = 0.0f;
  double nsum = 0.0;
  int rs = 0, nrun = 0;
  mg_load<DT, PPT>(X, ldx, ssv[0], D, x);
  for (int s = 0; s < n; ++s) {
    float cur[2 * PPT];
#pragma unroll
    for (int e = 0; e < 2 * PPT; ++e) cur[e] = x[e];
    if (s + 1 < n) mg_load<DT, PPT>(X, ldx, ssv[s + 1], D, x);
#pragma unroll
    for (int e = 0; e < 2 * PPT; ++e) acc[e] += cur[e];
    nsum += snrm[s];
    const int g = ssg[s];
    if (s == n - 1 || ssg[s + 1] != g) {
      const bool starts = (rs > 0) || (prev_g != g);
      const bool ends = (s < n - 1) || (next_g != g);
      // kind 0: whole bucket -> E; 1: head partial (slot 2c); 2: tail partial (slot 2c+1)
      const int kind = (starts && ends) ? 0 : (!starts ? 1 : 2);
      float* dst = (kind == 0) ? (E + (int64_t)g * D)
                               : (w.part + (int64_t)(2 * c + (kind == 2)) * D);
      float sq = 0.0f;
#pragma unroll
      for (int q = 0; q < PPT; ++q) {
        const int p = tid + 256 * q;
        if (2 * p < D) {
          *(float2*)(dst + 2 * p) = make_float2(acc[2 * q], acc[2 * q + 1]);
          sq += acc[2 * q] * acc[2 * q] + acc[2 * q + 1] * acc[2 * q + 1];
        }
      }
      sq = wave_sum_f32(sq);
      if (lane == 0) runsq[nrun][wave] = sq;
      if (tid == 0) {
        run_g[nrun] = g;
        run_len[nrun] = s - rs + 1;
        run_kind[nrun] = kind;
        run_nsum[nrun] = nsum;
        if (kind != 0) {
          const int slot = 2 * c + (kind == 2);
          w.part_seg[slot] = g;
          w.part_cnt[slot] = s - rs + 1;
          w.part_nsum[slot] = nsum;
          w.part_end[slot] = ends;
        }
      }
#pragma unroll
      for (int e = 0; e < 2 * PPT; ++e) acc[e] = 0.0f;
      nsum = 0.0;
      rs = s + 1;
      ++nrun;
    }
  }
  __syncthreads();
  if (tid == 0) {
    bool head = false, tail = false;
    for (int k = 0; k < nrun; ++k) {
      head |= run_kind[k] == 1;
      tail |= run_kind[k] == 2;
    }
    if (!head) w.part_seg[2 * c] = -1;
    if (!tail) w.part_seg[2 * c + 1] = -1;
  }
  // renormalise whole buckets: E = sum * (mean member norm) / |sum|  (Eq. 7)
  for (int k = 0; k < nrun; ++k) {
    if (run_kind[k] != 0) continue;
    const float sq = (runsq[k][0] + runsq[k][1]) + (runsq[k][2] + runsq[k][3]);
    const double nrm = sqrt((double)sq);
    const float scale = nrm > 0.0 ? (float)(run_nsum[k] / ((double)run_len[k] * nrm)) : 0.0f;
    float* dst = E + (int64_t)run_g[k] * D;
#pragma unroll
    for (int q = 0; q < PPT; ++q) {
      const int p = tid + 256 * q;
      if (2 * p < D) {
        float2 v = *(float2*)(dst + 2 * p);
        *(float2*)(dst + 2 * p) = make_float2(v.x * scale, v.y * scale);
      }
    }
  }
}

template <int PPT>
__global__ __launch_bounds__(256) void k_mg_combine(MergeWS w, float* __restrict__ E,
                                                    int nchunks) {
  const int c = blockIdx.x, tid = threadIdx.x;
  const int D = w.D;
  const int g = w.part_seg[2 * c + 1];
  if (g < 0) return;
  __shared__ float red[4];
  float acc[2 * PPT];
#pragma unroll
  for (int q = 0; q < PPT; ++q) {
    const int p = tid + 256 * q;
    float2 v = (2 * p < D) ? *(const float2*)(w.part + (int64_t)(2 * c + 1) * D + 2 * p)
                           : make_float2(0.f, 0.f);
    acc[2 * q] = v.x;
    acc[2 * q + 1] = v.y;
  }
  int cnt = w.part_cnt[2 * c + 1];
  double nsum = w.part_nsum[2 * c + 1];
  for (int cc = c + 1; cc < nchunks; ++cc) {
    const int slot = 2 * cc;
    if (w.part_seg[slot] != g) break;
#pragma unroll
    for (int q = 0; q < PPT; ++q) {
      const int p = tid + 256 * q;
      if (2 * p < D) {
        float2 v = *(const float2*)(w.part + (int64_t)slot * D + 2 * p);
        acc[2 * q] += v.x;
        acc[2 * q + 1] += v.y;
      }
    }
    cnt += w.part_cnt[slot];
    nsum += w.part_nsum[slot];
    if (w.part_end[slot]) break;
  }
  float sq = 0.0f;
#pragma unroll
  for (int e = 0; e < 2 * PPT; ++e) sq += acc[e] * acc[e];
  sq = wave_sum_f32(sq);
  if ((tid & 63) == 0) red[tid >> 6] = sq;
  __syncthreads();
  const float tsq = (red[0] + red[1]) + (red[2] + red[3]);
  const double nrm = sqrt((double)tsq);
  const float scale = nrm > 0.0 ? (float)(nsum / ((double)cnt * nrm)) : 0.0f;
  float* dst = E + (int64_t)g * D;
#pragma unroll
  for (int q = 0; q < PPT; ++q) {
    const int p = tid + 256 * q;
    if (2 * p < D) *(float2*)(dst + 2 * p) = make_float2(acc[2 * q] * scale, acc[2 * q + 1] * scale);
  }
}

template <int DT, int PPT>
static void launch_reduce_combine(const MergeWS& w, const void* X, int64_t ldx, float* E,
                                  int nchunks, hipStream_t s) {
  hipLaunchKernelGGL((k_mg_reduce<DT, PPT>), dim3(nchunks), dim3(256), 0, s, w, X, ldx, E);
  hipLaunchKernelGGL((k_mg_combine<PPT>), dim3(nchunks), dim3(256), 0, s, w, E, nchunks);
}

template <int DT>
static void dispatch_ppt(const MergeWS& w, const void* X, int64_t ldx, float* E, int nchunks,
                         hipStream_t s) {
  const int ppt = (w.D / 2 + 255) / 256;
  if (ppt <= 1) launch_reduce_combine<DT, 1>(w, X, ldx, E, nchunks, s);
  else if (ppt <= 2) launch_reduce_combine<DT, 2>(w, X, ldx, E, nchunks, s);
  else if (ppt <= 4) launch_reduce_combine<DT, 4>(w, X, ldx, E, nchunks, s);
  else if (ppt <= 8) launch_reduce_combine<DT, 8>(w, X, ldx, E, nchunks, s);
  else launch_reduce_combine<DT, 16>(w, X, ldx, E, nchunks, s);
}

int merge_nchunks(int64_t N, int CH) { return (int)((N + CH - 1) / CH); }

hipError_t launch_merge(const MergeWS& w, const void* X, int dtype, int64_t ldx, float* E,
                        int* P, int* tok2macro, hipStream_t s) {
  (void)hipGetLastError();
  hipLaunchKernelGGL(k_mg_book, dim3(w.n_win), dim3(1024), 0, s, w);
  hipLaunchKernelGGL(k_mg_wbase, dim3(1), dim3(1024), 0, s, w);
  hipLaunchKernelGGL(k_mg_finalize, dim3((unsigned)((w.N + 255) / 256)), dim3(256), 0, s, w, P,
                     tok2macro);
  const int nchunks = merge_nchunks(w.N, w.CH);
  if (dtype == 0) dispatch_ppt<0>(w, X, ldx, E, nchunks, s);
  else dispatch_ppt<1>(w, X, ldx, E, nchunks, s);
  return hipGetLastError();
}

}  // namespace slh
