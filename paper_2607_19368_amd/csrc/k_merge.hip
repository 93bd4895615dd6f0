// Macro-token construction (Eq. 7, section 3.4 max positions, section 3.6
// ordering by representative position).
//
// book      one workgroup per window.  Windows of up to 16384 tokens are sorted
//           in one block (k_mg_book_lds: LSD radix sort of (code, token) keys
//           by code in LDS, 8 bits per pass, ranks by ballot matching);
//           longer ones use global memory.  Spectral windows: stable LSD radix sort
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
// All orders are fixed, so results are bitwise reproducible.  Every kernel
// that passes data between its own passes through global memory is one
// workgroup per window, so a workgroup-scope fence and a barrier order those
// passes (a device-scope fence writes back and invalidates the L2 each time);
// only the re-ranking kernel, whose histogram uses global atomics, keeps one.
#include "slh_device.h"
#include "slh_internal.h"

#include <climits>

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
    __threadfence_block();
    __syncthreads();
  }
  const uint32_t* K = kb[(npass - 1) & 1];
  const int* V = vb[(npass - 1) & 1];
  int* flag = w.tmpi + base;      // token order: 1 = bucket representative
  int* segid = w.segid + base;    // sorted order: bucket ordinal (by code)
  int* segk = w.segk + base;      // bucket ordinal -> macro rank
  for (int s = tid; s < L; s += 1024) flag[s] = 0;
  __threadfence_block();
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
  __threadfence_block();
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
  __threadfence_block();
  __syncthreads();
  for (int s = tid; s < L; s += 1024)
    if (s == L - 1 || K[s + 1] != K[s]) segk[segid[s]] = flag[V[s] - base];
  __threadfence_block();
  __syncthreads();
  for (int s = tid; s < L; s += 1024) {
    w.sval[base + s] = V[s];
    w.sloc[base + s] = segk[segid[s]];
  }
  if (tid == 0) w.mw[win] = nseg;
}

// Book-keeping of a window of L <= 16384 tokens in one 1024-thread block: sort
// the keys (code << tb) | local token (tb = log2 P, P = L rounded up to a power
// of two) by code, stably, so each bucket's members stay in token order; flag
// each bucket's last member, rank the representatives by an exclusive scan
// over tokens, and give every sorted position its bucket's rank.  Same outputs
// as k_mg_book.
//
// Sort: LSD radix on the code, 8 bits per pass (codes have at most 16 bits, so
// at most two passes), keys in LDS.  Each of the 16 waves owns a contiguous
// range of positions: it counts its digits into its row of a 16 x 256 table
// (LDS integer atomics), one scan over (digit, wave) turns the table into
// output offsets, and a second sweep, 64 positions at a time in order, finds
// the lanes of each digit (8 ballots); the group's lowest lane takes the
// group's offsets with one atomic add, and every key goes to that offset plus
// its rank among the earlier lanes of its group, which keeps the pass stable.  The
// sorted keys are then held E = max(P, 1024) / 1024 per thread (thread t:
// positions t E .. t E + E - 1): a bucket's last member is found from the next
// position's code (a neighbour shuffle), and each position's bucket end by a
// reverse scan over the block.  Dynamic LDS: two buffers of L keys (the second
// reused for the token ranks).
template <int E>
__global__ __launch_bounds__(1024) void k_mg_book_lds(MergeWS w, int P, int tb) {
  extern __shared__ uint32_t mg_dyn[];
  const int L = w.L;
  uint32_t* bufA = mg_dyn;                            // [L]
  uint32_t* bufB = mg_dyn + L;                        // [L]
  __shared__ int hw[16][256];                         // per wave: digit counts, then offsets
  __shared__ int wsum[16];
  __shared__ uint32_t wfirst[16];
  __shared__ int wend[16];
  const int win = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t base = (int64_t)win * L;
  if (!w.route[win]) {
    const int k = w.chunk_k;
    for (int s = tid; s < L; s += 1024) {
      w.sval[base + s] = (int)(base + s);
      w.sloc[base + s] = s / k;
    }
    if (tid == 0) w.mw[win] = (L + k - 1) / k;
    return;
  }
  (void)P;
  const uint32_t tmask = (1u << tb) - 1u;
  for (int i = tid; i < L; i += 1024) bufA[i] = (w.codes[base + i] << tb) | (uint32_t)i;

  const int npass = (w.bits + 7) / 8;
  const int span = (L + 15) / 16;                     // positions per wave
  const int p0 = min(wave * span, L), p1 = min(p0 + span, L);
  const uint64_t lt = (1ull << lane) - 1ull;          // lanes below this one
  uint32_t* src = bufA;
  uint32_t* dst = bufB;
  // lanes of this wave whose digit equals this lane's (valid lanes only)
  auto match = [&](int d, bool valid) {
    uint64_t m = __ballot(valid);
#pragma unroll
    for (int bit = 0; bit < 8; ++bit) {
      const bool on = (d >> bit) & 1;
      const uint64_t bb = __ballot(on);
      m &= on ? bb : ~bb;
    }
    return m;
  };
  for (int pass = 0; pass < npass; ++pass) {
    const int sh = tb + 8 * pass;
    for (int q = lane; q < 256; q += 64) hw[wave][q] = 0;
    __syncthreads();                                  // keys of the previous pass complete
    // counts need no order: integer adds, every chunk's in flight at once
    for (int i = p0 + lane; i < p1; i += 64) atomicAdd(&hw[wave][(src[i] >> sh) & 255u], 1);
    __syncthreads();
    // offsets: digits in order, waves in order within a digit
    int cnt[16], tot = 0;
    if (tid < 256) {
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        cnt[q] = hw[q][tid];
        tot += cnt[q];
      }
    }
    int total;
    const int incl = block_incl_scan_1024(tid < 256 ? tot : 0, wsum, total);
    if (tid < 256) {
      int off = incl - tot;
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        hw[q][tid] = off;
        off += cnt[q];
      }
    }
    __syncthreads();
    for (int c0 = p0; c0 < p1; c0 += 64) {
      const int i = c0 + lane;
      const bool valid = i < p1;
      const uint32_t k = src[min(i, L - 1)];
      const int d = (int)((k >> sh) & 255u);
      const uint64_t m = match(d, valid);
      int off = 0;
      if (valid && (m & lt) == 0)                     // the group's lowest lane
        off = atomicAdd(&hw[wave][d], __popcll(m));
      off = __shfl(off, (__ffsll((long long)m) - 1) & 63, 64);
      if (valid) dst[off + __popcll(m & lt)] = k;
    }
    uint32_t* t = src;
    src = dst;
    dst = t;
  }
  __syncthreads();                                    // sorted keys in src
  int* R = (int*)dst;                                 // [L] token -> rank
  uint32_t v[E];
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int pos = tid * E + e;
    v[e] = (pos < L) ? src[pos] : 0xFFFFFFFFu;
  }

  // run ends: position s < L ends its bucket when s = L - 1 or the next code differs
  if (lane == 0) wfirst[wave] = v[0];
  __syncthreads();
  uint32_t nx = (uint32_t)__shfl_down((int)v[0], 1, 64);
  if (lane == 63) nx = (wave < 15) ? wfirst[wave + 1] : 0xFFFFFFFFu;
  bool fl[E];
  int first_end = -1;                                // token of this thread's first run end
#pragma unroll
  for (int e = E - 1; e >= 0; --e) {
    const int s = tid * E + e;
    const uint32_t nxt = (e + 1 < E) ? v[e + 1] : nx;
    fl[e] = (s < L) && (s == L - 1 || (nxt >> tb) != (v[e] >> tb));
    if (fl[e]) first_end = (int)(v[e] & tmask);
  }
  // representative flags in token order (every token < L is written once)
#pragma unroll
  for (int e = 0; e < E; ++e)
    if (tid * E + e < L) R[v[e] & tmask] = fl[e] ? 1 : 0;
  __syncthreads();
  // exclusive scan over tokens: R[t] = number of representatives before t
  int fr[E], loc = 0;
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int t = tid * E + e;
    fr[e] = (t < L) ? R[t] : 0;
    loc += fr[e];
  }
  int tot;
  const int incl = block_incl_scan_1024(loc, wsum, tot);
  int run = incl - loc;
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int t = tid * E + e;
    if (t < L) R[t] = run;
    run += fr[e];
  }
  // bucket end of each position: the first run end at or after it (reverse
  // scan of first_end over the block; -1 = none)
  int sf = first_end;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int q = __shfl_down(sf, o, 64);
    if (lane + o < 64 && sf < 0) sf = q;
  }
  if (lane == 0) wend[wave] = sf;
  __syncthreads();                                   // also publishes R
  int tail = -1;                                     // first run end in a later wave
  for (int q = 15; q > wave; --q)
    if (wend[q] >= 0) tail = wend[q];
  const int full = (sf >= 0) ? sf : tail;
  int cur = __shfl_down(full, 1, 64);
  if (lane == 63) cur = tail;
#pragma unroll
  for (int e = E - 1; e >= 0; --e) {
    const int s = tid * E + e;
    if (fl[e]) cur = (int)(v[e] & tmask);
    if (s < L) {
      w.sval[base + s] = (int)(base + (v[e] & tmask));
      w.sloc[base + s] = R[cur];
    }
  }
  if (tid == 0) w.mw[win] = tot;
}

// inclusive max-scan of one int per thread over a 1024-thread block
__device__ __forceinline__ int block_incl_max_1024(int v, int* wsum, int& total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    int t = __shfl_up(v, o, 64);
    if (lane >= o) v = max(v, t);
  }
  __syncthreads();
  if (lane == 63) wsum[wave] = v;
  __syncthreads();
  int pre = INT_MIN, tot = INT_MIN;
  for (int k = 0; k < 16; ++k) {
    int x = wsum[k];
    if (k < wave) pre = max(pre, x);
    tot = max(tot, x);
  }
  total = tot;
  return max(v, pre);
}

// Scans of n values over a 1024-thread block, one block scan per 16384
// positions: thread t takes the contiguous positions c0 + t E .. c0 + t E + E - 1
// of each such chunk (E = ceil(chunk / 1024) <= 16), holding their values in
// registers.  val(i) gives position i's value, put(i, x) receives the exclusive
// prefix sum at i; returns the total.
template <class VAL, class PUT>
__device__ __forceinline__ int blocked_excl_sum(int n, VAL val, PUT put, int* wsum) {
  int carry = 0;
  for (int c0 = 0; c0 < n; c0 += 16384) {
    const int nc = min(16384, n - c0), E = (nc + 1023) >> 10, i0 = c0 + threadIdx.x * E;
    int v[16], loc = 0;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      v[e] = (e < E && i0 + e < c0 + nc) ? val(i0 + e) : 0;
      loc += v[e];
    }
    int tot;
    int run = carry + block_incl_scan_1024(loc, wsum, tot) - loc;
#pragma unroll
    for (int e = 0; e < 16; ++e)
      if (e < E && i0 + e < c0 + nc) {
        put(i0 + e, run);
        run += v[e];
      }
    carry += tot;
    __syncthreads();                                // wsum is reused
  }
  return carry;
}
// The same blocking for the most recent start at or before each position:
// put(i, s) receives the largest s <= i with is_start(s) (INT_MIN if none).
template <class START, class PUT>
__device__ __forceinline__ void blocked_last_start(int n, START is_start, PUT put, int* wsum) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int carry = INT_MIN;
  for (int c0 = 0; c0 < n; c0 += 16384) {
    const int nc = min(16384, n - c0), E = (nc + 1023) >> 10, i0 = c0 + threadIdx.x * E;
    bool f[16];
    int lm = INT_MIN;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      f[e] = e < E && i0 + e < c0 + nc && is_start(i0 + e);
      if (f[e]) lm = i0 + e;                       // starts increase with the position
    }
    // exclusive max over the threads before this one (and the earlier chunks)
    int v = lm;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int t = __shfl_up(v, o, 64);
      if (lane >= o) v = max(v, t);
    }
    int ex = __shfl_up(v, 1, 64);
    if (lane == 0) ex = INT_MIN;
    __syncthreads();
    if (lane == 63) wsum[wave] = v;
    __syncthreads();
    int tot = INT_MIN;
    for (int k = 0; k < 16; ++k) {
      if (k < wave) ex = max(ex, wsum[k]);
      tot = max(tot, wsum[k]);
    }
    int run = max(ex, carry);
#pragma unroll
    for (int e = 0; e < 16; ++e)
      if (e < E && i0 + e < c0 + nc) {
        if (f[e]) run = i0 + e;
        put(i0 + e, run);
      }
    carry = max(carry, tot);
    __syncthreads();                                // wsum is reused
  }
}

// inclusive scan (sum) of one int64 per thread over a 1024-thread block
__device__ __forceinline__ long long block_incl_scan_i64(long long v, long long* wsum,
                                                         long long& total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    long long t = __shfl_up(v, o, 64);
    if (lane >= o) v += t;
  }
  __syncthreads();
  if (lane == 63) wsum[wave] = v;
  __syncthreads();
  long long pre = 0, tot = 0;
  for (int k = 0; k < 16; ++k) {
    long long x = wsum[k];
    if (k < wave) pre += x;
    tot += x;
  }
  total = tot;
  return v + pre;
}

__device__ __forceinline__ int mg_scheme_pos(int scheme, int first, int cnt, long long sum,
                                             int median_pos, int max_pos) {
  if (scheme == 1) return median_pos;
  if (scheme == 2) {                             // mean, rounded half to even
    long long q = sum / cnt, rem = sum - q * cnt;
    if (2 * rem > cnt || (2 * rem == cnt && (q & 1))) ++q;
    return (int)q;
  }
  (void)first;
  return max_pos;
}

// Position schemes other than max (section 3.4): each bucket's representative
// position is the lower median (scheme 1) or the mean rounded half to even
// (scheme 2) of its member positions, and the buckets of a spectral window are
// re-ranked by (that position, max position).  One 1024-thread block per window;
// it reuses the book-keeping's sorted member order (sval: members of a bucket
// are a run of ascending tokens) and runs (sloc).  Writes posv[s] = global
// representative position at each run end s and rewrites sloc with the new
// ranks.  Scratch (window slices of N-entry arrays): st run start per sorted
// position, pre int64 prefix sums of member positions, tp per token the
// representative of the bucket whose last member it is (-1 otherwise), cnt a
// histogram of representative positions, hb its exclusive scan, rk the new rank
// at each run start.  Ties (mean only) are counted directly: tied buckets scan
// the window's tokens below their max position.
__global__ __launch_bounds__(1024) void k_mg_rerank(MergeWS w, int scheme, int* __restrict__ posv,
                                                    int* __restrict__ st, long long* __restrict__ pre,
                                                    int* __restrict__ tp, int* __restrict__ cnt,
                                                    int* __restrict__ hb, int* __restrict__ rk) {
  const int win = blockIdx.x, tid = threadIdx.x;
  const int L = w.L;
  const int64_t base = (int64_t)win * L;
  __shared__ int wsum[16];
  __shared__ long long wsum64[16];
  if (!w.route[win]) {
    // chunk groups of k consecutive tokens (sorted order = token order)
    const int k = w.chunk_k;
    for (int g = tid; g < (L + k - 1) / k; g += 1024) {
      const int s0 = g * k, s1 = min(s0 + k, L), n = s1 - s0;
      const long long sum = (long long)n * (s0 + s1 - 1) / 2;
      posv[base + s1 - 1] = (int)base + mg_scheme_pos(scheme, s0, n, sum, s0 + (n - 1) / 2, s1 - 1);
    }
    return;
  }
  // run starts (max-scan of start indices) and prefix sums of member positions
  int carry = INT_MIN;
  long long csum = 0;
  for (int b0 = 0; b0 < L; b0 += 1024) {
    const int s = b0 + tid;
    int v = INT_MIN;
    long long pv = 0;
    if (s < L) {
      v = (s == 0 || w.sloc[base + s] != w.sloc[base + s - 1]) ? s : INT_MIN;
      pv = w.sval[base + s] - base;
    }
    int tot;
    long long tot64;
    const int inc = block_incl_max_1024(v, wsum, tot);
    const long long pinc = block_incl_scan_i64(pv, wsum64, tot64);
    if (s < L) {
      st[base + s] = max(inc, carry);
      pre[base + s] = csum + pinc;
    }
    carry = max(carry, tot);
    csum += tot64;
    __syncthreads();
  }
  for (int t = tid; t < L; t += 1024) {
    tp[base + t] = -1;
    cnt[base + t] = 0;
  }
  __threadfence_block();
  __syncthreads();
  // representative positions at run ends; histogram of them
  for (int e = tid; e < L; e += 1024) {
    if (e == L - 1 || w.sloc[base + e + 1] != w.sloc[base + e]) {
      const int s0 = st[base + e], n = e - s0 + 1;
      const long long sum = pre[base + e] - (s0 > 0 ? pre[base + s0 - 1] : 0);
      const int mx = w.sval[base + e] - (int)base;
      const int med = w.sval[base + s0 + (n - 1) / 2] - (int)base;
      const int p = mg_scheme_pos(scheme, s0, n, sum, med, mx);
      posv[base + e] = (int)base + p;
      tp[base + mx] = p;
      atomicAdd(&cnt[base + p], 1);
    }
  }
  __threadfence();
  __syncthreads();
  // buckets with a smaller representative position: exclusive scan of cnt
  int c2 = 0;
  for (int b0 = 0; b0 < L; b0 += 1024) {
    const int p = b0 + tid;
    const int v = (p < L) ? cnt[base + p] : 0;
    int tot;
    const int inc = block_incl_scan_1024(v, wsum, tot);
    if (p < L) hb[base + p] = c2 + inc - v;
    c2 += tot;
    __syncthreads();
  }
  __threadfence_block();
  __syncthreads();
  // rank = buckets with a smaller position + tied buckets with a smaller max
  for (int e = tid; e < L; e += 1024) {
    if (e == L - 1 || w.sloc[base + e + 1] != w.sloc[base + e]) {
      const int p = posv[base + e] - (int)base;
      const int mx = w.sval[base + e] - (int)base;
      int r = hb[base + p];
      if (cnt[base + p] > 1)
        for (int t = 0; t < mx; ++t) r += (tp[base + t] == p);
      rk[base + st[base + e]] = r;
    }
  }
  __threadfence_block();
  __syncthreads();
  for (int s = tid; s < L; s += 1024) w.sloc[base + s] = rk[base + st[base + s]];
}

// Exact target length (section 3.3: clusters are merged or split until their
// number matches the target; the paper gives no algorithm, so this follows one
// fixed reading).  Window budget T = w.tw[win] (> 0 for spectral windows); one
// block per window, after the book-keeping (sval: members by code, then token;
// sloc: macro rank by max position; mw: count M).
//   M > T: macro k joins new macro floor(k T / M) (runs of consecutive
//          macro-tokens in position order); members are regrouped, buckets in
//          rank order, so each new macro is a contiguous run ending with its
//          max-position member.
//   M < T: E = T - M extra pieces are apportioned in proportion to s_k - 1:
//          floor(E (s_k - 1) / (L - M)) each, then one more for the largest
//          remainders (ties: smaller k; ranked by direct counting); bucket k is
//          cut into n_k contiguous pieces of its member run (the first s mod n
//          of ceil(s / n) members), and pieces are ranked by their last member
//          with a scan over the window's tokens.
// Scratch (window slices of N-entry arrays): st run start per sorted position,
// rsz / rof size and start of rank k's run, t0 / t1 / fl int work arrays, rem
// int64 remainders.
__global__ __launch_bounds__(1024) void k_mg_target(MergeWS w, int* __restrict__ st,
                                                    int* __restrict__ rsz, int* __restrict__ rof,
                                                    int* __restrict__ t0, int* __restrict__ t1,
                                                    int* __restrict__ fl, long long* __restrict__ rem) {
  const int win = blockIdx.x, tid = threadIdx.x;
  const int L = w.L;
  const int64_t base = (int64_t)win * L;
  if (!w.route[win]) return;
  const int T = w.tw[win], M = w.mw[win];
  if (T <= 0 || T == M) return;
  __shared__ int wsum[16];
  __shared__ int sR;
  // run starts: the most recent start of a run at or before each sorted position
  blocked_last_start(L, [&](int s) { return s == 0 || w.sloc[base + s] != w.sloc[base + s - 1]; },
                     [&](int s, int x) { st[base + s] = x; }, wsum);
  __threadfence_block();
  __syncthreads();
  for (int e = tid; e < L; e += 1024)
    if (e == L - 1 || w.sloc[base + e + 1] != w.sloc[base + e]) {
      const int k = w.sloc[base + e];
      rsz[base + k] = e - st[base + e] + 1;
      rof[base + k] = st[base + e];
    }
  __threadfence_block();
  __syncthreads();
  if (M > T) {
    // exclusive prefix of the run sizes over ranks: new sorted position of each
    // bucket's first member
    (void)blocked_excl_sum(M, [&](int k) { return rsz[base + k]; },
                           [&](int k, int x) { t0[base + k] = x; }, wsum);
    __threadfence_block();
    __syncthreads();
    for (int s = tid; s < L; s += 1024) {
      const int k = w.sloc[base + s];
      const int dest = t0[base + k] + (s - st[base + s]);
      t1[base + dest] = w.sval[base + s];
      fl[base + dest] = (int)((long long)k * T / M);
    }
    __threadfence_block();
    __syncthreads();
    for (int s = tid; s < L; s += 1024) {
      w.sval[base + s] = t1[base + s];
      w.sloc[base + s] = fl[base + s];
    }
  } else {
    const int E = T - M;
    const long long den = (long long)L - M;      // > 0: a window with M = L has T <= L = M
    int part = 0;
    for (int k = tid; k < M; k += 1024) {
      const long long num = (long long)E * (rsz[base + k] - 1);
      t0[base + k] = (int)(num / den);
      rem[base + k] = num % den;
      part += (int)(num / den);
    }
    int tot;
    (void)block_incl_scan_1024(part, wsum, tot);
    if (tid == 0) sR = E - tot;
    __threadfence_block();
    __syncthreads();
    const int R = sR;
    // pieces per bucket: one more for the R largest remainders (ties: smaller k)
    for (int k = tid; k < M; k += 1024) {
      const long long rk = rem[base + k];
      int ahead = 0;
      if (R > 0)
        for (int q = 0; q < M; ++q) {
          const long long rq = rem[base + q];
          ahead += (rq > rk) || (rq == rk && q < k);
        }
      // at most one piece per member (guaranteed by the apportionment; kept as a bound)
      t1[base + k] = min(rsz[base + k], 1 + t0[base + k] + ((R > 0 && ahead < R) ? 1 : 0));
    }
    for (int t = tid; t < L; t += 1024) fl[base + t] = 0;
    __threadfence_block();
    __syncthreads();
    // flag each piece's last member (by token)
    for (int s = tid; s < L; s += 1024) {
      const int k = w.sloc[base + s];
      const int sz = rsz[base + k], n = t1[base + k];
      const int q = sz / n, rr = sz % n, o = s - st[base + s];
      const int j = (o < rr * (q + 1)) ? o / (q + 1) : rr + (o - rr * (q + 1)) / q;
      const int last = (j < rr) ? (j + 1) * (q + 1) - 1 : rr * (q + 1) + (j - rr + 1) * q - 1;
      if (o == last) fl[w.sval[base + s]] = 1;
    }
    __threadfence_block();
    __syncthreads();
    // rank of each piece = pieces whose last member precedes its own
    (void)blocked_excl_sum(L, [&](int t) { return fl[base + t]; },
                           [&](int t, int x) { t0[base + t] = x; }, wsum);
    __threadfence_block();
    __syncthreads();
    for (int s = tid; s < L; s += 1024) {
      const int k = w.sloc[base + s];
      const int sz = rsz[base + k], n = t1[base + k];
      const int q = sz / n, rr = sz % n, o = s - st[base + s];
      const int j = (o < rr * (q + 1)) ? o / (q + 1) : rr + (o - rr * (q + 1)) / q;
      const int last = (j < rr) ? (j + 1) * (q + 1) - 1 : rr * (q + 1) + (j - rr + 1) * q - 1;
      const int ltok = w.sval[base + rof[base + k] + last];
      fl[base + s] = t0[ltok];
    }
    __threadfence_block();
    __syncthreads();
    for (int s = tid; s < L; s += 1024) w.sloc[base + s] = fl[base + s];
  }
  if (tid == 0) w.mw[win] = T;
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
  if (end) P[g] = w.compact ? g : (w.posv ? w.posv[s] : tok);
}

// Member rows are read 8 columns per thread (one 16-byte load for bf16, two
// for fp32) by 512 threads, PPT passes of 4096 columns; D % 8 == 0.
template <int DT> struct MgRaw;
template <> struct MgRaw<0> { uint4 v; };
template <> struct MgRaw<1> { float4 lo, hi; };

template <int DT>
__device__ __forceinline__ MgRaw<DT> mg_load(const void* X, int64_t ldx, int tok, int col) {
  MgRaw<DT> r;
  if constexpr (DT == 0) {
    r.v = *(const uint4*)((const uint16_t*)X + (int64_t)tok * ldx + col);
  } else {
    const float4* p = (const float4*)((const float*)X + (int64_t)tok * ldx + col);
    r.lo = p[0];
    r.hi = p[1];
  }
  return r;
}

template <int DT>
__device__ __forceinline__ void mg_add(float* acc, const MgRaw<DT>& r) {
  if constexpr (DT == 0) {
    const uint32_t u[4] = {r.v.x, r.v.y, r.v.z, r.v.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      acc[2 * e] += __uint_as_float(u[e] << 16);
      acc[2 * e + 1] += __uint_as_float(u[e] & 0xFFFF0000u);
    }
  } else {
    acc[0] += r.lo.x; acc[1] += r.lo.y; acc[2] += r.lo.z; acc[3] += r.lo.w;
    acc[4] += r.hi.x; acc[5] += r.hi.y; acc[6] += r.hi.z; acc[7] += r.hi.w;
  }
}

__device__ __forceinline__ void mg_store8(float* dst, const float* v, float scale) {
  ((float4*)dst)[0] = make_float4(v[0] * scale, v[1] * scale, v[2] * scale, v[3] * scale);
  ((float4*)dst)[1] = make_float4(v[4] * scale, v[5] * scale, v[6] * scale, v[7] * scale);
}

// Sum over the 512 threads of one float per thread (fixed order); `red` holds
// 8 floats; all threads get the result.  Contains one barrier.
__device__ __forceinline__ float mg_block_sum(float v, float* red) {
  v = wave_sum_f32(v);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  return ((red[0] + red[1]) + (red[2] + red[3])) + ((red[4] + red[5]) + (red[6] + red[7]));
}

// One workgroup per chunk of CH sorted positions; member rows stream DEPTH at
// a time with the next DEPTH in flight (DEPTH sized to keep the row buffers at
// 64 registers).
template <int DT, int PPT>
__global__ __launch_bounds__(512) void k_mg_reduce(MergeWS w, const void* __restrict__ X,
                                                   int64_t ldx, float* __restrict__ E) {
  const int c = blockIdx.x, tid = threadIdx.x;
  const int D = w.D;
  const int64_t s0 = (int64_t)c * w.CH;
  const int n = (int)min((int64_t)w.CH, w.N - s0);
  __shared__ int ssv[MG_CHMAX], ssg[MG_CHMAX];
  __shared__ double snrm[MG_CHMAX];
  __shared__ int prev_g, next_g;
  __shared__ float red[2][8];
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
  int col[PPT];
  bool cin[PPT];
#pragma unroll
  for (int q = 0; q < PPT; ++q) {
    const int c8 = 8 * (tid + 512 * q);
    cin[q] = c8 < D;
    col[q] = min(c8, D - 8);
  }
  float acc[PPT][8];
#pragma unroll
  for (int q = 0; q < PPT; ++q)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[q][e] = 0.0f;
  constexpr int DEPTH = (8 / (PPT * (DT + 1))) > 0 ? 8 / (PPT * (DT + 1)) : 1;
  MgRaw<DT> rc[DEPTH][PPT], rn[DEPTH][PPT];
  auto load_batch = [&](MgRaw<DT> (&dst)[DEPTH][PPT], int b) {
#pragma unroll
    for (int e = 0; e < DEPTH; ++e) {
      const int tok = ssv[min(DEPTH * b + e, n - 1)];
#pragma unroll
      for (int q = 0; q < PPT; ++q) dst[e][q] = mg_load<DT>(X, ldx, tok, col[q]);
    }
  };
  double nsum = 0.0;
  int rs = 0, par = 0;
  bool had_head = false, had_tail = false;
  const int nbat = (n + DEPTH - 1) / DEPTH;
  load_batch(rc, 0);
  for (int b = 0; b < nbat; ++b) {
    if (b + 1 < nbat) load_batch(rn, b + 1);
#pragma unroll
    for (int e = 0; e < DEPTH; ++e) {
      const int s = DEPTH * b + e;
      if (s < n) {
#pragma unroll
        for (int q = 0; q < PPT; ++q)
          if (cin[q]) mg_add<DT>(acc[q], rc[e][q]);
        nsum += snrm[s];
        const int g = ssg[s];
        if (s == n - 1 || ssg[s + 1] != g) {
          const bool starts = (rs > 0) || (prev_g != g);
          const bool ends = (s < n - 1) || (next_g != g);
          // kind 0: whole bucket -> E (Eq. 7 renormalisation: sum * mean member norm / |sum|);
          // 1: head partial (slot 2c); 2: tail partial (slot 2c+1)
          const int kind = (starts && ends) ? 0 : (!starts ? 1 : 2);
          if (kind == 0) {
            float sq = 0.0f;
#pragma unroll
            for (int q = 0; q < PPT; ++q)
              if (cin[q])
#pragma unroll
                for (int k = 0; k < 8; ++k) sq += acc[q][k] * acc[q][k];
            const float tsq = mg_block_sum(sq, red[par]);
            par ^= 1;
            const double nrm = sqrt((double)tsq);
            const float scale = nrm > 0.0 ? (float)(nsum / ((double)(s - rs + 1) * nrm)) : 0.0f;
            float* dst = E + (int64_t)g * D;
#pragma unroll
            for (int q = 0; q < PPT; ++q)
              if (cin[q]) mg_store8(dst + col[q], acc[q], scale);
          } else {
            const int slot = 2 * c + (kind == 2);
            float* dst = w.part + (int64_t)slot * D;
#pragma unroll
            for (int q = 0; q < PPT; ++q)
              if (cin[q]) mg_store8(dst + col[q], acc[q], 1.0f);
            if (tid == 0) {
              w.part_seg[slot] = g;
              w.part_cnt[slot] = s - rs + 1;
              w.part_nsum[slot] = nsum;
              w.part_end[slot] = ends;
            }
            had_head |= kind == 1;
            had_tail |= kind == 2;
          }
#pragma unroll
          for (int q = 0; q < PPT; ++q)
#pragma unroll
            for (int k = 0; k < 8; ++k) acc[q][k] = 0.0f;
          nsum = 0.0;
          rs = s + 1;
        }
      }
    }
#pragma unroll
    for (int e = 0; e < DEPTH; ++e)
#pragma unroll
      for (int q = 0; q < PPT; ++q) rc[e][q] = rn[e][q];
  }
  if (tid == 0) {
    if (!had_head) w.part_seg[2 * c] = -1;
    if (!had_tail) w.part_seg[2 * c + 1] = -1;
  }
}

// A bucket cut by chunk edges: its tail partial in chunk c plus the head
// partials of chunks c+1 .. last, summed in chunk order (8 / PPT rows in flight),
// then renormalised.
template <int PPT>
__global__ __launch_bounds__(512) void k_mg_combine(MergeWS w, float* __restrict__ E,
                                                    int nchunks) {
  const int c = blockIdx.x, tid = threadIdx.x;
  const int D = w.D;
  const int g = w.part_seg[2 * c + 1];
  if (g < 0) return;
  __shared__ int s_last;
  __shared__ float red[8];
  __shared__ double dred[8];
  __shared__ int ired[8];
  // last chunk of the chain: the first cc > c whose head slot belongs to another
  // macro (then cc - 1) or ends the bucket (then cc)
  int last = nchunks - 1;
  for (int base = c + 1; base < nchunks; base += 512) {
    const int cc = base + tid;
    int x = nchunks - 1;
    if (cc < nchunks) {
      if (w.part_seg[2 * cc] != g) x = cc - 1;
      else if (w.part_end[2 * cc]) x = cc;
    }
    for (int o = 32; o >= 1; o >>= 1) x = min(x, __shfl_xor(x, o, 64));
    if ((tid & 63) == 0) ired[tid >> 6] = x;
    __syncthreads();
    if (tid == 0) {
      int m = ired[0];
      for (int k = 1; k < 8; ++k) m = min(m, ired[k]);
      s_last = m;
    }
    __syncthreads();
    last = s_last;
    if (last < base + 511) break;
    __syncthreads();
  }
  int col[PPT];
  bool cin[PPT];
#pragma unroll
  for (int q = 0; q < PPT; ++q) {
    const int c8 = 8 * (tid + 512 * q);
    cin[q] = c8 < D;
    col[q] = min(c8, D - 8);
  }
  float acc[PPT][8];
  {
    const float* src = w.part + (int64_t)(2 * c + 1) * D;
#pragma unroll
    for (int q = 0; q < PPT; ++q) {
      const MgRaw<1> r = mg_load<1>(src, 0, 0, col[q]);
      acc[q][0] = r.lo.x; acc[q][1] = r.lo.y; acc[q][2] = r.lo.z; acc[q][3] = r.lo.w;
      acc[q][4] = r.hi.x; acc[q][5] = r.hi.y; acc[q][6] = r.hi.z; acc[q][7] = r.hi.w;
    }
  }
  // head partials of chunks c+1 .. last, DEPTH at a time
  constexpr int DEPTH = (8 / PPT) > 0 ? 8 / PPT : 1;
  for (int cc0 = c + 1; cc0 <= last; cc0 += DEPTH) {
    MgRaw<1> r[DEPTH][PPT];
#pragma unroll
    for (int e = 0; e < DEPTH; ++e) {
      const float* src = w.part + (int64_t)(2 * min(cc0 + e, last)) * D;
#pragma unroll
      for (int q = 0; q < PPT; ++q) r[e][q] = mg_load<1>(src, 0, 0, col[q]);
    }
#pragma unroll
    for (int e = 0; e < DEPTH; ++e)
      if (cc0 + e <= last)
#pragma unroll
        for (int q = 0; q < PPT; ++q) mg_add<1>(acc[q], r[e][q]);
  }
  // member count and norm sum over the same slots (fixed order)
  int cnt = 0;
  double nsum = 0.0;
  for (int cc = c + 1 + tid; cc <= last; cc += 512) {
    cnt += w.part_cnt[2 * cc];
    nsum += w.part_nsum[2 * cc];
  }
  cnt = wave_sum_i32(cnt);
  nsum = wave_sum_f64(nsum);
  if ((tid & 63) == 0) {
    ired[tid >> 6] = cnt;
    dred[tid >> 6] = nsum;
  }
  float sq = 0.0f;
#pragma unroll
  for (int q = 0; q < PPT; ++q)
    if (cin[q])
#pragma unroll
      for (int k = 0; k < 8; ++k) sq += acc[q][k] * acc[q][k];
  const float tsq = mg_block_sum(sq, red);       // its barrier also publishes ired / dred
  int tcnt = w.part_cnt[2 * c + 1];
  double tns = w.part_nsum[2 * c + 1];
  for (int k = 0; k < 8; ++k) {
    tcnt += ired[k];
    tns += dred[k];
  }
  const double nrm = sqrt((double)tsq);
  const float scale = nrm > 0.0 ? (float)(tns / ((double)tcnt * nrm)) : 0.0f;
  float* dst = E + (int64_t)g * D;
#pragma unroll
  for (int q = 0; q < PPT; ++q)
    if (cin[q]) mg_store8(dst + col[q], acc[q], scale);
}

template <int DT, int PPT>
static void launch_reduce_combine(const MergeWS& w, const void* X, int64_t ldx, float* E,
                                  int nchunks, hipStream_t s) {
  hipLaunchKernelGGL((k_mg_reduce<DT, PPT>), dim3(nchunks), dim3(512), 0, s, w, X, ldx, E);
  hipLaunchKernelGGL((k_mg_combine<PPT>), dim3(nchunks), dim3(512), 0, s, w, E, nchunks);
}

template <int DT>
static void dispatch_ppt(const MergeWS& w, const void* X, int64_t ldx, float* E, int nchunks,
                         hipStream_t s) {
  const int ppt = (w.D + 4095) / 4096;
  if (ppt <= 1) launch_reduce_combine<DT, 1>(w, X, ldx, E, nchunks, s);
  else if (ppt <= 2) launch_reduce_combine<DT, 2>(w, X, ldx, E, nchunks, s);
  else if (ppt <= 4) launch_reduce_combine<DT, 4>(w, X, ldx, E, nchunks, s);
  else launch_reduce_combine<DT, 8>(w, X, ldx, E, nchunks, s);      // D <= 32768
}

// Preserved suffix (section 3.5: every backend can keep a fixed number of final
// tokens as they are; section 5.1: the last 12 by default): tail token N + t
// becomes macro-token M + t with its own row (Eq. 7 on one row gives the row)
// and position N + t (M + t in compact mode); M = the compressed part's count.
template <int DT>
__global__ __launch_bounds__(256) void k_mg_tail(const void* __restrict__ X, int64_t ldx, int D,
                                                 int64_t N, const int* __restrict__ Mtot,
                                                 int compact, float* __restrict__ E,
                                                 int* __restrict__ P, int* __restrict__ tok2macro) {
  const int t = blockIdx.x;
  const int M = *Mtot;
  const int64_t tok = N + t;
  float* dst = E + (int64_t)(M + t) * D;
  for (int c = threadIdx.x; c < D; c += 256) {
    if constexpr (DT == 0) dst[c] = bf16_to_f32(((const uint16_t*)X)[tok * ldx + c]);
    else dst[c] = ((const float*)X)[tok * ldx + c];
  }
  if (threadIdx.x == 0) {
    P[M + t] = compact ? M + t : (int)tok;
    if (tok2macro) tok2macro[tok] = M + t;
  }
}

// M and the resident Lanczos kernel's error word (0 without it) into host-pinned
// memory, in place of two copies; the event the host waits on is recorded after
// this kernel, and its system-scope release makes the two words visible
__global__ void k_mg_report(const int* __restrict__ Mtot, const unsigned* __restrict__ err,
                            unsigned* __restrict__ out) {
  out[0] = (unsigned)*Mtot;
  out[1] = err ? *err : 0u;
}

hipError_t launch_merge_report(const int* Mtot, const unsigned* err, unsigned* out, hipStream_t s) {
  (void)hipGetLastError();
  hipLaunchKernelGGL(k_mg_report, dim3(1), dim3(1), 0, s, Mtot, err, out);
  return hipGetLastError();
}

hipError_t launch_merge_tail(const void* X, int dtype, int64_t ldx, int D, int64_t N, int K,
                             const int* Mtot, int compact, float* E, int* P, int* tok2macro,
                             hipStream_t s) {
  (void)hipGetLastError();
  if (K <= 0) return hipSuccess;
  if (dtype == 0)
    hipLaunchKernelGGL(k_mg_tail<0>, dim3(K), dim3(256), 0, s, X, ldx, D, N, Mtot, compact, E, P,
                       tok2macro);
  else
    hipLaunchKernelGGL(k_mg_tail<1>, dim3(K), dim3(256), 0, s, X, ldx, D, N, Mtot, compact, E, P,
                       tok2macro);
  return hipGetLastError();
}

int merge_nchunks(int64_t N, int CH) { return (int)((N + CH - 1) / CH); }

hipError_t launch_merge(const MergeWS& w, const void* X, int dtype, int64_t ldx, float* E,
                        int* P, int* tok2macro, hipStream_t s) {
  (void)hipGetLastError();
  if (w.L <= 16384) {
    int P = 1, tb = 0;
    while (P < w.L) {
      P <<= 1;
      ++tb;
    }
    const int Pp = P > 1024 ? P : 1024;
    const size_t bytes = (size_t)2 * w.L * 4;
    const void* kf = (Pp == 1024)   ? (const void*)k_mg_book_lds<1>
                     : (Pp == 2048) ? (const void*)k_mg_book_lds<2>
                     : (Pp == 4096) ? (const void*)k_mg_book_lds<4>
                     : (Pp == 8192) ? (const void*)k_mg_book_lds<8>
                                    : (const void*)k_mg_book_lds<16>;
    if (bytes > 65536) {
      const hipError_t e = hipFuncSetAttribute(kf, hipFuncAttributeMaxDynamicSharedMemorySize,
                                               (int)bytes);
      if (e != hipSuccess) return e;
    }
    switch (Pp) {
      case 1024: hipLaunchKernelGGL(k_mg_book_lds<1>, dim3(w.n_win), dim3(1024), bytes, s, w, P, tb); break;
      case 2048: hipLaunchKernelGGL(k_mg_book_lds<2>, dim3(w.n_win), dim3(1024), bytes, s, w, P, tb); break;
      case 4096: hipLaunchKernelGGL(k_mg_book_lds<4>, dim3(w.n_win), dim3(1024), bytes, s, w, P, tb); break;
      case 8192: hipLaunchKernelGGL(k_mg_book_lds<8>, dim3(w.n_win), dim3(1024), bytes, s, w, P, tb); break;
      default: hipLaunchKernelGGL(k_mg_book_lds<16>, dim3(w.n_win), dim3(1024), bytes, s, w, P, tb); break;
    }
  } else {
    hipLaunchKernelGGL(k_mg_book, dim3(w.n_win), dim3(1024), 0, s, w);
  }
  if (w.tw)
    hipLaunchKernelGGL(k_mg_target, dim3(w.n_win), dim3(1024), 0, s, w, w.valA, w.segid, w.segk,
                       (int*)w.keyA, (int*)w.keyB, w.tg, w.pre);
  if (w.scheme != 0)
    hipLaunchKernelGGL(k_mg_rerank, dim3(w.n_win), dim3(1024), 0, s, w, w.scheme, w.posv, w.valA,
                       w.pre, w.tmpi, w.segid, w.segk, w.valB);
  hipLaunchKernelGGL(k_mg_wbase, dim3(1), dim3(1024), 0, s, w);
  hipLaunchKernelGGL(k_mg_finalize, dim3((unsigned)((w.N + 255) / 256)), dim3(256), 0, s, w, P,
                     tok2macro);
  const int nchunks = merge_nchunks(w.N, w.CH);
  if (dtype == 0) dispatch_ppt<0>(w, X, ldx, E, nchunks, s);
  else dispatch_ppt<1>(w, X, ldx, E, nchunks, s);
  return hipGetLastError();
}

}  // namespace slh
