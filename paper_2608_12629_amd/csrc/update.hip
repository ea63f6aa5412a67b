// update.hip -- the centroid update of the Lloyd iteration (paper Section 5:
// reduce the points of each cluster into per-cluster sums and counts).
//
// The paper calls this step bandwidth- and atomic-contention-sensitive.  Here
// it uses no floating-point atomics and is deterministic:
//   1. a stable radix sort of the point ids by cluster id (one or two passes of
//      histogram, scan and LDS-staged scatter; see below)
//   2. bounds     per cluster, its run [off_k, off_k+1) in the sorted order
//                 (after two packed passes: read off the second pass's
//                 histogram, no sorted keys needed)
//   3. segreduce  one wave per slice of consecutive sorted entries streams the
//                 whole rows X[perm[j]] and sums each cluster run in fp32 in a
//                 fixed order; a run cut by a chunk end leaves a partial
//   4. finalize   per cluster, the sum (or its partials, in chunk order) over
//                 the count; an empty cluster keeps its previous centroid.
#include <algorithm>

#include "fkm_device.h"

namespace fkm {

// ---------------------------------------------------------------------------
// Stable LSD radix sort of (cluster id, point id) by cluster id: one pass per
// digit of at most 8 bits (two passes for K <= 65536).  Each pass:
//   radix_hist     per chunk of RADIX_CHUNK entries, a histogram over the R bins
//   radix_scan     per bin, exclusive scan over chunks (+ the bin total); the
//                  scatter adds the bin's start to get each (bin, chunk) run start
//   radix_scatter  per chunk, four waves rank their quarters in entry order
//                  (ballot multi-split), stage the chunk sorted by bin in LDS,
//                  and write each bin's run out contiguously (coalesced)
// Pass one reads the assignment itself and ignores ids outside [0, K).
namespace {

__device__ __forceinline__ int digit_of(int key, int shift, int R) { return (key >> shift) & (R - 1); }

static_assert(RADIX_MAX_R == 256, "the scans give each bin one thread of a 256-thread workgroup");

// Exclusive scan of one value per thread over a workgroup of W waves: a
// shuffle scan inside each wave, then the wave totals through `wsum` (one
// barrier).  Returns the exclusive prefix; `total` gets the sum.
template <int W>
__device__ __forceinline__ int block_scan(int v, int* wsum, int& total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int x = v;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int y = __shfl_up(x, d);
    if (lane >= d) x += y;
  }
  if (lane == 63) wsum[w] = x;
  __syncthreads();
  int pre = 0;
  total = 0;
#pragma unroll
  for (int i = 0; i < W; ++i) {
    const int s = wsum[i];
    pre += i < w ? s : 0;
    total += s;
  }
  return pre + x - v;
}
__device__ __forceinline__ int block_scan256(int v, int* wsum, int& total) {
  return block_scan<4>(v, wsum, total);
}

// The second packed pass cuts each bin of the first pass (the entries with one
// low digit, contiguous after that pass: bin r holds T1[r] entries from its
// start) into chunks of at most RADIX_CHUNK entries, ceil(T1[r] / RADIX_CHUNK)
// of them, numbered bin by bin, so every chunk holds a single low digit.
// Chunk `ch` of instance b: entries [e0, e1) with low digit `lo` (an empty
// range past the last chunk).  sel[3..4] get the low digits whose first chunk
// (cq, the chunks before the digit's) is `ch`: the digit of a chunk that
// starts one and the empty digits just before it, or past the last chunk the
// empty digits at the end (an empty range: sel[3] > sel[4] otherwise).
// Called by all 256 threads; wsum: 8 ints, sel: 5.
__device__ inline void lo_chunk(const int32_t* __restrict__ T1, int b, int R1, int ch, int* wsum,
                                int* sel, int& e0, int& e1, int& lo) {
  const int t = threadIdx.x;
  const int cnt = t < R1 ? T1[(size_t)b * RADIX_MAX_R + t] : 0;
  const int q = (cnt + RADIX_CHUNK - 1) / RADIX_CHUNK;
  int all;
  const int start = block_scan256(cnt, wsum, all);
  const int cq = block_scan256(q, wsum + 4, all);
  if (t == 0) {
    sel[0] = sel[1] = sel[2] = 0;
    sel[3] = R1;
    sel[4] = -1;
  }
  __syncthreads();
  if (q > 0 && cq <= ch && ch < cq + q) {  // one thread at most
    const int a = start + (ch - cq) * RADIX_CHUNK;
    sel[0] = a;
    sel[1] = min(a + RADIX_CHUNK, start + cnt);
    sel[2] = t;
  }
  if (t < R1 && cq == ch) {  // cq is non-decreasing in t: a run of threads
    atomicMin(&sel[3], t);
    atomicMax(&sel[4], t);
  }
  __syncthreads();
  e0 = sel[0];
  e1 = sel[1];
  lo = sel[2];
}

}  // namespace

// pb > 0: the entries are packed words (digit above pb point-id bits) in the
// chunks of lo_chunk (T1: the first pass's bin totals).
__global__ __launch_bounds__(256) void radix_hist_kernel(const int32_t* __restrict__ keys, int N,
                                                         int K, const int32_t* __restrict__ total,
                                                         int shift, int R, int nch,
                                                         int32_t* __restrict__ H, int pb,
                                                         const int32_t* __restrict__ T1,
                                                         int lo_bits) {
  __shared__ int cnt[RADIX_MAX_R];
  __shared__ int wsum[8], sel[5];
  const int b = blockIdx.y, ch = blockIdx.x, t = threadIdx.x;
  int e0, e1, lo;
  if (pb) {
    lo_chunk(T1, b, 1 << lo_bits, ch, wsum, sel, e0, e1, lo);
  } else {
    const int n_in = total ? total[b] : N;  // later passes read the valid prefix only
    e0 = ch * RADIX_CHUNK;
    e1 = min(e0 + RADIX_CHUNK, n_in);
  }
  for (int r = t; r < R; r += 256) cnt[r] = 0;
  __syncthreads();
  const int32_t* kb = keys + (size_t)b * N;
  constexpr int PER = RADIX_CHUNK / 256;
  int k[PER];
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    const int i = e0 + u * 256 + t;
    k[u] = i < e1 ? kb[i] : -1;
  }
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    if (pb) {
      if (k[u] >= 0) atomicAdd(&cnt[(k[u] >> pb) & (R - 1)], 1);
    } else if ((unsigned)k[u] < (unsigned)K) {
      atomicAdd(&cnt[digit_of(k[u], shift, R)], 1);
    }
  }
  __syncthreads();
  for (int r = t; r < R; r += 256) H[((size_t)b * R + r) * nch + ch] = cnt[r];
}

// Per bin (one workgroup each): exclusive scan of the bin's chunk counts in
// place, and the bin total into T[b][bin].  Bin starts are the exclusive scan
// of T, done by each scatter workgroup on its own (R <= 256 values).
__global__ __launch_bounds__(256) void radix_scan_kernel(int32_t* __restrict__ H, int R, int nch,
                                                         int32_t* __restrict__ T) {
  __shared__ int wsum[4];
  const int r = blockIdx.x, b = blockIdx.y, t = threadIdx.x;
  int32_t* h = H + ((size_t)b * R + r) * nch;
  const int per = (nch + 255) / 256;
  const int i0 = min(nch, t * per), i1 = min(nch, i0 + per);
  int v[16];
  int sum = 0;
  for (int c0 = i0; c0 < i1; c0 += 16) {
#pragma unroll
    for (int u = 0; u < 16; ++u) v[u] = c0 + u < i1 ? h[c0 + u] : 0;
#pragma unroll
    for (int u = 0; u < 16; ++u) sum += v[u];
  }
  int bin_total;
  int run = block_scan256(sum, wsum, bin_total);
  for (int c0 = i0; c0 < i1; c0 += 16) {
#pragma unroll
    for (int u = 0; u < 16; ++u) v[u] = c0 + u < i1 ? h[c0 + u] : 0;
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      if (c0 + u < i1) h[c0 + u] = run;
      run += v[u];
    }
  }
  if (t == 0) T[(size_t)b * RADIX_MAX_R + r] = bin_total;
}

// MODE 0: (key, value) arrays in and out (values default to the entry index).
// MODE 1 (first of two passes, packed): keys in, one packed word out per entry,
//   (key >> lo_bits) << pb | point id.
// MODE 2 (second pass, packed): packed words in, in the chunks of lo_chunk,
//   so a chunk's low digit is known and restores each key; point ids out.
//
// Ranking.  Each wave takes a quarter of the chunk in entry order, in steps
// of 64 entries.  In a step the lanes holding one digit find each other with
// one ballot per digit bit; the lowest of them adds the group's size to the
// wave's count of that digit with an LDS atomic that returns the count before
// it, and the others read that from it.  A wave's atomics execute in program
// order, so these counts are exact and the same on every run; all its steps'
// atomics are issued back to back and waited for once.  After a scan over
// digits and waves, an entry's place in the chunk sorted by digit is the start
// of its digit + its wave's start within the digit + the count before its
// step + its rank among its step's lanes of that digit.  The chunk is staged
// there in LDS (the output word and the digit, one byte) and written out in
// sorted order, so each digit's run goes out contiguously (coalesced).
template <int DBITS, int MODE>
__global__ __launch_bounds__(256) void radix_scatter_kernel(
    const int32_t* __restrict__ keys_in, const int32_t* __restrict__ vals_in, int N, int K,
    const int32_t* __restrict__ total, int shift, int nch,
    const int32_t* __restrict__ H, const int32_t* __restrict__ T, int32_t* __restrict__ total_out,
    int32_t* __restrict__ keys_out, int32_t* __restrict__ vals_out, int lo_bits, int pb,
    const int32_t* __restrict__ T1, int32_t* __restrict__ off) {
  constexpr int STEPS = RADIX_CHUNK / 256;  // 64-entry steps per wave
  constexpr int R = 1 << DBITS;
  static_assert(R <= 256, "one thread per digit in the scans");
  __shared__ int sval[RADIX_CHUNK];                 // output words in sorted order
  __shared__ int skey[MODE == 0 ? RADIX_CHUNK : 1];  // keys too when they are written out
  __shared__ uint8_t sdg[RADIX_CHUNK];              // digit of each sorted entry
  __shared__ int cnt[4][R];                          // per-wave digit counts, then starts
  __shared__ int gdelta[R];
  __shared__ int wsum[4][4], sel[5];
  const int b = blockIdx.y, ch = blockIdx.x, t = threadIdx.x;
  const int lane = t & 63, w = t >> 6;
  int e0, e1, lo_c = 0;
  if constexpr (MODE == 2) {
    lo_chunk(T1, b, 1 << lo_bits, ch, &wsum[2][0], sel, e0, e1, lo_c);
  } else {
    const int n_in = total ? total[b] : N;
    e0 = ch * RADIX_CHUNK;
    e1 = min(e0 + RADIX_CHUNK, n_in);
  }
  const int32_t* kb = keys_in + (size_t)b * N;
  const int32_t* vb = vals_in ? vals_in + (size_t)b * N : nullptr;
  const int ibase = e0 + w * (RADIX_CHUNK / 4);

  // the input word of each entry; the packed modes rebuild key and output
  // word from it (and the entry index) when needed, so only MODE 0 keeps a
  // value per entry
  int k[STEPS], v[MODE == 0 ? STEPS : 1];
#pragma unroll
  for (int s = 0; s < STEPS; ++s) {
    const int i = ibase + s * 64 + lane;
    const bool in = i < e1;
    k[s] = in ? kb[i] : -1;
    if constexpr (MODE == 0) v[s] = in ? (vb ? vb[i] : i) : 0;
  }
  // this bin's total over all chunks and its count before this chunk
  const int tbin = t < R ? T[(size_t)b * RADIX_MAX_R + t] : 0;
  const int hrun = t < R ? H[((size_t)b * R + t) * nch + ch] : 0;
  if (t < R) {
#pragma unroll
    for (int ww = 0; ww < 4; ++ww) cnt[ww][t] = 0;
  }
  // bin starts: exclusive scan of the bin totals (its barrier also orders the zeroing)
  int n_valid;
  const int bstart = block_scan256(tbin, wsum[0], n_valid);
  if (total_out && ch == 0 && t == 0) total_out[b] = n_valid;
  const int pmask = (int)((1u << pb) - 1u);
  if constexpr (MODE == 2) {
    // Cluster offsets: key (hi, lo) starts where digit hi's entries of the
    // first chunk of low digit lo go (bin start + the count before that
    // chunk); low digits with no entries share the next chunk's, those past
    // the last one the chunk past the end (always in the grid).  The chunk
    // of those low digits writes them, one thread per high digit.
    if (t < R) {
      const int a = min(max(bstart + hrun, 0), n_valid);
      int32_t* ob = off + (size_t)b * (K + 1);
      for (int l = sel[3]; l <= sel[4]; ++l) {
        const int key = (t << lo_bits) | l;
        if (key < K) ob[key] = a;
      }
      if (ch == 0 && t == 0) ob[K] = n_valid;
    }
  }
  // rank in entry order within each wave (see above)
  const uint32_t blo = lane >= 32 ? ~0u : (1u << lane) - 1u;  // lanes below this one
  const uint32_t bhi = lane <= 32 ? 0u : ~0u >> (64 - lane);
  // per step: digit (bits 0-7), rank (8-13), the digit group's lowest lane
  // (16-21), 1 << 24 for an entry (every digit value of 8-bit digits is a real
  // digit); and the count before the step
  int meta[STEPS], old[STEPS];
#pragma unroll
  for (int s = 0; s < STEPS; ++s) {
    int key;
    if constexpr (MODE == 2)  // high digit above the chunk's low digit
      key = k[s] >= 0 ? ((k[s] >> pb) << lo_bits) | lo_c : -1;
    else
      key = k[s];
    const bool valid = (unsigned)key < (unsigned)K;
    const int dg = valid ? digit_of(key, shift, R) : 0;
    // lanes holding the same digit: for each bit keep the lanes that agree,
    // on the two 32-lane halves (invalid lanes hold digit 0 and are dropped
    // by the first ballot)
    const uint64_t vm = __ballot(valid);
    uint32_t mlo = (uint32_t)vm, mhi = (uint32_t)(vm >> 32);
#pragma unroll
    for (int bit = 0; bit < DBITS; ++bit) {
      const int m = (int)((uint32_t)dg << (31 - bit)) >> 31;  // all ones where the bit is set
      const uint64_t bb = __ballot(m != 0);
      mlo &= ~((uint32_t)bb ^ (uint32_t)m);
      mhi &= ~((uint32_t)(bb >> 32) ^ (uint32_t)m);
    }
    const int rank = __popc(mlo & blo) + __popc(mhi & bhi);
    const int lead = !valid ? lane : mlo ? __builtin_ctz(mlo) : 32 + __builtin_ctz(mhi);
    int ms = dg | (rank << 8) | (lead << 16) | (valid ? 1 << 24 : 0);
    // one register per step from here on: the fields are read back from it,
    // not kept apart (which took four per step)
    asm volatile("" : "+v"(ms));
    meta[s] = ms;
    int before = 0;  // a scalar across the branch (an array there is copied whole)
    if (valid && rank == 0) before = atomicAdd(&cnt[w][dg], __popc(mlo) + __popc(mhi));
    old[s] = before;
    // one step at a time: hoisting every step's ballots ahead of the atomics
    // took all 256 registers
    __builtin_amdgcn_sched_barrier(0);
  }
#pragma unroll
  for (int s = 0; s < STEPS; ++s)
    old[s] = __shfl(old[s], (meta[s] >> 16) & 63) + ((meta[s] >> 8) & 63);
  __syncthreads();
  // this chunk's count per bin -> exclusive scan over bins; wave starts per bin
  int c4[4], tot = 0;
#pragma unroll
  for (int ww = 0; ww < 4; ++ww) {
    c4[ww] = t < R ? cnt[ww][t] : 0;
    tot += c4[ww];
  }
  int nloc;
  const int ls = block_scan256(tot, wsum[1], nloc);
  if (t < R) {
    gdelta[t] = bstart + hrun - ls;  // output position = gdelta[digit] + sorted position
    int run = ls;
#pragma unroll
    for (int ww = 0; ww < 4; ++ww) {
      cnt[ww][t] = run;
      run += c4[ww];
    }
  }
  __syncthreads();
  // stage the chunk sorted by digit, with its output words
#pragma unroll
  for (int s = 0; s < STEPS; ++s) {
    const int ms = meta[s];
    const int dg = ms & 255;
    if (ms & (1 << 24)) {
      const int pos = cnt[w][dg] + old[s];
      int out;
      if constexpr (MODE == 0) {
        out = v[s];
        skey[pos] = k[s];
      } else if constexpr (MODE == 1) {  // high digit above the point id
        out = ((k[s] >> lo_bits) << pb) | (ibase + s * 64 + lane);
      } else {  // the point id
        out = k[s] & pmask;
      }
      sval[pos] = out;
      sdg[pos] = (uint8_t)dg;
    }
  }
  __syncthreads();
  // write each bin's run contiguously
  int32_t* ko = keys_out ? keys_out + (size_t)b * N : nullptr;
  int32_t* vo = vals_out + (size_t)b * N;
#pragma unroll 4
  for (int s = 0; s < STEPS; ++s) {
    const int j = s * 256 + t;
    if (j < nloc) {
      const int g = gdelta[sdg[j] & (R - 1)] + j;
      vo[g] = sval[j];
      if constexpr (MODE == 0)
        if (ko) ko[g] = skey[j];
    }
  }
}

// Cluster offsets from the sorted keys: off[k] = first position of a key >= k
// (binary search); the counts are off[k+1] - off[k].
__global__ __launch_bounds__(256) void bounds_kernel(const int32_t* __restrict__ sorted,
                                                     const int32_t* __restrict__ total, int N, int K,
                                                     int32_t* __restrict__ off) {
  const int k = blockIdx.x * 256 + threadIdx.x, b = blockIdx.y;
  if (k > K) return;
  const int n = total[b];
  const int32_t* s = sorted + (size_t)b * N;
  auto lower = [&](int key) {
    int lo = 0, hi = n;
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (s[mid] < key) lo = mid + 1; else hi = mid;
    }
    return lo;
  };
  off[(size_t)b * (K + 1) + k] = lower(k);
}

// ---------------------------------------------------------------------------
// Segmented sum.  A row of D elements is RC 16-byte chunks; LPR lanes share a
// row (CPLR chunks each, LPR * CPLR >= RC: lanes past the row's end idle) and
// a wave covers RPW = 64 / LPR rows per step.
template <int DT> struct Row;
template <> struct Row<DT_F32> {
  static constexpr int per16 = 4;
  __device__ static void add(const uint4& q, float* a) {
    a[0] += __uint_as_float(q.x);
    a[1] += __uint_as_float(q.y);
    a[2] += __uint_as_float(q.z);
    a[3] += __uint_as_float(q.w);
  }
};
template <> struct Row<DT_BF16> {
  static constexpr int per16 = 8;
  __device__ static void add(const uint4& q, float* a) {
    const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      a[2 * e] += __uint_as_float(w[e] << 16);
      a[2 * e + 1] += __uint_as_float(w[e] & 0xffff0000u);
    }
  }
};
template <> struct Row<DT_F16> {
  static constexpr int per16 = 8;
  __device__ static void add(const uint4& q, float* a) {
    const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      a[2 * e] += (float)__builtin_bit_cast(_Float16, (uint16_t)(w[e] & 0xffffu));
      a[2 * e + 1] += (float)__builtin_bit_cast(_Float16, (uint16_t)(w[e] >> 16));
    }
  }
};

template <int DT, int LPR, int CPLR>
__global__ __launch_bounds__(256) void segreduce_kernel(
    const uint4* __restrict__ X, const int32_t* __restrict__ perm, const int32_t* __restrict__ off,
    int N, int K, int RC, int nred, int cr, float* __restrict__ sums, float* __restrict__ carry) {
  constexpr int E = Row<DT>::per16;
  const int D = RC * E;
  constexpr int RPW = 64 / LPR;
  constexpr int NA = CPLR * E;
  constexpr int U = 8;  // rows in flight per lane
  const int lane = threadIdx.x & 63;
  const int w = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int b = blockIdx.y;
  if (w >= nred) return;
  const int32_t* ob = off + (size_t)b * (K + 1);
  const int j0 = w * cr;
  const int j1 = min(ob[K], j0 + cr);  // ob[K] = number of sorted (valid) entries
  if (j0 >= j1) return;
  const int32_t* pb = perm + (size_t)b * N;
  const uint4* xb = X + (size_t)b * N * RC;
  const int r = lane / LPR, q = lane % LPR;

  // last cluster whose run starts at or before j0 (it is non-empty and holds j0)
  int lo = 0, hi = K;  // invariant: ob[lo] <= j0 < ob[hi] (ob[K] = N > j0)
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (ob[mid] <= j0) lo = mid; else hi = mid;
  }
  int k = lo;
  int pos = j0;
  while (pos < j1) {
    while (ob[k + 1] <= pos) ++k;
    const int kstart = ob[k], kend = ob[k + 1];
    const int seg_end = min(kend, j1);
    float acc[NA];
#pragma unroll
    for (int a = 0; a < NA; ++a) acc[a] = 0.f;
    // U rows in flight per lane; the row ids of the next group are fetched
    // while the current group's rows are loading
    int pid[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int jj = pos + r + u * RPW;
      pid[u] = jj < seg_end ? pb[jj] : -1;
    }
    for (int j = pos + r; j < seg_end; j += U * RPW) {
      uint4 v[U][CPLR];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        if (pid[u] >= 0) {
          const uint4* row = xb + (size_t)pid[u] * RC + q * CPLR;
#pragma unroll
          for (int c = 0; c < CPLR; ++c)
            v[u][c] = q * CPLR + c < RC ? row[c] : make_uint4(0, 0, 0, 0);
        } else {
#pragma unroll
          for (int c = 0; c < CPLR; ++c) v[u][c] = make_uint4(0, 0, 0, 0);
        }
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int jj = j + (U + u) * RPW;
        pid[u] = jj < seg_end ? pb[jj] : -1;
      }
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int c = 0; c < CPLR; ++c) Row<DT>::add(v[u][c], acc + c * E);
    }
#pragma unroll
    for (int msk = LPR; msk < 64; msk <<= 1)
#pragma unroll
      for (int a = 0; a < NA; ++a) acc[a] += __shfl_xor(acc[a], msk);
    const bool complete = kstart >= j0 && kend <= j1;
    float* dst = complete ? sums + ((size_t)b * K + k) * D
                          : carry + (((size_t)b * nred + w) * 2 + (pos == j0 ? 0 : 1)) * D;
    if (r == 0) {
#pragma unroll
      for (int c = 0; c < CPLR; ++c) {
        if (q * CPLR + c >= RC) continue;
        float4* d4 = reinterpret_cast<float4*>(dst + (q * CPLR + c) * E);
#pragma unroll
        for (int e = 0; e < E; e += 4)
          d4[e / 4] = make_float4(acc[c * E + e], acc[c * E + e + 1], acc[c * E + e + 2],
                                  acc[c * E + e + 3]);
      }
    }
    pos = seg_end;
    ++k;
  }
}

// The tail of the update kernels inside kmeans_lloyd (NextStep): the new
// centroid row k, staged in LDS by the workgroup, becomes the next
// iteration's rounded row and score (wave 0, prep_row: the bits prep would
// write), and the workgroup of cluster 0 sums the instance's objective
// partials in fp64 in a fixed order.
__device__ inline void next_step_tail(const NextStep& nx, const float* row, int64_t b, int k,
                                      bool has_row, int D, int tt, int t, bool obj_block,
                                      double* red) {
  if (nx.chat && has_row && tt < 64) {  // the first wave of the cluster's thread group
    const int64_t r = b * nx.Kp + k;
    void* out = (char*)nx.chat + r * D * dt_bytes(nx.dt);
    if (nx.dt == DT_BF16) prep_row<DT_BF16>(row, false, D, tt, out, nx.cinit + r);
    else if (nx.dt == DT_F16) prep_row<DT_F16>(row, false, D, tt, out, nx.cinit + r);
    else prep_row<DT_F32>(row, false, D, tt, out, nx.cinit + r);
  }
  if (nx.objective && obj_block) {
    // a thread adds its partials (every 256th) in index order; the loads go
    // out OBJ_BATCH at a time (there can be tens of thousands of partials,
    // and the kernel lasts as long as this workgroup), the adds stay in order
    constexpr int OBJ_BATCH = 16;
    const double* pb = nx.objpart + b * nx.nparts;
    const int64_t last = nx.nparts - 1;
    double a = 0.0;
    for (int64_t i0 = t; i0 <= last; i0 += 256 * OBJ_BATCH) {
      double v[OBJ_BATCH];
#pragma unroll
      for (int u = 0; u < OBJ_BATCH; ++u) v[u] = pb[min(i0 + 256 * u, last)];
#pragma unroll
      for (int u = 0; u < OBJ_BATCH; ++u)
        if (i0 + 256 * u <= last) a += v[u];
    }
    red[t] = a;
    __syncthreads();
    for (int w = 128; w > 0; w >>= 1) {
      if (t < w) red[t] += red[t + w];
      __syncthreads();
    }
    if (t == 0) nx.objective[b * nx.iters + nx.t] = red[0];
  }
}

// The last update kernels give each cluster a group of threads: one wave for
// rows of up to 256 floats (four clusters per workgroup), else the whole
// workgroup.  Within a group each thread owns 4 consecutive dimensions and the
// group's (threads / (D/4)) row slots each add every slots-th partial in order
// (loads issued SUM_BATCH at a time, adds in that order); the slot sums are
// combined in slot order through LDS.  The group size depends on D only.
constexpr int SUM_BATCH = 8;
__host__ __device__ inline int final_threads(int D) { return D <= 256 ? 64 : 256; }

__device__ inline float4 f4add(float4 s, float4 v) {
  return make_float4(s.x + v.x, s.y + v.y, s.z + v.z, s.w + v.w);
}
__device__ inline float4 f4div(float4 s, float n) {
  return make_float4(s.x / n, s.y / n, s.z / n, s.w / n);
}

// Per cluster, the count (the length of its run in the sorted order, written
// out) and the sum (one slice, or the slices' carries in slice order) over
// the count; an empty cluster keeps its previous centroid.
__global__ __launch_bounds__(256) void finalize_kernel(
    const float* __restrict__ sums, const float* __restrict__ carry,
    int32_t* __restrict__ counts, const int32_t* __restrict__ off,
    const float* C_prev, int K, int D, int nred, int cr, float* C_out, NextStep nx) {
  __shared__ float4 part[256];
  extern __shared__ float4 row4_dyn[];  // the groups' new centroid rows (D floats each)
  __shared__ double red[256];
  const int t = threadIdx.x, b = blockIdx.y;
  const int D4 = D / 4;
  const int TPC = final_threads(D), G = 256 / TPC;
  const int g = t / TPC, tt = t % TPC;
  const int k = blockIdx.x * G + g;
  const bool valid = k < K;
  float4* row4 = row4_dyn + g * D4;
  const size_t rowoff = ((size_t)b * K + k) * D;
  int n = 0, j0 = 0, c0 = 0, c1 = 0;
  if (valid) {
    j0 = off[(size_t)b * (K + 1) + k];
    const int j1 = off[(size_t)b * (K + 1) + k + 1];
    n = j1 - j0;
    if (t % TPC == 0) counts[(size_t)b * K + k] = n;
    c0 = j0 / cr;
    c1 = n == 0 ? c0 : (j1 - 1) / cr;
  }
  const bool multi = valid && n > 0 && c0 != c1;
  const float fn = (float)n;
  const int slots = D4 >= TPC ? 1 : TPC / D4;
  const int slot = D4 >= TPC ? 0 : tt / D4;
  for (int d0 = 0; d0 < D4; d0 += TPC) {
    const int d = d0 + (D4 >= TPC ? tt : tt % D4);
    float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
    if (multi && slot < slots && d < D4) {
      // slice c holds the cluster's head run in entry 1 when the run starts
      // inside it (only possible for c0), else in entry 0
      for (int cb = c0 + slot; cb <= c1; cb += SUM_BATCH * slots) {
        float4 v[SUM_BATCH];
#pragma unroll
        for (int u = 0; u < SUM_BATCH; ++u) {
          const int c = min(cb + u * slots, c1);
          const int which = (c == c0 && j0 > c * cr) ? 1 : 0;
          v[u] = reinterpret_cast<const float4*>(carry + (((size_t)b * nred + c) * 2 + which) * D)[d];
        }
#pragma unroll
        for (int u = 0; u < SUM_BATCH; ++u)
          if (cb + u * slots <= c1) s = f4add(s, v[u]);
      }
    }
    if (slots > 1) {
      __syncthreads();
      part[t] = s;
      __syncthreads();
    }
    if (valid && slot == 0 && d < D4) {
      float4 m;
      if (n == 0) {
        m = reinterpret_cast<const float4*>(C_prev + rowoff)[d];
      } else if (!multi) {
        m = f4div(reinterpret_cast<const float4*>(sums + rowoff)[d], fn);
      } else {
        for (int u = 1; u < slots; ++u) s = f4add(s, part[g * TPC + u * D4 + tt % D4]);
        m = f4div(s, fn);
      }
      reinterpret_cast<float4*>(C_out + rowoff)[d] = m;
      row4[d] = m;
    }
  }
  __syncthreads();
  next_step_tail(nx, reinterpret_cast<const float*>(row4), b, k, valid, D, tt, t,
                 blockIdx.x == 0, red);
}

// ---------------------------------------------------------------------------
// Small-K update (smallk_ok: few clusters, K * D small): no global sort.  A
// workgroup of 16 waves takes SMALLK_CH consecutive points of one instance,
// sorts them by cluster id in LDS (stable: per-wave counts, a scan over
// clusters, then a ballot multi-split ranking in point order) and sums each
// cluster's rows in that order (rows strided over lane groups, then a xor
// butterfly) into the chunk's partial [K, D] and count.  smallk_combine adds
// a cluster's partials in chunk order and divides.  X is read once; no
// floating-point atomics; every sum has a fixed order.
template <int DT, int LPR, int CPLR>
__global__ __launch_bounds__(1024) void smallk_partials_kernel(
    const uint4* __restrict__ X, const int32_t* __restrict__ idx, int N, int K, int RC, int dbits,
    int nch, float* __restrict__ partial, int32_t* __restrict__ pcount) {
  constexpr int E = Row<DT>::per16;
  const int D = RC * E;
  constexpr int RPW = 64 / LPR;
  constexpr int NA = CPLR * E;
  constexpr int U = CPLR >= 8 ? 1 : 8 / CPLR;  // rows in flight per lane (4 waves per SIMD)
  constexpr int W = 16, CH = SMALLK_CH, PER = CH / W / 64;
  static_assert(PER * 64 * W == CH, "whole 64-entry steps per wave");
  __shared__ int cnt[W][SMALLK_MAX_K];  // per-wave counts, then per-wave run starts
  __shared__ int kst[SMALLK_MAX_K + 1];  // cluster run starts within the chunk
  __shared__ int plist[CH];              // chunk offsets of the points, sorted by cluster
  __shared__ int wsum[W];
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int ch = blockIdx.x, b = blockIdx.y;
  const int i0 = ch * CH;
  const int nin = min(CH, N - i0);
  const int32_t* ib = idx + (size_t)b * N + i0;

  int k[PER];
#pragma unroll
  for (int s = 0; s < PER; ++s) {
    const int e = (w * PER + s) * 64 + lane;
    k[s] = e < nin ? ib[e] : -1;
  }
  for (int r = t; r < W * SMALLK_MAX_K; r += 1024) (&cnt[0][0])[r] = 0;
  __syncthreads();
#pragma unroll
  for (int s = 0; s < PER; ++s)
    if ((unsigned)k[s] < (unsigned)K) atomicAdd(&cnt[w][k[s]], 1);  // integer: exact
  __syncthreads();
  int c16[W], tot = 0;
#pragma unroll
  for (int ww = 0; ww < W; ++ww) {
    c16[ww] = t < K ? cnt[ww][t] : 0;
    tot += c16[ww];
  }
  int total;
  const int ex = block_scan<W>(tot, wsum, total);
  if (t < K) {
    kst[t] = ex;
    int run = ex;
#pragma unroll
    for (int ww = 0; ww < W; ++ww) {
      cnt[ww][t] = run;
      run += c16[ww];
    }
  }
  if (t == 0) kst[K] = total;
  __syncthreads();
  const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
#pragma unroll
  for (int s = 0; s < PER; ++s) {
    const bool valid = (unsigned)k[s] < (unsigned)K;
    const int dg = valid ? k[s] : 0;
    uint64_t match = __ballot(valid);
    for (int bit = 0; bit < dbits; ++bit) {
      const int on = (dg >> bit) & 1;
      const uint64_t bb = __ballot(on);
      match &= bb ^ (uint64_t)(int64_t)(on - 1);
    }
    if (valid) {
      const int rank = __popcll(match & below);
      const int start = cnt[w][dg];
      if (rank == 0) cnt[w][dg] = start + __popcll(match);
      plist[start + rank] = (w * PER + s) * 64 + lane;
    }
  }
  __syncthreads();

  const uint4* xb = X + ((size_t)b * N + i0) * RC;
  const int r = lane / LPR, q = lane % LPR;
  float* pb = partial + ((size_t)b * nch + ch) * K * D;
  for (int kk = w; kk < K; kk += W) {
    const int s0 = kst[kk], s1 = kst[kk + 1];
    float acc[NA];
#pragma unroll
    for (int a = 0; a < NA; ++a) acc[a] = 0.f;
    for (int j = s0 + r; j < s1; j += U * RPW) {
      uint4 v[U][CPLR];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int jj = j + u * RPW;
        if (jj < s1) {
          const uint4* row = xb + (size_t)plist[jj] * RC + q * CPLR;
#pragma unroll
          for (int c = 0; c < CPLR; ++c)
            v[u][c] = q * CPLR + c < RC ? row[c] : make_uint4(0, 0, 0, 0);
        } else {
#pragma unroll
          for (int c = 0; c < CPLR; ++c) v[u][c] = make_uint4(0, 0, 0, 0);
        }
      }
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int c = 0; c < CPLR; ++c) Row<DT>::add(v[u][c], acc + c * E);
    }
#pragma unroll
    for (int msk = LPR; msk < 64; msk <<= 1)
#pragma unroll
      for (int a = 0; a < NA; ++a) acc[a] += __shfl_xor(acc[a], msk);
    if (r == 0) {
#pragma unroll
      for (int c = 0; c < CPLR; ++c) {
        if (q * CPLR + c >= RC) continue;
        float4* d4 = reinterpret_cast<float4*>(pb + (size_t)kk * D + (q * CPLR + c) * E);
#pragma unroll
        for (int e = 0; e < E; e += 4)
          d4[e / 4] = make_float4(acc[c * E + e], acc[c * E + e + 1], acc[c * E + e + 2],
                                  acc[c * E + e + 3]);
      }
    }
    if (lane == 0) pcount[((size_t)b * nch + ch) * K + kk] = s1 - s0;
  }
}

// Per cluster (thread groups as in finalize_kernel): the count (integer sum
// over chunks), then the chunk partials added in chunk order and divided by
// the count.  An empty cluster keeps its previous centroid.
__global__ __launch_bounds__(256) void smallk_combine_kernel(
    const float* __restrict__ partial, const int32_t* __restrict__ pcount, const float* C_prev,
    int K, int D, int nch, float* C_out, int32_t* __restrict__ counts, NextStep nx) {
  __shared__ int gcount[4];
  __shared__ float4 part[256];
  extern __shared__ float4 row4_dyn[];  // the groups' new centroid rows (D floats each)
  __shared__ double red[256];
  const int t = threadIdx.x, b = blockIdx.y;
  const int D4 = D / 4;
  const int TPC = final_threads(D), G = 256 / TPC;
  const int g = t / TPC, tt = t % TPC;
  const int k = blockIdx.x * G + g;
  const bool valid = k < K;
  float4* row4 = row4_dyn + g * D4;
  const size_t rowoff = ((size_t)b * K + k) * D;
  if (tt < 64) {  // the group's first wave counts
    int n = 0;
    if (valid)
      for (int c = tt; c < nch; c += 64) n += pcount[((size_t)b * nch + c) * K + k];
#pragma unroll
    for (int m = 1; m < 64; m <<= 1) n += __shfl_xor(n, m);
    if (tt == 0) gcount[g] = n;
  }
  __syncthreads();
  const int total = gcount[g];
  if (valid && tt == 0) counts[(size_t)b * K + k] = total;
  const float fn = (float)total;
  const int slots = D4 >= TPC ? 1 : TPC / D4;
  const int slot = D4 >= TPC ? 0 : tt / D4;
  const float4* pb = reinterpret_cast<const float4*>(partial + ((size_t)b * nch * K + k) * D);
  const size_t cstride = (size_t)K * D4;  // float4s from one chunk's row k to the next chunk's
  for (int d0 = 0; d0 < D4; d0 += TPC) {
    const int d = d0 + (D4 >= TPC ? tt : tt % D4);
    float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
    if (valid && total > 0 && slot < slots && d < D4) {
      for (int cb = slot; cb < nch; cb += SUM_BATCH * slots) {
        float4 v[SUM_BATCH];
#pragma unroll
        for (int u = 0; u < SUM_BATCH; ++u) v[u] = pb[min(cb + u * slots, nch - 1) * cstride + d];
#pragma unroll
        for (int u = 0; u < SUM_BATCH; ++u)
          if (cb + u * slots < nch) s = f4add(s, v[u]);
      }
    }
    if (slots > 1) {
      __syncthreads();
      part[t] = s;
      __syncthreads();
    }
    if (valid && slot == 0 && d < D4) {
      float4 m;
      if (total == 0) {
        m = reinterpret_cast<const float4*>(C_prev + rowoff)[d];
      } else {
        for (int u = 1; u < slots; ++u) s = f4add(s, part[g * TPC + u * D4 + tt % D4]);
        m = f4div(s, fn);
      }
      reinterpret_cast<float4*>(C_out + rowoff)[d] = m;
      row4[d] = m;
    }
  }
  __syncthreads();
  next_step_tail(nx, reinterpret_cast<const float*>(row4), b, k, valid, D, tt, t,
                 blockIdx.x == 0, red);
}

template <int DT, int LPR, int CPLR>
static void launch_smallk(const void* X, const int32_t* idx, const Workspace& w, int64_t B,
                          int64_t N, int64_t K, int rc, int dbits, hipStream_t s) {
  smallk_partials_kernel<DT, LPR, CPLR><<<dim3((unsigned)w.n_sk_chunks, (unsigned)B), 1024, 0, s>>>(
      (const uint4*)X, idx, (int)N, (int)K, rc, dbits, (int)w.n_sk_chunks, w.partial, w.pcount);
}

// Lanes per row (LPR) x chunks per lane (CPLR) for a row of rc 16-byte
// chunks: the smallest power-of-two cover of rc.
static int row_lanes(int64_t rc) {
  int c = 2;
  while (c < rc) c *= 2;
  return c;  // 2 .. 512
}

template <int DT>
static hipError_t launch_smallk_dt(const void* X, const int32_t* idx, const Workspace& w, int64_t B,
                                   int64_t N, int64_t D, int64_t K, int dbits, hipStream_t s) {
  const int rc = (int)(D * dt_bytes(DT) / 16);  // 16-byte chunks per row
  switch (row_lanes(rc)) {
    case 2: launch_smallk<DT, 2, 1>(X, idx, w, B, N, K, rc, dbits, s); break;
    case 4: launch_smallk<DT, 4, 1>(X, idx, w, B, N, K, rc, dbits, s); break;
    case 8: launch_smallk<DT, 8, 1>(X, idx, w, B, N, K, rc, dbits, s); break;
    case 16: launch_smallk<DT, 16, 1>(X, idx, w, B, N, K, rc, dbits, s); break;
    case 32: launch_smallk<DT, 32, 1>(X, idx, w, B, N, K, rc, dbits, s); break;
    case 64: launch_smallk<DT, 64, 1>(X, idx, w, B, N, K, rc, dbits, s); break;
    case 128: launch_smallk<DT, 64, 2>(X, idx, w, B, N, K, rc, dbits, s); break;
    case 256: launch_smallk<DT, 64, 4>(X, idx, w, B, N, K, rc, dbits, s); break;
    case 512: launch_smallk<DT, 64, 8>(X, idx, w, B, N, K, rc, dbits, s); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

static hipError_t launch_update_smallk(const void* X, int dt, const int32_t* idx,
                                       const float* C_prev, const Workspace& w, int64_t B,
                                       int64_t N, int64_t D, int64_t K, float* C_out,
                                       int32_t* counts, const NextStep& nx, hipStream_t s) {
  int dbits = 0;
  while ((1ll << dbits) < K) ++dbits;
  hipError_t e;
  if (dt == DT_BF16) e = launch_smallk_dt<DT_BF16>(X, idx, w, B, N, D, K, dbits, s);
  else if (dt == DT_F16) e = launch_smallk_dt<DT_F16>(X, idx, w, B, N, D, K, dbits, s);
  else e = launch_smallk_dt<DT_F32>(X, idx, w, B, N, D, K, dbits, s);
  if (e != hipSuccess) return e;
  return launch_combine(w, w.n_sk_chunks, C_prev, B, K, D, C_out, counts, nx, s);
}

// ---------------------------------------------------------------------------
template <int DT, int LPR, int CPLR>
static void launch_segreduce(const void* X, const Workspace& w, int64_t B, int64_t N, int64_t K,
                             int rc, hipStream_t s) {
  const dim3 grid((unsigned)((w.n_red_chunks + 3) / 4), (unsigned)B), block(256);
  segreduce_kernel<DT, LPR, CPLR><<<grid, block, 0, s>>>((const uint4*)X, w.perm, w.off, (int)N,
                                                         (int)K, rc, (int)w.n_red_chunks,
                                                         (int)w.red_cr, w.sums, w.carry);
}

template <int DT>
static hipError_t launch_segreduce_dt(const void* X, const Workspace& w, int64_t B, int64_t N,
                                      int64_t D, int64_t K, hipStream_t s) {
  const int rc = (int)(D * dt_bytes(DT) / 16);  // 16-byte chunks per row
  switch (row_lanes(rc)) {
    case 2: launch_segreduce<DT, 2, 1>(X, w, B, N, K, rc, s); break;
    case 4: launch_segreduce<DT, 4, 1>(X, w, B, N, K, rc, s); break;
    case 8: launch_segreduce<DT, 8, 1>(X, w, B, N, K, rc, s); break;
    case 16: launch_segreduce<DT, 16, 1>(X, w, B, N, K, rc, s); break;
    case 32: launch_segreduce<DT, 32, 1>(X, w, B, N, K, rc, s); break;
    case 64: launch_segreduce<DT, 64, 1>(X, w, B, N, K, rc, s); break;
    case 128: launch_segreduce<DT, 64, 2>(X, w, B, N, K, rc, s); break;
    case 256: launch_segreduce<DT, 64, 4>(X, w, B, N, K, rc, s); break;
    case 512: launch_segreduce<DT, 64, 8>(X, w, B, N, K, rc, s); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t update_init() { return hipSuccess; }

template <int MODE, typename... A>
static hipError_t launch_scatter(int dbits, dim3 grid, hipStream_t s, A... a) {
  switch (dbits) {
    case 1: radix_scatter_kernel<1, MODE><<<grid, 256, 0, s>>>(a...); break;
    case 2: radix_scatter_kernel<2, MODE><<<grid, 256, 0, s>>>(a...); break;
    case 3: radix_scatter_kernel<3, MODE><<<grid, 256, 0, s>>>(a...); break;
    case 4: radix_scatter_kernel<4, MODE><<<grid, 256, 0, s>>>(a...); break;
    case 5: radix_scatter_kernel<5, MODE><<<grid, 256, 0, s>>>(a...); break;
    case 6: radix_scatter_kernel<6, MODE><<<grid, 256, 0, s>>>(a...); break;
    case 7: radix_scatter_kernel<7, MODE><<<grid, 256, 0, s>>>(a...); break;
    case 8: radix_scatter_kernel<8, MODE><<<grid, 256, 0, s>>>(a...); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// Digit widths: the key needs `bits` bits; one pass for <= 8 bits, else two
// passes of about half each.
static void radix_plan(int64_t K, int& passes, int& d1, int& d2) {
  int bits = 1;
  while ((1ll << bits) < K) ++bits;
  passes = bits <= RADIX_MAX_BITS ? 1 : 2;
  d1 = passes == 1 ? bits : (bits + 1) / 2;
  d2 = bits - (passes == 1 ? 0 : d1);
}

// Bits that hold a point id below N (at least 1).
static int pid_bits(int64_t N) {
  int p = 1;
  while ((1ll << p) < N) ++p;
  return p;
}

// Digits of the packed passes: the second pass's chunks hold one low digit
// each, so the low digit gets at most log2(N / RADIX_CHUNK) bits (bins of at
// least a chunk on average) but at least what leaves the high digit <= 8
// bits; within that, the split nearest to half.
static void radix_plan_packed(int64_t N, int64_t K, int& d1, int& d2) {
  int bits = 1;
  while ((1ll << bits) < K) ++bits;
  int fill = 0;
  while ((RADIX_CHUNK << (fill + 1)) <= N) ++fill;
  d1 = std::max(bits - RADIX_MAX_BITS, std::min((bits + 1) / 2, fill));
  d2 = bits - d1;
}

// Two passes go over one array of packed words when the high digit and the
// point id fit a non-negative int (31 bits).
static bool sort_packed(int64_t N, int64_t K) {
  int passes, d1, d2;
  radix_plan(K, passes, d1, d2);
  if (passes != 2) return false;
  radix_plan_packed(N, K, d1, d2);
  return d2 + pid_bits(N) <= 31;
}

hipError_t launch_combine(const Workspace& w, int64_t nch, const float* C_prev, int64_t B,
                          int64_t K, int64_t D, float* C_out, int32_t* counts,
                          const NextStep& nx, hipStream_t s) {
  const int64_t G = 256 / final_threads((int)D);
  smallk_combine_kernel<<<dim3((unsigned)((K + G - 1) / G), (unsigned)B), 256,
                          G * D * sizeof(float), s>>>(
      w.partial, w.pcount, C_prev, (int)K, (int)D, (int)nch, C_out, counts, nx);
  return hipGetLastError();
}

hipError_t launch_update(const void* X, int dt, const int32_t* idx, const float* C_prev,
                         const Workspace& w, int64_t B, int64_t N, int64_t D, int64_t K,
                         float* C_out, int32_t* counts, const NextStep& nx, hipStream_t s) {
  if (sums_ok(dt, D, K)) {
    const hipError_t e = launch_sums(X, dt, w, B, N, D, K, SUMS_ONLY, const_cast<int32_t*>(idx),
                                     nullptr, s);
    if (e != hipSuccess) return e;
    return launch_combine(w, w.n_sk_chunks, C_prev, B, K, D, C_out, counts, nx, s);
  }
  if (smallk_ok(dt, D, K))
    return launch_update_smallk(X, dt, idx, C_prev, w, B, N, D, K, C_out, counts, nx, s);
  hipError_t e;
  const int nch = (int)w.n_sort_chunks;
  const dim3 cgrid(nch, (unsigned)B);
  int passes, d1, d2;
  radix_plan(K, passes, d1, d2);
  if (sort_packed(N, K)) {
    radix_plan_packed(N, K, d1, d2);
    // two passes over one array: pass 1 sorts by the low digit and writes
    // (high digit, point id) words; pass 2 sorts those by the high digit in
    // chunks of one low digit each and writes the point ids; the offsets and
    // counts come from pass 2's histogram
    const int pb = pid_bits(N);
    const int R1 = 1 << d1, R2 = 1 << d2;
    const int nch2 = nch + R1;  // chunks of one low digit: at most this many
    radix_hist_kernel<<<cgrid, 256, 0, s>>>(idx, (int)N, (int)K, nullptr, 0, R1, nch, w.rhist, 0,
                                            nullptr, 0);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    radix_scan_kernel<<<dim3(R1, (unsigned)B), 256, 0, s>>>(w.rhist, R1, nch, w.rbin1);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = launch_scatter<1>(d1, cgrid, s, idx, (const int32_t*)nullptr, (int)N, (int)K,
                               (const int32_t*)nullptr, 0, nch, (const int32_t*)w.rhist,
                               (const int32_t*)w.rbin1, w.rtotal, (int32_t*)nullptr, w.keys_a, d1,
                               pb, (const int32_t*)nullptr, (int32_t*)nullptr)) != hipSuccess)
      return e;
    const dim3 cgrid2(nch2, (unsigned)B);
    radix_hist_kernel<<<cgrid2, 256, 0, s>>>(w.keys_a, (int)N, (int)K, nullptr, 0, R2, nch2,
                                             w.rhist, pb, w.rbin1, d1);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    radix_scan_kernel<<<dim3(R2, (unsigned)B), 256, 0, s>>>(w.rhist, R2, nch2, w.rbin);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = launch_scatter<2>(d2, cgrid2, s, (const int32_t*)w.keys_a, (const int32_t*)nullptr,
                               (int)N, (int)K, (const int32_t*)nullptr, d1, nch2,
                               (const int32_t*)w.rhist, (const int32_t*)w.rbin, (int32_t*)nullptr,
                               (int32_t*)nullptr, w.perm, d1, pb,
                               (const int32_t*)w.rbin1, w.off)) != hipSuccess)
      return e;
  } else {
    // pass 1: idx (raw) -> (keys_a, vals_a) sorted by the low digit; with one
    // pass the values go straight to perm and the keys to keys_b
    const int R = 1 << d1;
    radix_hist_kernel<<<cgrid, 256, 0, s>>>(idx, (int)N, (int)K, nullptr, 0, R, nch, w.rhist, 0,
                                            nullptr, 0);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    radix_scan_kernel<<<dim3(R, (unsigned)B), 256, 0, s>>>(w.rhist, R, nch, w.rbin);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = launch_scatter<0>(d1, cgrid, s, idx, (const int32_t*)nullptr, (int)N, (int)K,
                               (const int32_t*)nullptr, 0, nch, (const int32_t*)w.rhist,
                               (const int32_t*)w.rbin, w.rtotal,
                               passes == 1 ? w.keys_b : w.keys_a, passes == 1 ? w.perm : w.vals_a,
                               0, 0, (const int32_t*)nullptr, (int32_t*)nullptr)) != hipSuccess)
      return e;
    if (passes == 2) {
      const int R2 = 1 << d2;
      radix_hist_kernel<<<cgrid, 256, 0, s>>>(w.keys_a, (int)N, (int)K, w.rtotal, d1, R2, nch,
                                              w.rhist, 0, nullptr, 0);
      if ((e = hipGetLastError()) != hipSuccess) return e;
      radix_scan_kernel<<<dim3(R2, (unsigned)B), 256, 0, s>>>(w.rhist, R2, nch, w.rbin);
      if ((e = hipGetLastError()) != hipSuccess) return e;
      if ((e = launch_scatter<0>(d2, cgrid, s, (const int32_t*)w.keys_a, (const int32_t*)w.vals_a,
                                 (int)N, (int)K, (const int32_t*)w.rtotal, d1, nch,
                                 (const int32_t*)w.rhist, (const int32_t*)w.rbin, (int32_t*)nullptr,
                                 w.keys_b, w.perm, 0, 0, (const int32_t*)nullptr,
                                 (int32_t*)nullptr)) != hipSuccess)  // the same total
        return e;
    }
    bounds_kernel<<<dim3((unsigned)((K + 1 + 255) / 256), (unsigned)B), 256, 0, s>>>(
        w.keys_b, w.rtotal, (int)N, (int)K, w.off);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  if (dt == DT_BF16) e = launch_segreduce_dt<DT_BF16>(X, w, B, N, D, K, s);
  else if (dt == DT_F16) e = launch_segreduce_dt<DT_F16>(X, w, B, N, D, K, s);
  else e = launch_segreduce_dt<DT_F32>(X, w, B, N, D, K, s);
  if (e != hipSuccess) return e;
  const int64_t G = 256 / final_threads((int)D);
  finalize_kernel<<<dim3((unsigned)((K + G - 1) / G), (unsigned)B), 256, G * D * sizeof(float), s>>>(
      w.sums, w.carry, counts, w.off, C_prev, (int)K, (int)D, (int)w.n_red_chunks, (int)w.red_cr,
      C_out, nx);
  return hipGetLastError();
}

}  // namespace fkm
