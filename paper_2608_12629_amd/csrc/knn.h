// knn.h -- KNN search on the assignment kernel's layout (bf16/fp16 rows,
// D a multiple of 16 up to 256): for every query, the k database rows at the
// smallest squared Euclidean distance, nearest first, ties to the lowest
// index.  The paper lists KNN build and search beside KMeans among the
// dispatcher-backed families of Section 6 (recall 1.0); this is the same fused
// distance contraction with a top-k in place of the arg-min, and the k x N
// distance matrix is never stored.  Instantiated once per storage type in
// knn_bf16.hip and knn_f16.hip.
//
// Queries play the points' role: each wave keeps 32 queries in registers
// (one 32-column MFMA tile).  Database rows play the centroids' role: a
// preparation pass copies them into the padded, staged layout with their
// -|r|^2/2 scores (the rows are already in the storage type, so nothing is
// rounded), and they stream through LDS in the assignment kernel's stages
// (direct L2-to-LDS loads, XOR-swizzled rows, double buffering).
//
// Top-k.  Lane 32 h + n holds, for query n, the 16 scores of rows
// 8 q + 4 h + r of each 32-row tile, and keeps its own list of the KMAX best
// (score, index) in registers, best first.  Rows reach a lane in increasing
// index order, so a strict compare keeps equal scores in index order.  A tile
// costs one compare per score against the lane's KMAX-th best when no lane of
// the wave improves; otherwise a score enters by a compare-exchange pass down
// the list (branch-free per lane, one wave-uniform branch).  At the end the
// two halves' lists of a query merge by (score, then lower index), and the
// first k entries are written with d = max(0, |q|^2 - 2 s).
#pragma once

#include "assign_pipe.h"

namespace fkm {

// Database rows to the staged layout: row j of each instance to chat (padded to
// Np rows: zero rows with score -FLT_MAX; rows of Din elements widened to D
// with zeros), and its -|r|^2/2 (one wave per row, lane-strided then a fixed
// xor butterfly).
template <int DT>
__global__ __launch_bounds__(256) void knn_prep_kernel(const uint16_t* __restrict__ R, int64_t B,
                                                       int N, int Np, int Din, int D,
                                                       uint16_t* __restrict__ chat,
                                                       float* __restrict__ cinit) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= B * Np) return;
  const int64_t b = row / Np;
  const int j = (int)(row % Np);
  const bool pad = j >= N;
  const uint16_t* r = R + (b * N + (pad ? 0 : j)) * Din;
  uint16_t* out = chat + row * D;
  float ss = 0.f;
  for (int d = lane; d < D; d += 64) {
    const uint16_t h = (pad || d >= Din) ? (uint16_t)0 : r[d];
    out[d] = h;
    const float v = Elem<DT>::widen(h);
    ss = __builtin_fmaf(v, v, ss);
  }
#pragma unroll
  for (int m = 1; m < 64; m <<= 1) ss += __shfl_xor(ss, m);
  if (lane == 0) cinit[row] = pad ? -0x1.fffffep127f : -0.5f * ss;
}

// Insert (s, i) into a best-first list: a compare-exchange pass down the list
// carries the displaced entry along; the last one falls off.
template <int KMAX>
__device__ __forceinline__ void knn_insert(float (&v)[KMAX], int (&ix)[KMAX], float s, int i) {
#pragma unroll
  for (int t = 0; t < KMAX; ++t) {
    const bool up = s > v[t];
    const float vt = v[t];
    const int it = ix[t];
    v[t] = up ? s : vt;
    ix[t] = up ? i : it;
    s = up ? vt : s;
    i = up ? it : i;
  }
}

// The same, ordering equal scores by index (merging two lists).
template <int KMAX>
__device__ __forceinline__ void knn_insert_by_index(float (&v)[KMAX], int (&ix)[KMAX], float s,
                                                    int i) {
#pragma unroll
  for (int t = 0; t < KMAX; ++t) {
    const bool up = s > v[t] || (s == v[t] && i < ix[t]);
    const float vt = v[t];
    const int it = ix[t];
    v[t] = up ? s : vt;
    ix[t] = up ? i : it;
    s = up ? vt : s;
    i = up ? it : i;
  }
}

// The MFMAs of one 32-row tile (tile index at run time) into acc, one
// accumulator per 32-query tile: each row fragment read from LDS feeds NSUB
// MFMAs, and the scores are read once for all of them.
template <int DT, int CPL, int NSUB, int LOADS>
__device__ __forceinline__ void knn_mfma_tile(f32x16 (&acc)[NSUB], const uint4 (&xr)[NSUB][CPL],
                                              char* buf, const PipeOffsets<CPL, LOADS>& o,
                                              int tile) {
  using L = PipeLayout<CPL>;
  f32x16 cin;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const f32x4 v = lds_at<f32x4>(buf, o.n_read + (tile * 32 + 8 * q) * 4, 0);
    cin[4 * q + 0] = v[0];
    cin[4 * q + 1] = v[1];
    cin[4 * q + 2] = v[2];
    cin[4 * q + 3] = v[3];
  }
#pragma unroll
  for (int c = 0; c < CPL; ++c) {
    const uint4 a = lds_at<uint4>(buf, o.a[c] + tile * L::TILE, 0);
#pragma unroll
    for (int p = 0; p < NSUB; ++p) acc[p] = mfma32_chunk<DT>(a, xr[p][c], c == 0 ? cin : acc[p]);
  }
}

// Score j of the tile (a select chain: j differs per lane).
__device__ __forceinline__ float knn_pick(const f32x16& acc, int j) {
  float s = acc[0];
#pragma unroll
  for (int t = 1; t < 16; ++t) s = j == t ? acc[t] : s;
  return s;
}

// The top-k update of one tile: unless no lane's best score of the tile beats
// its KMAX-th best, the scores that do are marked, and while any lane has a
// mark left, each lane inserts its lowest marked score (so rows still enter
// in index order).
template <int KMAX>
__device__ __forceinline__ void knn_update(const f32x16& acc, int base, float (&v)[KMAX],
                                           int (&ix)[KMAX]) {
  // first the tile's best score (a max3 tree): once the lists have filled, no
  // lane's usually beats its KMAX-th best, and the tile costs 8 instructions
  const float t0 = __builtin_fmaxf(__builtin_fmaxf(acc[0], acc[1]), acc[2]);
  const float t1 = __builtin_fmaxf(__builtin_fmaxf(acc[3], acc[4]), acc[5]);
  const float t2 = __builtin_fmaxf(__builtin_fmaxf(acc[6], acc[7]), acc[8]);
  const float t3 = __builtin_fmaxf(__builtin_fmaxf(acc[9], acc[10]), acc[11]);
  const float t4 = __builtin_fmaxf(__builtin_fmaxf(acc[12], acc[13]), acc[14]);
  const float mx = __builtin_fmaxf(__builtin_fmaxf(__builtin_fmaxf(t0, t1), t2),
                                   __builtin_fmaxf(__builtin_fmaxf(t3, t4), acc[15]));
  if (!__ballot(mx > v[KMAX - 1])) return;
  uint32_t mark = 0;
#pragma unroll
  for (int j = 0; j < 16; ++j) mark |= (acc[j] > v[KMAX - 1] ? 1u : 0u) << j;
  while (__ballot(mark != 0)) {
    if (mark != 0) {
      const int j = __builtin_ctz(mark);
      mark &= mark - 1;
      const float sc = knn_pick(acc, j);
      // an earlier insertion may have raised the bar
      if (sc > v[KMAX - 1]) knn_insert<KMAX>(v, ix, sc, base + 8 * (j >> 2) + (j & 3));
    }
  }
}

// One stage in `cur`: start the next stage into `nxt` (a different LDS array,
// so no read of `cur` waits for it), then per 32-row tile the MFMAs and the
// top-k update; with 32-entry lists (one wave per SIMD, nothing else to hide
// behind) the MFMAs of the next tile run beside this tile's update (two
// accumulator sets: the matrix pipe and the vector ALU overlap only within a
// wave's own instruction stream).  Store the next stage's scores, wait for
// its loads and sync.
template <int DT, int CPL, int NSUB, int KMAX, int LOADS>
__device__ __forceinline__ void knn_stage(int st, int nst, char* cur, char* nxt,
                                          const PipeOffsets<CPL, LOADS>& o,
                                          const uint4 (&xr)[NSUB][CPL], const u32x4* chat4,
                                          const float* cinit, int tid, int h,
                                          float (&v)[NSUB][KMAX], int (&ix)[NSUB][KMAX]) {
  using L = PipeLayout<CPL>;
  const bool more = st + 1 < nst;
  float nn = 0.f;
  if (more) nn = pipe_issue_stage<CPL, LOADS>(chat4, cinit, st + 1, tid, o, nxt);
  if constexpr (KMAX > 16) {
    static_assert(NSUB == 1, "32-entry lists keep one query tile per wave");
    f32x16 acc[2][1];
    knn_mfma_tile<DT, CPL, 1, LOADS>(acc[0], xr, cur, o, 0);
#pragma unroll
    for (int tile = 0; tile < L::TILES; ++tile) {
      if (tile + 1 < L::TILES)
        knn_mfma_tile<DT, CPL, 1, LOADS>(acc[(tile + 1) & 1], xr, cur, o, tile + 1);
      knn_update<KMAX>(acc[tile & 1][0], (st * L::TILES + tile) * 32 + 4 * h, v[0], ix[0]);
    }
  } else {
    // within 256 registers the second accumulator set costs spills
    for (int tile = 0; tile < L::TILES; ++tile) {
      f32x16 acc[NSUB];
      knn_mfma_tile<DT, CPL, NSUB, LOADS>(acc, xr, cur, o, tile);
#pragma unroll
      for (int p = 0; p < NSUB; ++p)
        knn_update<KMAX>(acc[p], (st * L::TILES + tile) * 32 + 4 * h, v[p], ix[p]);
    }
  }
  if (more) lds_at<float>(nxt, o.n_store, 0) = nn;
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
}

// Lists of 8 or 16 fit two waves per SIMD (the update's latency then hides
// behind the other wave's MFMAs); 32 entries take the whole register file.
// NSUB 32-query tiles per wave: with two, each row fragment read from LDS
// feeds two MFMAs (with one, the four SIMDs' fragment and score reads ask
// more of the LDS than the matrix pipes take in).
template <int DT, int CPL, int NSUB, int KMAX>
__global__ __launch_bounds__(ASSIGN_THREADS, KMAX <= 16 ? 2 : 1) void knn_kernel(
    const uint4* __restrict__ Q, const uint4* __restrict__ chat, const float* __restrict__ cinit,
    int M, int Np, int k, int32_t* __restrict__ nbr_idx, float* __restrict__ nbr_dist) {
  using L = PipeLayout<CPL>;
  constexpr int RC = L::RC;
  constexpr int LOADS = L::TCS * L::RCP / ASSIGN_THREADS;
  static_assert(LOADS >= 1 && LOADS * ASSIGN_THREADS == L::TCS * L::RCP, "stage must split evenly");
  constexpr int QPW = 32 * NSUB, QPB = 4 * QPW;  // queries per wave, per workgroup

  __shared__ __attribute__((aligned(16))) char buf0[L::STAGE];
  __shared__ __attribute__((aligned(16))) char buf1[L::STAGE];

  const int b = blockIdx.y;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int n = lane & 31, h = lane >> 5;
  Q += (size_t)b * M * RC;
  const u32x4* chat4 = reinterpret_cast<const u32x4*>(chat) + (size_t)b * Np * RC;
  cinit += (size_t)b * Np;
  const int nst = Np / L::TCS;

  PipeOffsets<CPL, LOADS> o;
  pipe_offsets<CPL, LOADS>(o, tid, n, h);
  float nn = pipe_issue_stage<CPL, LOADS>(chat4, cinit, 0, tid, o, buf0);

  const int q0 = blockIdx.x * QPB + wave * QPW + n;  // this lane's query of tile 0
  uint4 xr[NSUB][CPL];
  float ss[NSUB];
#pragma unroll
  for (int p = 0; p < NSUB; ++p) {
    const int qt = q0 + 32 * p;
    float a = 0.f;
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
      xr[p][c] = qt < M ? Q[(size_t)qt * RC + h * CPL + c] : make_uint4(0, 0, 0, 0);
      a = chunk_sumsq<DT>(xr[p][c], a);
    }
    ss[p] = a + __shfl_xor(a, 32);
  }

  float v[NSUB][KMAX];
  int ix[NSUB][KMAX];
#pragma unroll
  for (int p = 0; p < NSUB; ++p)
#pragma unroll
    for (int t = 0; t < KMAX; ++t) {
      v[p][t] = -__builtin_inff();
      ix[p][t] = 0x7fffffff;
    }

  lds_at<float>(buf0, o.n_store, 0) = nn;
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  int st = 0;
  for (; st + 2 <= nst; st += 2) {  // two stages per trip: each buffer is a fixed array
    knn_stage<DT, CPL, NSUB, KMAX, LOADS>(st, nst, buf0, buf1, o, xr, chat4, cinit, tid, h, v, ix);
    knn_stage<DT, CPL, NSUB, KMAX, LOADS>(st + 1, nst, buf1, buf0, o, xr, chat4, cinit, tid, h, v,
                                          ix);
  }
  if (st < nst)
    knn_stage<DT, CPL, NSUB, KMAX, LOADS>(st, nst, buf0, buf1, o, xr, chat4, cinit, tid, h, v, ix);

#pragma unroll
  for (int p = 0; p < NSUB; ++p) {
    // merge the other half's list (rows 4..7 of each group of 8) into lane h = 0's
#pragma unroll
    for (int t = 0; t < KMAX; ++t) {
      const float so = __shfl_xor(v[p][t], 32);
      const int io = __shfl_xor(ix[p][t], 32);
      if (h == 0) knn_insert_by_index<KMAX>(v[p], ix[p], so, io);
    }
    const int qt = q0 + 32 * p;
    if (h == 0 && qt < M) {
      int32_t* oi = nbr_idx + ((size_t)b * M + qt) * k;
      float* od = nbr_dist + ((size_t)b * M + qt) * k;
#pragma unroll
      for (int t = 0; t < KMAX; ++t) {
        if (t < k) {
          oi[t] = ix[p][t];
          od[t] = __builtin_fmaxf(__builtin_fmaf(-2.f, v[p][t], ss[p]), 0.f);
        }
      }
    }
  }
}

// Two query tiles per wave where the lists leave room for them (16 entries
// and D <= 128, which keeps two waves per SIMD), else one.
template <int CPL, int KMAX>
constexpr int knn_nsub() { return KMAX <= 16 && CPL <= 8 ? 2 : 1; }

template <int DT, int CPL, int KMAX>
hipError_t launch_knn_cpl(const void* Q, const void* chat, const float* cinit, int64_t B,
                          int64_t M, int64_t Np, int k, int32_t* nbr_idx, float* nbr_dist,
                          hipStream_t s) {
  constexpr int NSUB = knn_nsub<CPL, KMAX>();
  constexpr int QPB = 4 * 32 * NSUB;
  const dim3 grid((unsigned)((M + QPB - 1) / QPB), (unsigned)B), block(ASSIGN_THREADS);
  knn_kernel<DT, CPL, NSUB, KMAX><<<grid, block, 0, s>>>((const uint4*)Q, (const uint4*)chat,
                                                         cinit, (int)M, (int)Np, k, nbr_idx,
                                                         nbr_dist);
  return hipGetLastError();
}

template <int DT, int KMAX>
hipError_t launch_knn_k(const void* Q, const void* chat, const float* cinit, int64_t B, int64_t M,
                        int64_t Np, int64_t D, int k, int32_t* nbr_idx, float* nbr_dist,
                        hipStream_t s) {
  switch (D / 16) {
#define FKM_KNN_CASE(c) \
  case c: return launch_knn_cpl<DT, c, KMAX>(Q, chat, cinit, B, M, Np, k, nbr_idx, nbr_dist, s);
    FKM_KNN_CASE(1) FKM_KNN_CASE(2) FKM_KNN_CASE(3) FKM_KNN_CASE(4)
    FKM_KNN_CASE(5) FKM_KNN_CASE(6) FKM_KNN_CASE(7) FKM_KNN_CASE(8)
    FKM_KNN_CASE(9) FKM_KNN_CASE(10) FKM_KNN_CASE(11) FKM_KNN_CASE(12)
    FKM_KNN_CASE(13) FKM_KNN_CASE(14) FKM_KNN_CASE(15) FKM_KNN_CASE(16)
#undef FKM_KNN_CASE
    default: return hipErrorInvalidValue;
  }
}

// prep + search for one storage type; k <= KNN_MAX_K.  R has rows of Din
// elements, Q (already padded) and the staged rows have D, D % 16 == 0, D <= 256.
template <int DT>
hipError_t launch_knn_dt(const void* Q, const void* R, int64_t B, int64_t M, int64_t N,
                         int64_t Din, int64_t D, int k, void* chat, float* cinit, int64_t Np,
                         int32_t* nbr_idx, float* nbr_dist, hipStream_t s) {
  if (D % 16 != 0 || D > 256 || Din > D || k < 1 || k > KNN_MAX_K || Np % ASSIGN_KPAD != 0)
    return hipErrorInvalidValue;
  knn_prep_kernel<DT><<<dim3((unsigned)((B * Np + 3) / 4)), 256, 0, s>>>(
      (const uint16_t*)R, B, (int)N, (int)Np, (int)Din, (int)D, (uint16_t*)chat, cinit);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (k <= 8) return launch_knn_k<DT, 8>(Q, chat, cinit, B, M, Np, D, k, nbr_idx, nbr_dist, s);
  if (k <= 10) return launch_knn_k<DT, 10>(Q, chat, cinit, B, M, Np, D, k, nbr_idx, nbr_dist, s);
  if (k <= 16) return launch_knn_k<DT, 16>(Q, chat, cinit, B, M, Np, D, k, nbr_idx, nbr_dist, s);
  return launch_knn_k<DT, KNN_MAX_K>(Q, chat, cinit, B, M, Np, D, k, nbr_idx, nbr_dist, s);
}

}  // namespace fkm
