// update.hip -- the centroid update of the Lloyd iteration (paper Section 5:
// reduce the points of each cluster into per-cluster sums and counts).
//
// The paper calls this step bandwidth- and atomic-contention-sensitive.  Here
// it uses no floating-point atomics and is deterministic:
//   1. hist      per chunk of SORT_WC points, a histogram over the K clusters
//   2. colsum    per segment of SORT_SEG chunks, the sum of those histograms
//   3. colscan   per cluster, an exclusive scan over segments; the total is count_k
//   4. kscan     per instance, an exclusive scan of the counts: cluster offsets
//   5. downsweep per (chunk, cluster), the absolute start of that chunk's run
//   6. scatter   one wave per chunk ranks its points in order (ballot
//                multi-split) and writes them to their sorted slots: a stable
//                counting sort of the point ids by cluster
//   7. segreduce one wave per RED_CR consecutive sorted entries streams the
//                whole rows X[perm[j]] and sums each cluster run in fp32 in a
//                fixed order; a run cut by a chunk end leaves a partial
//   8. finalize  per cluster, the sum (or its partials, in chunk order) over
//                the count; an empty cluster keeps its previous centroid.
#include "fkm_internal.h"

namespace fkm {

// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void hist_kernel(const int32_t* __restrict__ idx, int N, int K,
                                                   int nch, int32_t* __restrict__ H) {
  extern __shared__ int32_t cnt[];
  const int b = blockIdx.y, ch = blockIdx.x;
  for (int k = threadIdx.x; k < K; k += 256) cnt[k] = 0;
  __syncthreads();
  const int i0 = ch * SORT_WC;
  const int i1 = min(N, i0 + SORT_WC);
  const int32_t* ib = idx + (size_t)b * N;
  constexpr int PER = SORT_WC / 256;
  int keys[PER];
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    const int i = i0 + u * 256 + (int)threadIdx.x;
    keys[u] = i < i1 ? ib[i] : -1;
  }
#pragma unroll
  for (int u = 0; u < PER; ++u)
    if ((unsigned)keys[u] < (unsigned)K) atomicAdd(&cnt[keys[u]], 1);  // out-of-range ids are ignored
  __syncthreads();
  int32_t* out = H + ((size_t)b * nch + ch) * K;
  for (int k = threadIdx.x; k < K; k += 256) out[k] = cnt[k];
}

__global__ __launch_bounds__(256) void colsum_kernel(const int32_t* __restrict__ H, int K, int nch,
                                                     int nseg, int32_t* __restrict__ T) {
  const int k = blockIdx.x * 256 + threadIdx.x;
  const int s = blockIdx.y, b = blockIdx.z;
  if (k >= K) return;
  const int c0 = s * SORT_SEG, c1 = min(nch, c0 + SORT_SEG);
  const int32_t* h = H + (size_t)b * nch * K + k;
  int sum = 0;
#pragma unroll 8
  for (int c = c0; c < c1; ++c) sum += h[(size_t)c * K];
  T[((size_t)b * nseg + s) * K + k] = sum;
}

__global__ __launch_bounds__(256) void colscan_kernel(int32_t* __restrict__ T, int K, int nseg,
                                                      int32_t* __restrict__ counts) {
  const int k = blockIdx.x * 256 + threadIdx.x;
  const int b = blockIdx.y;
  if (k >= K) return;
  int32_t* t = T + (size_t)b * nseg * K + k;
  int run = 0;
  for (int s0 = 0; s0 < nseg; s0 += 16) {   // 16 independent loads in flight
    int v[16];
#pragma unroll
    for (int u = 0; u < 16; ++u) v[u] = s0 + u < nseg ? t[(size_t)(s0 + u) * K] : 0;
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      if (s0 + u < nseg) t[(size_t)(s0 + u) * K] = run;
      run += v[u];
    }
  }
  counts[(size_t)b * K + k] = run;
}

// Exclusive scan of one instance's K counts into K+1 offsets (1024 threads).
__global__ __launch_bounds__(1024) void kscan_kernel(const int32_t* __restrict__ counts, int K,
                                                     int32_t* __restrict__ off) {
  __shared__ int32_t part[1024];
  const int b = blockIdx.x, t = threadIdx.x;
  const int per = (K + 1023) / 1024;
  const int k0 = min(K, t * per), k1 = min(K, k0 + per);
  const int32_t* c = counts + (size_t)b * K;
  int sum = 0;
  for (int k = k0; k < k1; ++k) sum += c[k];
  part[t] = sum;
  __syncthreads();
  for (int w = 1; w < 1024; w <<= 1) {  // Hillis-Steele inclusive scan
    const int v = t >= w ? part[t - w] : 0;
    __syncthreads();
    part[t] += v;
    __syncthreads();
  }
  int run = part[t] - sum;
  int32_t* o = off + (size_t)b * (K + 1);
  for (int k = k0; k < k1; ++k) {
    o[k] = run;
    run += c[k];
  }
  if (t == 1023) o[K] = part[1023];
}

__global__ __launch_bounds__(256) void downsweep_kernel(int32_t* __restrict__ H,
                                                        const int32_t* __restrict__ T,
                                                        const int32_t* __restrict__ off, int K,
                                                        int nch, int nseg) {
  const int k = blockIdx.x * 256 + threadIdx.x;
  const int s = blockIdx.y, b = blockIdx.z;
  if (k >= K) return;
  int base = off[(size_t)b * (K + 1) + k] + T[((size_t)b * nseg + s) * K + k];
  const int c0 = s * SORT_SEG, c1 = min(nch, c0 + SORT_SEG);
  int32_t* h = H + (size_t)b * nch * K + k;
  int v[SORT_SEG];
#pragma unroll
  for (int u = 0; u < SORT_SEG; ++u) v[u] = c0 + u < c1 ? h[(size_t)(c0 + u) * K] : 0;
#pragma unroll
  for (int u = 0; u < SORT_SEG; ++u) {
    if (c0 + u < c1) h[(size_t)(c0 + u) * K] = base;
    base += v[u];
  }
}

// One wave per chunk: points are taken 64 at a time in index order; lanes
// that share a cluster id find each other with one ballot per key bit, rank
// themselves by lane order, and the first of them advances the LDS cursor.
// The chunk's ids are loaded into registers up front, so no step waits on
// global memory.
__global__ __launch_bounds__(64) void scatter_kernel(const int32_t* __restrict__ idx,
                                                     const int32_t* __restrict__ P, int N, int K,
                                                     int nch, int nbits,
                                                     int32_t* __restrict__ perm) {
  constexpr int STEPS = SORT_WC / 64;
  extern __shared__ int32_t cur[];
  const int b = blockIdx.y, ch = blockIdx.x;
  const int lane = threadIdx.x;
  const int32_t* ib = idx + (size_t)b * N;
  int32_t* pb = perm + (size_t)b * N;
  const int i0 = ch * SORT_WC;
  const int i1 = min(N, i0 + SORT_WC);
  int keys[STEPS];
#pragma unroll
  for (int s = 0; s < STEPS; ++s) {
    const int i = i0 + s * 64 + lane;
    keys[s] = i < i1 ? ib[i] : -1;
  }
  // this chunk's run starts: K ints, copied 16 loads in flight at a time
  const int32_t* p = P + ((size_t)b * nch + ch) * K;
  for (int k0 = 0; k0 < K; k0 += 16 * 64) {
    int v[16];
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      const int k = k0 + u * 64 + lane;
      v[u] = k < K ? p[k] : 0;
    }
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      const int k = k0 + u * 64 + lane;
      if (k < K) cur[k] = v[u];
    }
  }
  __syncthreads();
  const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
#pragma unroll
  for (int s = 0; s < STEPS; ++s) {
    const int raw = keys[s];
    const bool valid = (unsigned)raw < (unsigned)K;  // out-of-range ids (and the tail) are ignored
    const int key = valid ? raw : 0;
    uint64_t match = __ballot(valid);
    for (int bit = 0; bit < nbits; ++bit) {
      const bool on = (key >> bit) & 1;
      const uint64_t bb = __ballot(valid && on);
      match &= on ? bb : ~bb;
    }
    if (valid) {
      const int rank = __popcll(match & below);
      const int start = cur[key];
      if (rank == 0) cur[key] = start + __popcll(match);
      pb[start + rank] = i0 + s * 64 + lane;
    }
  }
}

// ---------------------------------------------------------------------------
// Segmented sum.  A row of D elements is RC 16-byte chunks; LPR lanes share a
// row (CPLR chunks each) and a wave covers RPW = 64 / LPR rows per step.
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
    int N, int K, int nred, float* __restrict__ sums, float* __restrict__ carry) {
  constexpr int E = Row<DT>::per16;
  constexpr int RC = LPR * CPLR;
  constexpr int D = RC * E;
  constexpr int RPW = 64 / LPR;
  constexpr int NA = CPLR * E;
  constexpr int U = 8;  // rows in flight per lane
  const int lane = threadIdx.x & 63;
  const int w = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int b = blockIdx.y;
  if (w >= nred) return;
  const int32_t* ob = off + (size_t)b * (K + 1);
  const int j0 = w * RED_CR;
  const int j1 = min(ob[K], j0 + RED_CR);  // ob[K] = number of sorted (valid) entries
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
          for (int c = 0; c < CPLR; ++c) v[u][c] = row[c];
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

// One workgroup per cluster: each thread owns 4 consecutive dimensions; the
// (256 / (D/4)) row slots split a long list of partials and are combined in
// a fixed order through LDS.
__global__ __launch_bounds__(256) void finalize_kernel(
    const float* __restrict__ sums, const float* __restrict__ carry,
    const int32_t* __restrict__ counts, const int32_t* __restrict__ off,
    const float* C_prev, int K, int D, int nred, float* C_out) {
  extern __shared__ float4 part[];
  const int k = blockIdx.x, b = blockIdx.y;
  const int t = threadIdx.x;
  const int D4 = D / 4;
  const int slots = D4 >= 256 ? 1 : 256 / D4;
  const size_t rowoff = ((size_t)b * K + k) * D;
  const int n = counts[(size_t)b * K + k];
  if (n == 0) {
    for (int d = t; d < D4; d += 256)
      reinterpret_cast<float4*>(C_out + rowoff)[d] = reinterpret_cast<const float4*>(C_prev + rowoff)[d];
    return;
  }
  const int j0 = off[(size_t)b * (K + 1) + k], j1 = off[(size_t)b * (K + 1) + k + 1];
  const int c0 = j0 / RED_CR, c1 = (j1 - 1) / RED_CR;
  const float fn = (float)n;
  if (c0 == c1) {
    for (int d = t; d < D4; d += 256) {
      const float4 s = reinterpret_cast<const float4*>(sums + rowoff)[d];
      reinterpret_cast<float4*>(C_out + rowoff)[d] =
          make_float4(s.x / fn, s.y / fn, s.z / fn, s.w / fn);
    }
    return;
  }
  const int slot = (D4 >= 256) ? 0 : t / D4;
  for (int d0 = 0; d0 < D4; d0 += 256) {
    const int d = d0 + (D4 >= 256 ? t : t % D4);
    float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
    if (slot < slots && d < D4) {
      for (int c = c0 + slot; c <= c1; c += slots) {
        const int which = (c == c0 && j0 > c * RED_CR) ? 1 : 0;
        const float4 v = reinterpret_cast<const float4*>(
            carry + (((size_t)b * nred + c) * 2 + which) * D)[d];
        s.x += v.x; s.y += v.y; s.z += v.z; s.w += v.w;
      }
    }
    __syncthreads();
    part[t] = s;
    __syncthreads();
    if (slot == 0 && d < D4) {
      for (int u = 1; u < slots; ++u) {
        const float4 v = part[u * D4 + (t % D4)];
        s.x += v.x; s.y += v.y; s.z += v.z; s.w += v.w;
      }
      reinterpret_cast<float4*>(C_out + rowoff)[d] =
          make_float4(s.x / fn, s.y / fn, s.z / fn, s.w / fn);
    }
  }
}

// ---------------------------------------------------------------------------
template <int DT, int LPR, int CPLR>
static void launch_segreduce(const void* X, const Workspace& w, int64_t B, int64_t N, int64_t K,
                             hipStream_t s) {
  const dim3 grid((unsigned)((w.n_red_chunks + 3) / 4), (unsigned)B), block(256);
  segreduce_kernel<DT, LPR, CPLR><<<grid, block, 0, s>>>((const uint4*)X, w.perm, w.off, (int)N,
                                                         (int)K, (int)w.n_red_chunks, w.sums,
                                                         w.carry);
}

template <int DT>
static hipError_t launch_segreduce_dt(const void* X, const Workspace& w, int64_t B, int64_t N,
                                      int64_t D, int64_t K, hipStream_t s) {
  const int64_t rc = D * dt_bytes(DT) / 16;  // 16-byte chunks per row (D % 32 == 0 => rc % 4 == 0)
  if (rc <= 64) {
    switch (rc) {
      case 4: launch_segreduce<DT, 4, 1>(X, w, B, N, K, s); break;
      case 8: launch_segreduce<DT, 8, 1>(X, w, B, N, K, s); break;
      case 16: launch_segreduce<DT, 16, 1>(X, w, B, N, K, s); break;
      case 32: launch_segreduce<DT, 32, 1>(X, w, B, N, K, s); break;
      case 64: launch_segreduce<DT, 64, 1>(X, w, B, N, K, s); break;
      default: return hipErrorInvalidValue;
    }
  } else {
    switch (rc / 64) {
      case 2: if (rc == 128) { launch_segreduce<DT, 64, 2>(X, w, B, N, K, s); break; } return hipErrorInvalidValue;
      case 4: if (rc == 256) { launch_segreduce<DT, 64, 4>(X, w, B, N, K, s); break; } return hipErrorInvalidValue;
      case 8: if (rc == 512) { launch_segreduce<DT, 64, 8>(X, w, B, N, K, s); break; } return hipErrorInvalidValue;
      default: return hipErrorInvalidValue;
    }
  }
  return hipGetLastError();
}

hipError_t update_init() {
  // The histogram and scatter kernels keep K int32 counters in dynamic LDS.
  const int bytes = 4 * MAX_K;
  hipError_t e = hipFuncSetAttribute((const void*)hist_kernel,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
  if (e != hipSuccess) return e;
  return hipFuncSetAttribute((const void*)scatter_kernel,
                             hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
}

hipError_t launch_update(const void* X, int dt, const int32_t* idx, const float* C_prev,
                         const Workspace& w, int64_t B, int64_t N, int64_t D, int64_t K,
                         float* C_out, int32_t* counts, hipStream_t s) {
  hipError_t e;
  const int nch = (int)w.n_sort_chunks, nseg = (int)w.n_seg;
  const unsigned kb = (unsigned)((K + 255) / 256);
  hist_kernel<<<dim3(nch, (unsigned)B), 256, K * sizeof(int32_t), s>>>(idx, (int)N, (int)K, nch,
                                                                      w.hist);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  colsum_kernel<<<dim3(kb, nseg, (unsigned)B), 256, 0, s>>>(w.hist, (int)K, nch, nseg, w.segsum);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  colscan_kernel<<<dim3(kb, (unsigned)B), 256, 0, s>>>(w.segsum, (int)K, nseg, counts);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  kscan_kernel<<<dim3((unsigned)B), 1024, 0, s>>>(counts, (int)K, w.off);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  downsweep_kernel<<<dim3(kb, nseg, (unsigned)B), 256, 0, s>>>(w.hist, w.segsum, w.off, (int)K,
                                                               nch, nseg);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  int nbits = 0;
  while ((1ll << nbits) < K) ++nbits;
  scatter_kernel<<<dim3(nch, (unsigned)B), 64, K * sizeof(int32_t), s>>>(idx, w.hist, (int)N,
                                                                        (int)K, nch, nbits, w.perm);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (dt == DT_BF16) e = launch_segreduce_dt<DT_BF16>(X, w, B, N, D, K, s);
  else if (dt == DT_F16) e = launch_segreduce_dt<DT_F16>(X, w, B, N, D, K, s);
  else e = launch_segreduce_dt<DT_F32>(X, w, B, N, D, K, s);
  if (e != hipSuccess) return e;
  const size_t part_bytes = 256 * sizeof(float4);
  finalize_kernel<<<dim3((unsigned)K, (unsigned)B), 256, part_bytes, s>>>(
      w.sums, w.carry, counts, w.off, C_prev, (int)K, (int)D, (int)w.n_red_chunks, C_out);
  return hipGetLastError();
}

}  // namespace fkm
