// assign_tiled.hip -- the assignment step for wide rows (16-bit points with
// D >= 512), where a point no longer fits in registers.
//
// The distance contraction is tiled like a GEMM: a workgroup owns 256 points
// (4 waves x 64) and TILED_CBG consecutive 128-centroid blocks; for each block
// it streams D in 32-dimension stages through LDS (points and centroids, both
// double-buffered) and runs 32x32x16 MFMAs, 8 independent accumulators per
// wave (2 point tiles x 4 centroid tiles).  After each block an exact
// compare-and-select keeps each lane's best (score, index); after the group
// the workgroup merges its result into a per-point 64-bit key with atomicMax.
// The key is the score mapped to an order-preserving unsigned integer in the
// high half and the complemented index in the low half, so the maximum is the
// largest score and, among equal scores, the lowest index: the same result
// as a sequential scan, whatever order the workgroups finish in.
//
// Block order is XCD-aware: consecutive workgroup ids go to different XCDs,
// so the ids are remapped for each XCD to own whole point blocks (all their
// centroid groups run on one XCD and find the point block in that XCD's L2).
#include "fkm_device.h"

namespace fkm {

namespace {

constexpr int BP = 256;           // points per workgroup
constexpr int BC = TILED_BC;      // centroids per block
constexpr int DC = 32;            // dimensions per LDS stage
constexpr int CPS = DC * 2 / 16;  // 16-byte chunks of a row in one stage (4)
static_assert(BC == 128, "four 32-row tiles per centroid block");

// Row r of a stage keeps its 4 chunks in slots c ^ f(r); f spreads 16
// consecutive rows over distinct banks for 16-byte reads.
__device__ __forceinline__ int swz(int r) { return ((r >> 1) & 3) ^ ((r >> 3) & 1); }

__device__ __forceinline__ uint32_t ordered(float v) {
  const uint32_t u = __float_as_uint(v);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float unordered(uint32_t u) {
  return __uint_as_float((u & 0x80000000u) ? (u & 0x7fffffffu) : ~u);
}

struct TiledStage {
  u32x4 x[4], c[2];  // native vectors: the stage stays in registers
  float n;
};

__device__ __forceinline__ void tiled_load(TiledStage& g, const uint4* __restrict__ X,
                                           const uint4* __restrict__ chat,
                                           const float* __restrict__ cinit, int s, int nds, int p0,
                                           int cb0, int N, int RC, int tid) {
  const int gb = s / nds, ds = s % nds;
  const u32x4* x4 = reinterpret_cast<const u32x4*>(X);
  const u32x4* c4 = reinterpret_cast<const u32x4*>(chat);
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int q = tid + u * 256, r = q >> 2, c = q & 3;
    g.x[u] = p0 + r < N ? x4[(size_t)(p0 + r) * RC + ds * CPS + c] : u32x4{0u, 0u, 0u, 0u};
  }
  const int crow = (cb0 + gb) * BC;
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int q = tid + u * 256, r = q >> 2, c = q & 3;
    g.c[u] = c4[(size_t)(crow + r) * RC + ds * CPS + c];
  }
  g.n = cinit[crow + (tid & (BC - 1))];
}

__device__ __forceinline__ void tiled_store(const TiledStage& g, uint4* lx, uint4* lc, float* ln,
                                            int tid) {
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int q = tid + u * 256, r = q >> 2, c = q & 3;
    reinterpret_cast<u32x4*>(lx)[r * CPS + (c ^ swz(r))] = g.x[u];
  }
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int q = tid + u * 256, r = q >> 2, c = q & 3;
    reinterpret_cast<u32x4*>(lc)[r * CPS + (c ^ swz(r))] = g.c[u];
  }
  ln[tid & (BC - 1)] = g.n;
}

}  // namespace

template <int DT>
__global__ __launch_bounds__(256, 2) void assign_tiled_kernel(
    const uint4* __restrict__ X, const uint4* __restrict__ chat, const float* __restrict__ cinit,
    int N, int D, int Kp, int npb, int ncbg, uint64_t* __restrict__ keys,
    float* __restrict__ xnorm) {
  __shared__ uint4 lx[2][BP * CPS];                              // 2 x 16 KiB
  __shared__ uint4 lc[2][BC * CPS];                              // 2 x 8 KiB
  __shared__ __attribute__((aligned(16))) float ln[2][BC];

  const int b = blockIdx.y;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int n = lane & 31, h = lane >> 5;
  // XCD-aware remap: XCD x (= id % 8) takes point blocks x, x + 8, ... in turn,
  // each with all of its centroid groups
  const int xcd = blockIdx.x & 7, j = blockIdx.x >> 3;
  const int pb = xcd + 8 * (j / ncbg), cbg = j % ncbg;
  if (pb >= npb) return;
  const int ncb = Kp / BC;
  const int cb0 = cbg * TILED_CBG;
  const int ncbw = min(TILED_CBG, ncb - cb0);  // centroid blocks of this workgroup
  const int RC = D / 8;                         // 16-byte chunks per row
  const int nds = D / DC;                       // stages per centroid block
  const int S = ncbw * nds;
  X += (size_t)b * N * RC;
  chat += (size_t)b * Kp * RC;
  cinit += (size_t)b * Kp;
  const int p0 = pb * BP;
  const bool do_norm = cbg == 0;

  // stage s: centroid block cb0 + s / nds, dimensions [32 (s % nds), +32)
  TiledStage pre;
  f32x16 acc[2][4];
  float best[2] = {-__builtin_inff(), -__builtin_inff()};
  int bidx[2] = {0, 0};
  float xs = 0.f;  // squared norm of point p0 + tid (first group only)

  tiled_load(pre, X, chat, cinit, 0, nds, p0, cb0, N, RC, tid);
  tiled_store(pre, lx[0], lc[0], ln[0], tid);
  __syncthreads();
  for (int s = 0; s < S; ++s) {
    const int buf = s & 1;
    const int g = s / nds, ds = s % nds;
    if (s + 1 < S) tiled_load(pre, X, chat, cinit, s + 1, nds, p0, cb0, N, RC, tid);
    if (ds == 0) {
#pragma unroll
      for (int tc = 0; tc < 4; ++tc) {
        f32x16 cin;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const f32x4 v = *reinterpret_cast<const f32x4*>(&ln[buf][tc * 32 + 8 * q + 4 * h]);
          cin[4 * q + 0] = v[0];
          cin[4 * q + 1] = v[1];
          cin[4 * q + 2] = v[2];
          cin[4 * q + 3] = v[3];
        }
        acc[0][tc] = cin;
        acc[1][tc] = cin;
      }
    }
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const int c = 2 * ks + h;
      uint4 a[4], bx[2];
#pragma unroll
      for (int tc = 0; tc < 4; ++tc) {
        const int r = tc * 32 + n;
        a[tc] = lc[buf][r * CPS + (c ^ swz(r))];
      }
#pragma unroll
      for (int tp = 0; tp < 2; ++tp) {
        const int r = wave * 64 + tp * 32 + n;
        bx[tp] = lx[buf][r * CPS + (c ^ swz(r))];
      }
#pragma unroll
      for (int tp = 0; tp < 2; ++tp)
#pragma unroll
        for (int tc = 0; tc < 4; ++tc) acc[tp][tc] = mfma32_chunk<DT>(a[tc], bx[tp], acc[tp][tc]);
    }
    if (do_norm && g == 0) {  // |x|^2 of point p0 + tid, in dimension order
      const int r = tid;
#pragma unroll
      for (int c = 0; c < CPS; ++c) xs = chunk_sumsq<DT>(lx[buf][r * CPS + (c ^ swz(r))], xs);
    }
    if (ds == nds - 1) {  // this centroid block is complete: exact running arg-max
      const int kb = (cb0 + g) * BC;
#pragma unroll
      for (int tp = 0; tp < 2; ++tp)
#pragma unroll
        for (int tc = 0; tc < 4; ++tc)
#pragma unroll
          for (int jj = 0; jj < 16; ++jj) {
            const float v = acc[tp][tc][jj];
            const bool gt = v > best[tp];
            best[tp] = gt ? v : best[tp];
            bidx[tp] = gt ? kb + tc * 32 + 8 * (jj >> 2) + (jj & 3) : bidx[tp];
          }
    }
    if (s + 1 < S) tiled_store(pre, lx[buf ^ 1], lc[buf ^ 1], ln[buf ^ 1], tid);
    __syncthreads();
  }

  // merge the two row halves of each point, then one atomic per point
#pragma unroll
  for (int tp = 0; tp < 2; ++tp) {
    float v = best[tp];
    int i = bidx[tp] + 4 * h;
    const float vo = __shfl_xor(v, 32);
    const int io = __shfl_xor(i, 32);
    const bool take = (vo > v) || (vo == v && io < i);
    v = take ? vo : v;
    i = take ? io : i;
    const int pt = p0 + wave * 64 + tp * 32 + n;
    if (h == 0 && pt < N) {
      const uint64_t key = ((uint64_t)ordered(v) << 32) | (uint64_t)(0xffffffffu - (uint32_t)i);
      atomicMax((unsigned long long*)&keys[(size_t)b * N + pt], (unsigned long long)key);
    }
  }
  if (do_norm && p0 + tid < N) xnorm[(size_t)b * N + p0 + tid] = xs;
}

__global__ __launch_bounds__(256) void fill_keys_kernel(uint64_t* __restrict__ keys, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n) keys[i] = 0;
}

// idx, min_dist and per-block objective partials from the keys.
__global__ __launch_bounds__(256) void decode_keys_kernel(const uint64_t* __restrict__ keys,
                                                          const float* __restrict__ xnorm, int N,
                                                          int32_t* __restrict__ idx,
                                                          float* __restrict__ min_dist,
                                                          double* __restrict__ objpart) {
  __shared__ double s[256];
  const int b = blockIdx.y;
  const int i = blockIdx.x * 256 + threadIdx.x;
  double md = 0.0;
  if (i < N) {
    const uint64_t key = keys[(size_t)b * N + i];
    const float v = unordered((uint32_t)(key >> 32));
    const float d = __builtin_fmaxf(__builtin_fmaf(-2.f, v, xnorm[(size_t)b * N + i]), 0.f);
    idx[(size_t)b * N + i] = (int32_t)(0xffffffffu - (uint32_t)key);
    min_dist[(size_t)b * N + i] = d;
    md = d;
  }
  s[threadIdx.x] = md;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) s[threadIdx.x] += s[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) objpart[(size_t)b * gridDim.x + blockIdx.x] = s[0];
}

hipError_t launch_assign_tiled(const void* X, int dt, const Workspace& w, int64_t B, int64_t N,
                               int64_t D, int32_t* idx, float* min_dist, hipStream_t s) {
  const int64_t nk = B * N;
  fill_keys_kernel<<<dim3((unsigned)((nk + 255) / 256)), 256, 0, s>>>(w.keys, nk);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int npb = (int)((N + BP - 1) / BP);
  const int ncb = (int)(w.Kp / BC);
  const int ncbg = (ncb + TILED_CBG - 1) / TILED_CBG;
  const int npb8 = (npb + 7) / 8 * 8;
  const dim3 grid((unsigned)(npb8 * ncbg), (unsigned)B);
  if (dt == DT_BF16)
    assign_tiled_kernel<DT_BF16><<<grid, 256, 0, s>>>((const uint4*)X, (const uint4*)w.chat,
                                                      w.cinit, (int)N, (int)D, (int)w.Kp, npb,
                                                      ncbg, w.keys, w.xnorm);
  else
    assign_tiled_kernel<DT_F16><<<grid, 256, 0, s>>>((const uint4*)X, (const uint4*)w.chat,
                                                     w.cinit, (int)N, (int)D, (int)w.Kp, npb,
                                                     ncbg, w.keys, w.xnorm);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  decode_keys_kernel<<<dim3((unsigned)w.n_assign_blocks, (unsigned)B), 256, 0, s>>>(
      w.keys, w.xnorm, (int)N, idx, min_dist, w.objpart);
  return hipGetLastError();
}

}  // namespace fkm
