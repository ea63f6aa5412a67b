// assign_smallk.h -- the Lloyd step for small K (16-bit rows of 32 to 96
// elements, K <= 256) in one pass over X: each workgroup assigns 2,048
// consecutive points and sums them per cluster, so the update's partial sums
// cost no second read of the points.  The same kernel without the sums is the
// assignment for these shapes, and without the assignment (indices read from
// memory) the update's sums, so a fused iteration and an assignment followed
// by an update give identical bits.
// Instantiated once per storage type in assign_smallk_bf16.hip and
// assign_smallk_f16.hip.
//
// Layout.  A workgroup (4 waves) walks 16 tiles of 128 points; each wave
// holds its 32 points of a tile in registers in the assignment's B-operand
// layout (lane 32 h + n: point n, dimensions 8 (h CPL + c) + e), and loads the
// next tile's points while it works on this one.  The centroids (at most two
// 128-row stages) stay in LDS for all 16 tiles.  Scores are shifted per point
// (the packed-key epilogue of the streaming kernel with each point's own
// bound), since one shift per workgroup would change from tile to tile.
//
// Sums.  S[k][d] = sum of x_i[d] over the points i with idx_i = k comes from
// MFMAs with a one-hot matrix.  The contraction must run over points, so each
// wave writes its tile transposed into its own LDS area (dimension-major, 64
// bytes of 32 points per dimension); for each 16-point step the A operand of
// lane 32 h + m is the one-hot column of cluster 32 kt + m over points
// 8 h .. 8 h + 7 (1.0 where the point's index is the cluster, else 0) and B is
// dimension 32 dt + n of the same points, one 16-byte LDS read.  A wave
// accumulates KTM x DTL 32x32 tiles in registers over all its tiles; at the
// end the four waves' tiles are added in wave order through LDS and written
// as the workgroup's partial [K, D]; counts come from LDS integer adds.  No
// floating-point atomic is used and every addition has a fixed order, so the
// sums are bitwise repeatable; products with the one-hot are exact and the
// sums accumulate in fp32.
#pragma once

#include "assign_pipe.h"

namespace fkm {

constexpr int SK_TILE = 128;                    // points per workgroup tile
constexpr int SK_TILES = SMALLK_CH / SK_TILE;   // tiles per workgroup

template <int CPL>
struct SkLayout {
  static constexpr int DTL = (CPL + 1) / 2;          // 32-dimension tiles
  static constexpr int XT = 32 * DTL * 64;           // bytes of one wave's transposed tile
  static constexpr int XT_ALL = 4 * XT > 16384 ? 4 * XT : 16384;  // also holds 4 fp32 32x32 tiles
};

// 8 one-hot 16-bit values (1.0 where iv == cl) packed into an MFMA operand.
template <int DT>
__device__ __forceinline__ uint4 onehot8(const int (&iv)[8], int cl) {
  constexpr uint32_t ONE = DT == DT_BF16 ? 0x3F80u : 0x3C00u;
  uint32_t w[4];
#pragma unroll
  for (int e = 0; e < 4; ++e)
    w[e] = (iv[2 * e] == cl ? ONE : 0u) | ((iv[2 * e + 1] == cl ? ONE : 0u) << 16);
  return make_uint4(w[0], w[1], w[2], w[3]);
}

// The first NT (2 or 4) 32-centroid tiles of one resident stage, in index
// order: K <= 64 needs only two (the rest of the stage is padding).
template <int DT, int CPL, int LOADS, int NT>
__device__ __forceinline__ void sk_stage(const uint4 (&xr)[1][CPL], char* buf,
                                         const PipeOffsets<CPL, LOADS>& o, uint32_t tb,
                                         const float (&Qp)[1], float (&best)[1],
                                         uint32_t (&code)[1]) {
  static_assert(NT == 2 || NT == 4, "two or four tiles");
  f32x16 a0[1], a1[1];
  pipe_mfma_tile<DT, 0, CPL, 1, LOADS>(a0, xr, buf, o);
  pipe_mfma_tile<DT, 1, CPL, 1, LOADS>(a1, xr, buf, o);
  pipe_epilogue<1, true>(a0, tb << 4, best, code, Qp);
  if constexpr (NT == 4) {
    pipe_mfma_tile<DT, 2, CPL, 1, LOADS>(a0, xr, buf, o);
    pipe_epilogue<1, true>(a1, (tb + 1) << 4, best, code, Qp);
    pipe_mfma_tile<DT, 3, CPL, 1, LOADS>(a1, xr, buf, o);
    pipe_epilogue<1, true>(a0, (tb + 2) << 4, best, code, Qp);
    pipe_epilogue<1, true>(a1, (tb + 3) << 4, best, code, Qp);
  } else {
    pipe_epilogue<1, true>(a1, (tb + 1) << 4, best, code, Qp);
  }
}

// The LDS area a wave transposes through is its own, so between its writes
// and its reads only this wave's LDS accesses need to be complete: wait for
// them (lgkmcnt(0); the vector-memory loads of the next tile stay in flight,
// where a memory fence would wait for them too) and keep the compiler from
// moving LDS accesses across.
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_s_waitcnt(0xC07F);  // vmcnt and expcnt at their maxima, lgkmcnt 0
  __builtin_amdgcn_wave_barrier();
  asm volatile("" ::: "memory");
}

// One wave's tile of 32 points into its sum tiles.
template <int DT, int CPL, int KTM>
__device__ __forceinline__ void sk_sums(const uint4 (&xr)[1][CPL], int i, bool ok, char* xt,
                                        int* widx, int* lds_cnt, int n, int h, int K, int KT,
                                        f32x16 (&S)[KTM][SkLayout<CPL>::DTL]) {
  constexpr int DTL = SkLayout<CPL>::DTL;
  // a point outside every cluster enters as zeros (its one-hot column is zero,
  // and zero times a non-finite coordinate would still be NaN)
  const bool in = ok && i >= 0 && i < K;
#pragma unroll
  for (int c = 0; c < CPL; ++c) {
    const uint32_t w[4] = {in ? xr[0][c].x : 0u, in ? xr[0][c].y : 0u, in ? xr[0][c].z : 0u,
                           in ? xr[0][c].w : 0u};
    const int d0 = (h * CPL + c) * 8;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      *reinterpret_cast<uint16_t*>(xt + (d0 + 2 * e) * 64 + n * 2) = (uint16_t)(w[e] & 0xffffu);
      *reinterpret_cast<uint16_t*>(xt + (d0 + 2 * e + 1) * 64 + n * 2) = (uint16_t)(w[e] >> 16);
    }
  }
  if (h == 0) {
    widx[n] = in ? i : -1;
    if (in) atomicAdd(&lds_cnt[i], 1);
  }
  wave_lds_sync();
#pragma unroll
  for (int s2 = 0; s2 < 2; ++s2) {
    const int4 i0 = *reinterpret_cast<const int4*>(widx + 16 * s2 + 8 * h);
    const int4 i1 = *reinterpret_cast<const int4*>(widx + 16 * s2 + 8 * h + 4);
    const int iv[8] = {i0.x, i0.y, i0.z, i0.w, i1.x, i1.y, i1.z, i1.w};
    uint4 bx[DTL];
#pragma unroll
    for (int dt = 0; dt < DTL; ++dt)
      bx[dt] = *reinterpret_cast<const uint4*>(xt + (32 * dt + n) * 64 + (16 * s2 + 8 * h) * 2);
#pragma unroll
    for (int kt = 0; kt < KTM; ++kt) {
      if (kt < KT) {
        const uint4 a = onehot8<DT>(iv, 32 * kt + n);
#pragma unroll
        for (int dt = 0; dt < DTL; ++dt) S[kt][dt] = mfma32_chunk<DT>(a, bx[dt], S[kt][dt]);
      }
    }
  }
  wave_lds_sync();
}

template <int DT, int CPL, int KTM, int MODE>
__global__ __launch_bounds__(ASSIGN_THREADS, 2) void assign_smallk_kernel(
    const uint4* __restrict__ X, const uint4* __restrict__ chat, const float* __restrict__ cinit,
    int N, int K, int Kp, int32_t* __restrict__ idx, float* __restrict__ min_dist,
    double* __restrict__ objpart, float* __restrict__ partial, int32_t* __restrict__ pcount) {
  static_assert(DT != DT_F32 && CPL >= 2 && CPL <= 6, "16-bit rows of 32 to 96 elements");
  using L = PipeLayout<CPL>;
  using SL = SkLayout<CPL>;
  constexpr int RC = L::RC, D = 16 * CPL, DTL = SL::DTL;
  static_assert(L::TILES == 4 && KTM * DTL <= 8, "128-row stages; at most 8 sum tiles");
  constexpr int LOADS = L::TCS * L::RCP / ASSIGN_THREADS;
  // K <= 128 takes one stage; two only when K > 128, which needs KTM = 8 (DTL = 1)
  constexpr bool TWO = KTM * 32 > L::TCS;

  constexpr bool ASSIGN = MODE != SUMS_ONLY, SUMS = MODE != SUMS_ASSIGN;
  __shared__ __attribute__((aligned(16))) char buf0[ASSIGN ? L::STAGE : 16];
  __shared__ __attribute__((aligned(16))) char buf1[ASSIGN && TWO ? L::STAGE : 16];
  __shared__ __attribute__((aligned(16))) char xt_all[SUMS ? SL::XT_ALL : 16];
  __shared__ __attribute__((aligned(16))) int lds_idx[4 * 32];
  __shared__ int lds_cnt[256];
  __shared__ double lds_obj[4];
  // the chunk's indices and distances, stored to memory after the last tile:
  // global stores under a lane condition inside the loop would make the
  // compiler wait for every load in flight (the prefetch would stall)
  __shared__ int lds_oidx[ASSIGN ? SMALLK_CH : 1];
  __shared__ float lds_omd[ASSIGN ? SMALLK_CH : 1];

  const int b = blockIdx.y;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int n = lane & 31, h = lane >> 5;
  X += (size_t)b * N * RC;
  idx += (size_t)b * N;
  const int KT = (K + 31) / 32;  // <= KTM (checked by the host)
  char* xt = xt_all + wave * SL::XT;
  int* widx = lds_idx + wave * 32;

  if constexpr (SUMS) {
    for (int k = tid; k < 256; k += ASSIGN_THREADS) lds_cnt[k] = 0;
    if constexpr (D < 32 * DTL)  // the padding dimensions of the last tile stay zero
      *reinterpret_cast<uint4*>(xt + D * 64 + lane * 16) = make_uint4(0, 0, 0, 0);
  }

  PipeOffsets<CPL, LOADS> o;
  pipe_offsets<CPL, LOADS>(o, tid, n, h);
  if constexpr (ASSIGN) {
    const u32x4* chat4 = reinterpret_cast<const u32x4*>(chat) + (size_t)b * Kp * RC;
    cinit += (size_t)b * Kp;
    min_dist += (size_t)b * N;
    const float s0 = pipe_issue_stage<CPL, LOADS>(chat4, cinit, 0, tid, o, buf0);
    lds_at<float>(buf0, o.n_store, 0) = s0;
    if constexpr (TWO) {
      if (Kp > L::TCS) {
        const float s1 = pipe_issue_stage<CPL, LOADS>(chat4, cinit, 1, tid, o, buf1);
        lds_at<float>(buf1, o.n_store, 0) = s1;
      }
    }
    __builtin_amdgcn_s_waitcnt(0);
  }
  __syncthreads();

  f32x16 S[KTM][DTL];
#pragma unroll
  for (int kt = 0; kt < KTM; ++kt)
#pragma unroll
    for (int dt = 0; dt < DTL; ++dt)
#pragma unroll
      for (int j = 0; j < 16; ++j) S[kt][dt][j] = 0.f;

  // Tiles t + 1 and t + 2 are in flight while tile t is worked on (one tile
  // ahead leaves the loop waiting for memory): three register sets in a ring,
  // the loop unrolled by three so that no set is copied (a copy would wait for
  // its loads).  A lane past N loads row N - 1 instead: the loads stay
  // unconditional (a branch around them would make every wait a full one),
  // its results are never stored and its one-hot column is zero.
  const int p0 = blockIdx.x * SMALLK_CH + wave * 32 + n;  // this lane's point in tile 0
  auto load = [&](int pt, uint4 (&v)[1][CPL], int& iv) {
    const int r = pt < N ? pt : N - 1;
#pragma unroll
    for (int c = 0; c < CPL; ++c) v[0][c] = X[(size_t)r * RC + h * CPL + c];
    if constexpr (MODE == SUMS_ONLY) iv = idx[r];
  };
  uint4 x0[1][CPL], x1[1][CPL], x2[1][CPL];
  int i0 = -1, i1 = -1, i2 = -1;
  double obj = 0.0;
  // tile t from xr / ir, with tile t + 2 started into xn / in_; false past the last tile
  auto step = [&](int t, const uint4 (&xr)[1][CPL], int ir, uint4 (&xn)[1][CPL], int& in_) {
    if (t >= SK_TILES || (int)blockIdx.x * SMALLK_CH + t * SK_TILE >= N) return false;  // uniform
    const int pt = p0 + t * SK_TILE;
    const bool ok = pt < N;
    // past the last tile, the last tile again (an L2 hit; a branch here would make waits full)
    load(pt + (t + 2 < SK_TILES ? 2 : SK_TILES - 1 - t) * SK_TILE, xn, in_);
    int i = ir;
    if constexpr (ASSIGN) {
      float ss = 0.f;
#pragma unroll
      for (int c = 0; c < CPL; ++c) ss = chunk_sumsq<DT>(xr[0][c], ss);
      ss += __shfl_xor(ss, 32);
      // Q >= |x|^2 / 2 with a relative margin of 2^-8 (far above fp32 rounding)
      const float Qp[1] = {__builtin_fmaf(0.5f * ss, 1.0f + 0x1p-8f, 1e-30f)};
      float best[1] = {-__builtin_inff()};
      uint32_t code[1] = {0};
      sk_stage<DT, CPL, LOADS, KTM < 4 ? 2 : 4>(xr, buf0, o, 0, Qp, best, code);
      if constexpr (TWO)
        if (Kp > L::TCS) sk_stage<DT, CPL, LOADS, 4>(xr, buf1, o, 4, Qp, best, code);
      float v = best[0];
      const uint32_t j = code[0] & 15u;
      i = (int)((code[0] >> 4) * 32 + 8 * (j >> 2) + 4 * h + (j & 3));
      const float vo = __shfl_xor(v, 32);
      const int io = __shfl_xor(i, 32);
      const bool take = (vo > v) || (vo == v && io < i);
      v = take ? vo : v;
      i = take ? io : i;
      // unassigned: a norm that is not finite, or no real centroid's score finite
      const bool asg = ss <= __FLT_MAX__ && v > -__FLT_MAX__;
      i = asg ? i : -1;
      if (h == 0) {
        const float md = __builtin_fmaxf(__builtin_fmaf(-2.f, v + Qp[0], ss), 0.f);
        lds_oidx[t * SK_TILE + wave * 32 + n] = i;
        lds_omd[t * SK_TILE + wave * 32 + n] = asg ? md : __builtin_nanf("");
        if (ok && asg) obj += (double)md;
      }
    }
    if constexpr (SUMS) sk_sums<DT, CPL, KTM>(xr, i, ok, xt, widx, lds_cnt, n, h, K, KT, S);
    return true;
  };
  load(p0, x0, i0);
  load(p0 + SK_TILE, x1, i1);
  for (int t = 0;; t += 3) {
    if (!step(t, x0, i0, x2, i2)) break;
    if (!step(t + 1, x1, i1, x0, i0)) break;
    if (!step(t + 2, x2, i2, x1, i1)) break;
  }

  const size_t blk = (size_t)b * gridDim.x + blockIdx.x;
  if constexpr (ASSIGN) {
#pragma unroll
    for (int msk = 1; msk < 64; msk <<= 1) obj += __shfl_xor(obj, msk);
    if (lane == 0) lds_obj[wave] = obj;
  }
  __syncthreads();
  if constexpr (ASSIGN) {
    if (tid == 0) objpart[blk] = ((lds_obj[0] + lds_obj[1]) + lds_obj[2]) + lds_obj[3];
    const int c0 = blockIdx.x * SMALLK_CH;
    const int np = N - c0 < SMALLK_CH ? N - c0 : SMALLK_CH;
    for (int k = tid; k < np; k += ASSIGN_THREADS) {
      idx[c0 + k] = lds_oidx[k];
      min_dist[c0 + k] = lds_omd[k];
    }
  }
  if constexpr (!SUMS) return;

  // the four waves' tiles, added in wave order; lane l of a wave holds rows
  // 8 q + 4 h + r of column n of each tile
  partial += blk * K * D;
  float4* wt = reinterpret_cast<float4*>(xt_all + wave * 4096);
  const float4* wr = reinterpret_cast<const float4*>(xt_all);
  const int q = tid >> 6;  // the read-back slot of this thread is (q, lane)
#pragma unroll
  for (int kt = 0; kt < KTM; ++kt) {
    if (kt < KT) {
#pragma unroll
      for (int dt = 0; dt < DTL; ++dt) {
#pragma unroll
        for (int qq = 0; qq < 4; ++qq)
          wt[qq * 64 + lane] = make_float4(S[kt][dt][4 * qq], S[kt][dt][4 * qq + 1],
                                           S[kt][dt][4 * qq + 2], S[kt][dt][4 * qq + 3]);
        __syncthreads();
        const float4 a = wr[q * 64 + lane], bb = wr[256 + q * 64 + lane],
                     c = wr[512 + q * 64 + lane], d = wr[768 + q * 64 + lane];
        const float v[4] = {((a.x + bb.x) + c.x) + d.x, ((a.y + bb.y) + c.y) + d.y,
                            ((a.z + bb.z) + c.z) + d.z, ((a.w + bb.w) + c.w) + d.w};
        const int dim = 32 * dt + n;
        if (dim < D) {
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int cl = 32 * kt + 8 * q + 4 * h + r;
            if (cl < K) partial[(size_t)cl * D + dim] = v[r];
          }
        }
        __syncthreads();
      }
    }
  }
  for (int k = tid; k < K; k += ASSIGN_THREADS) pcount[blk * K + k] = lds_cnt[k];
}

template <int DT, int CPL, int KTM>
hipError_t launch_smallk_k(const void* X, const Workspace& w, int64_t B, int64_t N, int64_t K,
                           int mode, int32_t* idx, float* min_dist, hipStream_t s) {
  const dim3 grid((unsigned)w.n_sk_chunks, (unsigned)B), block(ASSIGN_THREADS);
  const uint4* Xv = (const uint4*)X;
  const uint4* ch = (const uint4*)w.chat;
  if (mode == SUMS_ASSIGN) {
    assign_smallk_kernel<DT, CPL, KTM, SUMS_ASSIGN><<<grid, block, 0, s>>>(
        Xv, ch, w.cinit, (int)N, (int)K, (int)w.Kp, idx, min_dist, w.objpart, nullptr, nullptr);
  } else if (mode == SUMS_FUSED) {
    // more sum tiles beside the assignment would spill (fused_ok excludes them)
    if constexpr (KTM * SkLayout<CPL>::DTL <= 4)
      assign_smallk_kernel<DT, CPL, KTM, SUMS_FUSED><<<grid, block, 0, s>>>(
          Xv, ch, w.cinit, (int)N, (int)K, (int)w.Kp, idx, min_dist, w.objpart, w.partial,
          w.pcount);
    else
      return hipErrorInvalidValue;
  } else
    assign_smallk_kernel<DT, CPL, KTM, SUMS_ONLY><<<grid, block, 0, s>>>(
        Xv, nullptr, nullptr, (int)N, (int)K, 0, idx, nullptr, nullptr, w.partial, w.pcount);
  return hipGetLastError();
}

template <int DT, int CPL>
hipError_t launch_smallk_c(const void* X, const Workspace& w, int64_t B, int64_t N, int64_t K,
                           int mode, int32_t* idx, float* min_dist, hipStream_t s) {
  constexpr int DTL = SkLayout<CPL>::DTL;
  const int64_t kt = (K + 31) / 32;
  if (kt <= 2) return launch_smallk_k<DT, CPL, 2>(X, w, B, N, K, mode, idx, min_dist, s);
  if constexpr (DTL <= 2)
    if (kt <= 4) return launch_smallk_k<DT, CPL, 4>(X, w, B, N, K, mode, idx, min_dist, s);
  if constexpr (DTL == 1)
    if (kt <= 8) return launch_smallk_k<DT, CPL, 8>(X, w, B, N, K, mode, idx, min_dist, s);
  return hipErrorInvalidValue;
}

// One of the three SumsMode kernels; shapes with sums_ok.
template <int DT>
hipError_t launch_sums_dt(const void* X, const Workspace& w, int64_t B, int64_t N, int64_t D,
                          int64_t K, int mode, int32_t* idx, float* min_dist, hipStream_t s) {
  if (!sums_ok(DT, D, K) || (mode != SUMS_ONLY && w.Kp > 2 * ASSIGN_KPAD)) return hipErrorInvalidValue;
  switch (D / 16) {
    case 2: return launch_smallk_c<DT, 2>(X, w, B, N, K, mode, idx, min_dist, s);
    case 3: return launch_smallk_c<DT, 3>(X, w, B, N, K, mode, idx, min_dist, s);
    case 4: return launch_smallk_c<DT, 4>(X, w, B, N, K, mode, idx, min_dist, s);
    case 5: return launch_smallk_c<DT, 5>(X, w, B, N, K, mode, idx, min_dist, s);
    case 6: return launch_smallk_c<DT, 6>(X, w, B, N, K, mode, idx, min_dist, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace fkm
