// assign_tiled.hip -- the assignment step for wide rows (16-bit points with
// D > 256, a multiple of 32), where a point no longer fits in registers.
//
// The distance contraction is tiled like a GEMM.  A workgroup owns 256 points
// and up to TILED_CBG consecutive 256-centroid blocks; its eight waves split
// each 256 x 256 block 2 x 4, so a wave owns 128 points x 64 centroids: 4 x 2
// 32x32x16 MFMA tiles, 8 independent accumulators, and two waves share each
// SIMD (one wave of 4 x 4 tiles per SIMD left every LDS and barrier latency
// exposed).  Per 16-dimension step a wave reads 2 centroid and 4 point
// fragments from LDS for 8 MFMAs.
//
// Staging.  D streams through LDS in 32-dimension stages holding both
// operands and the block's scores.  Each stage goes from L2 straight into LDS
// (global_load_lds: lane l of a wave fills slot base + 16 l, so each lane
// fetches the chunk the swizzled layout puts there).  Four stage buffers let
// the loads run two to three stages ahead: a barrier without a memory fence
// (an explicit vmcnt wait for exactly the stage needed next, then s_barrier)
// keeps the later stages in flight across it.  The loads are issued by
// inline assembly, so the compiler adds no waits of its own for them; the
// buffers are separate LDS arrays and the stage loop is unrolled by four.
// The barrier sits in the middle of a stage: the second 16-dimension step's
// MFMAs run after it, beside the reads of the next stage's first fragments.
// (One barrier per two stages, with the loads one pair ahead instead of two
// to three stages, measured 3% slower.)
//
// Scores.  The accumulator of point p and centroid c starts at
// -|c^|^2/2 - Q_p, with Q_p a bound on the point's own |x_p|^2/2 (from a
// row-norm pass) plus a margin, so every score is negative and the packed-key
// epilogue applies: the lane's position j in the tile goes into the 4 low
// mantissa bits, a max3 tree picks the tile's best, and a strict compare on
// the masked value keeps the earliest tile (scores within 16 ulp count as
// ties and go to the lowest index).  The shift is per point, so that window
// is relative to each point's own norm and distance, whatever the norms of
// the other points in the workgroup; it costs 16 subtractions per tile and
// block, against 2 D / 16 MFMAs.  The two waves sharing a point range merge
// through LDS at the end, and the workgroup merges its result into a
// per-point 64-bit key with atomicMax: the masked score mapped to an
// order-preserving unsigned integer in the high half and the complemented
// index in the low half, so the maximum is the largest score and, among equal
// scores, the lowest index, whatever order the workgroups finish in.  Q_p
// depends only on the point's norm, so every workgroup uses the same Q_p for
// a point, and the decode pass recomputes it the same way.
//
// Blocks of D.  A block of centroids takes nds = D / 32 stages, padded to a
// multiple of four (the buffer rotation).  A padding stage reloads the block's
// last point stage and loads its centroid chunks from a zeroed scratch area,
// so every stage issues the same loads and runs the same code: its MFMAs add
// a finite x times zero, which is exactly zero.
//
// Block order is XCD-aware: workgroup ids go round-robin over the 8 XCDs, and
// each XCD walks super-tiles of 8 point blocks x all centroid groups (point
// block fastest), so the workgroups resident on an XCD share both operands
// through that XCD's L2.
#include "fkm_device.h"

namespace fkm {

namespace {

constexpr int TT = 512;                  // threads per workgroup (8 waves)
constexpr int BP = TILED_BP;             // points per workgroup
constexpr int BC = TILED_BC;             // centroids per block
constexpr int DC = 32;                   // dimensions per LDS stage
constexpr int CPS = DC * 2 / 16;         // 16-byte chunks of a row in one stage (4)
constexpr int XB = BP * CPS * 16;        // bytes of point chunks per stage
constexpr int CB = BC * CPS * 16;        // bytes of centroid chunks per stage
// + the block's scores, and a second copy that the upper four waves load so
// that every wave issues the same number of loads
constexpr int STAGE = XB + CB + 2 * BC * 4;
constexpr int LX = BP * CPS / TT;        // point chunks per thread per stage
constexpr int LC = BC * CPS / TT;        // centroid chunks per thread per stage
constexpr int LOADS = LX + LC + 1;       // loads per thread per stage (+ one score)
constexpr int RSTEP = TT / CPS;          // rows between a thread's loads (128)
static_assert(BP == 256 && BC == 256, "2 x 4 waves of 128 x 64");
static_assert(2 * LOADS <= 63, "vmcnt counts at most 63 loads");
static_assert(CB <= TILED_ZERO_BYTES, "a padding stage's centroid chunks fit the zero area");

// L2 -> LDS copies of 16 (or 4) bytes per lane into the wave's slots at
// `lds` (lane l at lds + 16 l, or + 4 l), issued by inline assembly: with the
// compiler's builtin for them in flight, its own waits around the fragment
// reads became full drains (vmcnt(0), lgkmcnt(0)) that also waited for the
// stages loading two and three ahead.  Outside the compiler's view the loads
// count only in the hardware's in-order vmcnt, which the explicit waits
// before each barrier govern; M0 (the LDS base) is set in the same statement,
// one wait state before the load reads it, and used by nothing else in this
// kernel.
__device__ __forceinline__ void dma16(const void* src, char* lds) {
  const uint32_t base = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)(lds);
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
               :
               : "v"(src), "s"(base)
               : "memory");
}
__device__ __forceinline__ void dma4(const void* src, char* lds) {
  const uint32_t base = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)(lds);
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dword %0, off"
               :
               : "v"(src), "s"(base)
               : "memory");
}

// Wait until at most n of this wave's loads are in flight and its LDS
// accesses are done, then a barrier without a memory fence, so the loads
// started into other buffers stay in flight across it.
template <int n>
__device__ __forceinline__ void wait_loads_and_sync() {
  __builtin_amdgcn_s_waitcnt((n & 0xF) | ((n >> 4) << 14) | (7 << 4));
  asm volatile("s_barrier" ::: "memory");
}

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

// Q_p >= |x_p|^2 / 2 with a relative margin of 2^-8; the same bits wherever
// it is computed from the same norm.
__device__ __forceinline__ float point_q(float xn) {
  return __builtin_fmaf(0.5f * xn, 1.0f + 0x1p-8f, 1e-30f);
}

template <typename T>
__device__ __forceinline__ T& lds_at(char* base, int off) {
  return *reinterpret_cast<T*>(base + off);
}

struct TiledCtx {
  const char* X;       // the workgroup's first point row
  const char* chat;    // this instance's rounded centroids
  const float* cinit;  // this instance's -|c^|^2/2
  const char* zero;    // CB zeroed bytes: the centroid chunks of a padding stage
  uint32_t xoff;       // lane byte offset of its first point chunk (row clamped to the last point)
  uint32_t coff;       // lane byte offset of its first centroid chunk
  uint32_t rowsstep;   // bytes of RSTEP rows
  int last;            // last valid row of the point block
  int nds;             // stages of 32 dimensions per block (D / 32)
  int ndsv;            // stages per block, padded to a multiple of 4
  int cb0, RC, tid, S, loff0, loff1, wp, wc;
};

// Stage s = (block s / ndsv, dimensions 32 (s % ndsv) ..): start its loads into buf.
// Load u of a thread covers slot tid + 512 u: row tid / 4 + 128 u, chunk
// (tid % 4) ^ swz(row) (swz has period 16, so the chunk order repeats).
__device__ __forceinline__ void tiled_issue(const TiledCtx& c, int s, char* buf) {
  const int g = s / c.ndsv, dv = s % c.ndsv, ds = min(dv, c.nds - 1);
  const bool pad = dv >= c.nds;
  const int wave = __builtin_amdgcn_readfirstlane(c.tid >> 6);
  const char* xb = c.X + ds * CPS * 16;
#pragma unroll
  for (int u = 0; u < LX; ++u) {
    // rows past the last point reload the last point (their results are dropped)
    const uint32_t off = (c.tid >> 2) + RSTEP * u <= c.last
                             ? c.xoff + u * c.rowsstep
                             : (uint32_t)((c.last * c.RC + ((c.tid & 3) ^ swz(c.tid >> 2))) * 16);
    dma16(xb + off, buf + (u * TT + wave * 64) * 16);
  }
  const int krow = (c.cb0 + g) * BC;
  const char* cbp = c.chat + ((size_t)krow * c.RC + ds * CPS) * 16;
#pragma unroll
  for (int u = 0; u < LC; ++u) {
    const char* src = pad ? c.zero + (u * TT + c.tid) * 16 : cbp + c.coff + u * c.rowsstep;
    dma16(src, buf + XB + (u * TT + wave * 64) * 16);
  }
  // the block's scores ride with every stage, so every stage issues LOADS loads
  // (waves 4 .. 7 load a second copy, never read)
  dma4(c.cinit + krow + (c.tid & (BC - 1)), buf + XB + CB + wave * 256);
}

// Fragments of one 16-dimension step: 4 centroid tiles and 4 point tiles.
constexpr int TCW = 2;  // 32-centroid tiles per wave
struct TiledFrag {
  uint4 a[TCW], b[4];
};

__device__ __forceinline__ void tiled_read(TiledFrag& f, char* buf, int lo, int wp, int wc) {
#pragma unroll
  for (int tc = 0; tc < TCW; ++tc)
    f.a[tc] = lds_at<uint4>(buf, XB + (wc * 32 * TCW + tc * 32) * 64 + lo);
#pragma unroll
  for (int tp = 0; tp < 4; ++tp) f.b[tp] = lds_at<uint4>(buf, (wp * 128 + tp * 32) * 64 + lo);
}

template <int DT>
__device__ __forceinline__ void tiled_mfma(f32x16 (&acc)[4][TCW], const TiledFrag& f) {
#pragma unroll
  for (int tp = 0; tp < 4; ++tp)
#pragma unroll
    for (int tc = 0; tc < TCW; ++tc) acc[tp][tc] = mfma32_chunk<DT>(f.a[tc], f.b[tp], acc[tp][tc]);
}

// A new block: the accumulator of point tile tp starts at its centroid's
// -|c^|^2/2 minus the lane's point's Q_p.
__device__ __forceinline__ void tiled_init(f32x16 (&acc)[4][TCW], char* buf, int wc, int h,
                                           const float (&Qp)[4]) {
#pragma unroll
  for (int tc = 0; tc < TCW; ++tc) {
    f32x16 cin;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const f32x4 v =
          lds_at<f32x4>(buf, XB + CB + (wc * 32 * TCW + tc * 32 + 8 * q + 4 * h) * 4);
      cin[4 * q + 0] = v[0];
      cin[4 * q + 1] = v[1];
      cin[4 * q + 2] = v[2];
      cin[4 * q + 3] = v[3];
    }
#pragma unroll
    for (int tp = 0; tp < 4; ++tp)
#pragma unroll
      for (int j = 0; j < 16; ++j) acc[tp][tc][j] = cin[j] - Qp[tp];
  }
}

// Stage s in `cur` (its first-step fragments already in f0): read the second
// step's, run the first step's MFMAs, wait for stage s + 1 and sync, start
// stage s + 3 into `ahead` (the buffer of stage s - 1, which every wave has
// now finished), read stage s + 1's first-step fragments from `nxt`, run the
// second step's MFMAs.  TAIL: stages past the end may follow.
template <int DT, bool TAIL>
__device__ __forceinline__ void tiled_stage(const TiledCtx& c, int s, char* cur, char* nxt,
                                            char* ahead, f32x16 (&acc)[4][TCW], TiledFrag& f0,
                                            TiledFrag& f1) {
  tiled_read(f1, cur, c.loff1, c.wp, c.wc);
  tiled_mfma<DT>(acc, f0);
  if (!TAIL || s + 2 < c.S) wait_loads_and_sync<LOADS>();
  else wait_loads_and_sync<0>();
  if (!TAIL || s + 3 < c.S) tiled_issue(c, s + 3, ahead);
  if (!TAIL || s + 1 < c.S) tiled_read(f0, nxt, c.loff0, c.wp, c.wc);
  tiled_mfma<DT>(acc, f1);
}

// Four stages; stage s0 is in buffer 0.
template <int DT, bool TAIL>
__device__ __forceinline__ void tiled_quad(const TiledCtx& c, int s0, char* b0, char* b1, char* b2,
                                           char* b3, f32x16 (&acc)[4][TCW], TiledFrag& f0,
                                           TiledFrag& f1) {
  tiled_stage<DT, TAIL>(c, s0, b0, b1, b3, acc, f0, f1);
  tiled_stage<DT, TAIL>(c, s0 + 1, b1, b2, b0, acc, f0, f1);
  tiled_stage<DT, TAIL>(c, s0 + 2, b2, b3, b1, acc, f0, f1);
  tiled_stage<DT, TAIL>(c, s0 + 3, b3, b0, b2, acc, f0, f1);
}

// The block is complete: packed-key arg-max of each tile into the running
// (best, code) of each point tile; tiles are visited in increasing index order.
__device__ __forceinline__ void tiled_epilogue(const f32x16 (&acc)[4][TCW], float (&best)[4],
                                               uint32_t (&code)[4], uint32_t tile0) {
#pragma unroll
  for (int tp = 0; tp < 4; ++tp)
#pragma unroll
    for (int tc = 0; tc < TCW; ++tc) {
      float k[16];
#pragma unroll
      for (int j = 0; j < 16; ++j)
        k[j] = __uint_as_float((__float_as_uint(acc[tp][tc][j]) & ~15u) | (uint32_t)j);
      const float t0 = __builtin_fmaxf(__builtin_fmaxf(k[0], k[1]), k[2]);
      const float t1 = __builtin_fmaxf(__builtin_fmaxf(k[3], k[4]), k[5]);
      const float t2 = __builtin_fmaxf(__builtin_fmaxf(k[6], k[7]), k[8]);
      const float t3 = __builtin_fmaxf(__builtin_fmaxf(k[9], k[10]), k[11]);
      const float t4 = __builtin_fmaxf(__builtin_fmaxf(k[12], k[13]), k[14]);
      const float u0 = __builtin_fmaxf(__builtin_fmaxf(t0, t1), t2);
      const float u1 = __builtin_fmaxf(__builtin_fmaxf(t3, t4), k[15]);
      const uint32_t mb = __float_as_uint(__builtin_fmaxf(u0, u1));
      const float mm = __uint_as_float(mb & ~15u);
      const bool gt = mm > best[tp];
      best[tp] = gt ? mm : best[tp];
      code[tp] = gt ? ((mb & 15u) | ((tile0 + tc) << 4)) : code[tp];
    }
}

}  // namespace

template <int DT>
__global__ __launch_bounds__(TT, 1) void assign_tiled_kernel(
    const uint4* __restrict__ X, const uint4* __restrict__ chat, const float* __restrict__ cinit,
    const float* __restrict__ xnorm, const uint4* __restrict__ zero, int N, int D, int Kp, int npb,
    int ncbg, uint64_t* __restrict__ keys) {
  __shared__ __attribute__((aligned(16))) char buf0[STAGE];
  __shared__ __attribute__((aligned(16))) char buf1[STAGE];
  __shared__ __attribute__((aligned(16))) char buf2[STAGE];
  __shared__ __attribute__((aligned(16))) char buf3[STAGE];

  const int b = blockIdx.y;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int n = lane & 31, h = lane >> 5;
  const int wp = wave & 1, wc = wave >> 1;  // point half, centroid quarter
  const int xcd = blockIdx.x & 7, j = blockIdx.x >> 3;
  const int sup = j / (8 * ncbg), cbg = (j / 8) % ncbg;
  const int pb = (sup * 8 + xcd) * 8 + (j & 7);
  if (pb >= npb) return;
  const int p0 = pb * BP;
  const int RC = D / 8;  // 16-byte chunks per row
  const int nds = D / DC;
  const int ndsv = (nds + 3) / 4 * 4;
  const int cb0 = cbg * TILED_CBG;
  const int ncbw = min(TILED_CBG, Kp / BC - cb0);  // centroid blocks of this workgroup

  TiledCtx c;
  c.X = reinterpret_cast<const char*>(X + ((size_t)b * N + p0) * RC);
  c.chat = reinterpret_cast<const char*>(chat + (size_t)b * Kp * RC);
  c.cinit = cinit + (size_t)b * Kp;
  c.zero = reinterpret_cast<const char*>(zero);
  c.last = min(BP, N - p0) - 1;
  c.xoff = (uint32_t)((min(tid >> 2, c.last) * RC + ((tid & 3) ^ swz(tid >> 2))) * 16);
  c.coff = (uint32_t)(((tid >> 2) * RC + ((tid & 3) ^ swz(tid >> 2))) * 16);
  c.rowsstep = (uint32_t)(RSTEP * RC * 16);
  c.nds = nds;
  c.ndsv = ndsv;
  c.cb0 = cb0;
  c.RC = RC;
  c.tid = tid;
  c.S = ncbw * ndsv;
  // fragment reads: lane 32 h + n takes row (tile base + n), chunk 2 ks + h
  c.loff0 = n * 64 + ((0 + h) ^ swz(n)) * 16;
  c.loff1 = n * 64 + ((2 + h) ^ swz(n)) * 16;
  c.wp = wp;
  c.wc = wc;

  // Q_p of the lane's four points (column n of point tile tp)
  float Qp[4];
#pragma unroll
  for (int tp = 0; tp < 4; ++tp) {
    const int r = wp * 128 + tp * 32 + n;
    Qp[tp] = point_q(r <= c.last ? xnorm[(size_t)b * N + p0 + r] : 0.f);
  }

  // stages 0 .. 2 in flight before the loop; stage 0 complete
  const int S = c.S;
  tiled_issue(c, 0, buf0);
  if (1 < S) tiled_issue(c, 1, buf1);
  if (2 < S) tiled_issue(c, 2, buf2);
  if (2 < S) wait_loads_and_sync<2 * LOADS>();
  else if (1 < S) wait_loads_and_sync<LOADS>();
  else wait_loads_and_sync<0>();

  f32x16 acc[4][TCW];
  float best[4];
  uint32_t code[4];
#pragma unroll
  for (int tp = 0; tp < 4; ++tp) {
    best[tp] = -__builtin_inff();
    code[tp] = 0;
  }
  TiledFrag f0, f1;
  tiled_read(f0, buf0, c.loff0, wp, wc);
  const int nq = ndsv / 4;  // every block starts in buffer 0
  for (int g = 0; g < ncbw; ++g) {
    tiled_init(acc, buf0, wc, h, Qp);
    const int s0 = g * ndsv;
    const int full = g == ncbw - 1 ? nq - 1 : nq;  // quads with no stage past the end
    for (int q = 0; q < full; ++q)
      tiled_quad<DT, false>(c, s0 + 4 * q, buf0, buf1, buf2, buf3, acc, f0, f1);
    if (full < nq) tiled_quad<DT, true>(c, s0 + 4 * full, buf0, buf1, buf2, buf3, acc, f0, f1);
    tiled_epilogue(acc, best, code, (uint32_t)((cb0 + g) * (BC / 32) + wc * TCW));
  }

  // merge the two row halves of each point, then the four centroid quarters
  // of the workgroup (waves wc = 1 .. 3 hand theirs over through LDS; wave
  // wc = 0 takes them in quarter order)
  float* mv = reinterpret_cast<float*>(buf0);
  int* mi = reinterpret_cast<int*>(buf0 + 4 * BP * 4);
  float v[4];
  int ix[4];
#pragma unroll
  for (int tp = 0; tp < 4; ++tp) {
    const uint32_t jj = code[tp] & 15u;
    const int i = (int)((code[tp] >> 4) * 32 + 8 * (jj >> 2) + 4 * h + (jj & 3));
    const float vo = __shfl_xor(best[tp], 32);
    const int io = __shfl_xor(i, 32);
    const bool take = (vo > best[tp]) || (vo == best[tp] && io < i);
    v[tp] = take ? vo : best[tp];
    ix[tp] = take ? io : i;
  }
  if (wc != 0 && h == 0) {
#pragma unroll
    for (int tp = 0; tp < 4; ++tp) {
      mv[wc * BP + wp * 128 + tp * 32 + n] = v[tp];
      mi[wc * BP + wp * 128 + tp * 32 + n] = ix[tp];
    }
  }
  __syncthreads();
  if (wc == 0 && h == 0) {
#pragma unroll
    for (int tp = 0; tp < 4; ++tp) {
      const int r = wp * 128 + tp * 32 + n;
      float vv = v[tp];
      int ii = ix[tp];
#pragma unroll
      for (int q = 1; q < 4; ++q) {
        const float vo = mv[q * BP + r];
        const int io = mi[q * BP + r];
        const bool take = (vo > vv) || (vo == vv && io < ii);
        vv = take ? vo : vv;
        ii = take ? io : ii;
      }
      if (r <= c.last) {
        const uint64_t key = ((uint64_t)ordered(vv) << 32) | (uint64_t)(0xffffffffu - (uint32_t)ii);
        atomicMax((unsigned long long*)&keys[(size_t)b * N + p0 + r], (unsigned long long)key);
      }
    }
  }
}

// Squared norms of the points, one wave per row: lane-strided, then a fixed
// xor butterfly (the same bits on every call).
template <int DT>
__global__ __launch_bounds__(256) void row_norm_kernel(const uint4* __restrict__ X, int64_t rows,
                                                       int RC, float* __restrict__ xnorm) {
  const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (r >= rows) return;
  const uint4* row = X + r * RC;
  float ss = 0.f;
  for (int cc = lane; cc < RC; cc += 64) ss = chunk_sumsq<DT>(row[cc], ss);
#pragma unroll
  for (int m = 1; m < 64; m <<= 1) ss += __shfl_xor(ss, m);
  if (lane == 0) xnorm[r] = ss;
}

__global__ __launch_bounds__(256) void fill_keys_kernel(uint64_t* __restrict__ keys, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n) keys[i] = 0;
}

// idx, min_dist and per-block objective partials from the keys; each point's
// Q_p is recomputed from the same norm.
__global__ __launch_bounds__(256) void decode_keys_kernel(const uint64_t* __restrict__ keys,
                                                          const float* __restrict__ xnorm, int N,
                                                          int32_t* __restrict__ idx,
                                                          float* __restrict__ min_dist,
                                                          double* __restrict__ objpart) {
  __shared__ double s[256];
  const int b = blockIdx.y;
  const int t = threadIdx.x;
  const int i = blockIdx.x * 256 + t;
  const float xn = i < N ? xnorm[(size_t)b * N + i] : 0.f;
  double md = 0.0;
  if (i < N) {
    const uint64_t key = keys[(size_t)b * N + i];
    const float v = unordered((uint32_t)(key >> 32));
    // unassigned: a norm that is not finite, or no real centroid's score finite
    const bool asg = xn <= __FLT_MAX__ && v > -__FLT_MAX__;
    const float d = __builtin_fmaxf(__builtin_fmaf(-2.f, v + point_q(xn), xn), 0.f);
    idx[(size_t)b * N + i] = asg ? (int32_t)(0xffffffffu - (uint32_t)key) : -1;
    min_dist[(size_t)b * N + i] = asg ? d : __builtin_nanf("");
    md = asg ? d : 0.0;
  }
  s[t] = md;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (t < w) s[t] += s[t + w];
    __syncthreads();
  }
  if (t == 0) objpart[(size_t)b * gridDim.x + blockIdx.x] = s[0];
}

hipError_t launch_assign_tiled(const void* X, int dt, const Workspace& w, int64_t B, int64_t N,
                               int64_t D, int32_t* idx, float* min_dist, hipStream_t s) {
  if (D % DC != 0 || w.Kp % BC != 0) return hipErrorInvalidValue;
  const int64_t nk = B * N;
  // the keys, then TILED_ZERO_BYTES of zeros for padding stages (16-byte aligned)
  const int64_t nz = (nk + 1) & ~int64_t(1);
  const int64_t nfill = nz + TILED_ZERO_BYTES / 8;
  fill_keys_kernel<<<dim3((unsigned)((nfill + 255) / 256)), 256, 0, s>>>(w.keys, nfill);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int RC = (int)(D / 8);
  if (dt == DT_BF16)
    row_norm_kernel<DT_BF16><<<dim3((unsigned)((nk + 3) / 4)), 256, 0, s>>>((const uint4*)X, nk, RC,
                                                                          w.xnorm);
  else
    row_norm_kernel<DT_F16><<<dim3((unsigned)((nk + 3) / 4)), 256, 0, s>>>((const uint4*)X, nk, RC,
                                                                         w.xnorm);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  const int npb = (int)((N + BP - 1) / BP);
  const int ncb = (int)(w.Kp / BC);
  const int ncbg = (ncb + TILED_CBG - 1) / TILED_CBG;
  const int npb64 = (npb + 63) / 64 * 64;  // whole super-tiles on every XCD
  const dim3 grid((unsigned)(npb64 * ncbg), (unsigned)B);
  if (dt == DT_BF16)
    assign_tiled_kernel<DT_BF16><<<grid, TT, 0, s>>>((const uint4*)X, (const uint4*)w.chat,
                                                      w.cinit, w.xnorm, (const uint4*)(w.keys + nz),
                                                      (int)N, (int)D, (int)w.Kp, npb, ncbg, w.keys);
  else
    assign_tiled_kernel<DT_F16><<<grid, TT, 0, s>>>((const uint4*)X, (const uint4*)w.chat,
                                                     w.cinit, w.xnorm, (const uint4*)(w.keys + nz),
                                                     (int)N, (int)D, (int)w.Kp, npb, ncbg, w.keys);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  decode_keys_kernel<<<dim3((unsigned)w.n_assign_blocks, (unsigned)B), 256, 0, s>>>(
      w.keys, w.xnorm, (int)N, idx, min_dist, w.objpart);
  return hipGetLastError();
}

}  // namespace fkm
