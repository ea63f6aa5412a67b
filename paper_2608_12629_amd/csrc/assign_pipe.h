// assign_pipe.h -- the software-pipelined resident-X assignment kernel for
// bf16/fp16 points (D <= 256) and its launcher, instantiated once per storage
// type in assign_pipe_bf16.hip and assign_pipe_f16.hip.
#pragma once

#include "fkm_device.h"

namespace fkm {

// ---------------------------------------------------------------------------
// Resident-X assignment on 32x32x16 bf16/fp16 MFMA tiles, software-pipelined.
//
// Tile layout: 32 centroids (A rows) x 32 points (B columns) per instruction.
// Lane l = 32 h + n supplies point column n and centroid row n for the
// k-slice h (each lane group holds one contiguous half of the D dimensions)
// and receives accumulator rows 8 q + 4 h + r (q, r = 0..3) of column n.
// Each wave keeps NSUB 32-point column tiles in registers for the whole
// kernel; centroids stream through LDS in stages of TCS rows (four tiles, or
// two for 512-byte rows, so that two stage buffers of two workgroups fit).
//
// Staging.  Each stage goes from L2 straight into LDS (global_load_lds, 16
// bytes per lane, no registers, no LDS store instructions): lane l of a wave
// fills LDS slot base + 16 l, so each lane fetches the centroid chunk that the
// swizzled layout puts in its slot.  The two stage buffers are separate LDS
// arrays: the compiler then sees that a load in flight into one buffer cannot
// alias the reads of the other and does not wait for it before reading.
//
// Pipelining.  On this GPU the matrix pipe and the vector ALU overlap only
// within one wave's instruction stream (a wave that only issues vector
// instructions does not run beside another wave's MFMAs).  So the MFMAs of
// tile t and the epilogue of tile t-1 are written into the same basic block,
// on two accumulator sets, for the scheduler to interleave; NSUB independent
// accumulation chains keep the matrix pipe fed, and each MFMA is followed by
// a few vector instructions and one LDS read of a later A operand.
//
// Epilogue.  The accumulator starts at -|c^|^2/2 - Q, with Q a bound on
// |x|^2/2 over the workgroup's points plus a margin, so every score
// s' = <x, c^> - |c^|^2/2 - Q is strictly negative and orders the centroids
// like the distance does.  The lane's position j = 4 q + r is written into the
// 4 low mantissa bits of each score (one and-or), an integer min3 tree over
// the keys picks the tile's best (for negative floats the larger value has
// the smaller bit pattern, and on equal upper bits the lowest position wins),
// and a strict compare on the masked value keeps the earliest tile.  Scores within 16 ulp of each other
// therefore count as ties and go to the lowest index; nothing else changes.
// Since |s'| is up to about Q, that window (and the error of min_dist) is
// relative to the workgroup's largest norm; a workgroup whose points' norms
// spread widely subtracts each point's own bound instead (below).
// Padding rows score -FLT_MAX (or -inf once shifted); a NaN key, of either
// sign, reads as an integer above every finite negative key and never wins.
// Non-finite values: a centroid with a NaN or infinite coordinate scores NaN
// or -inf against every point and never wins; a point whose squared norm is
// not finite, or whose best score is not above -FLT_MAX (no real centroid
// scored finitely), is left unassigned (idx -1, min_dist NaN, no objective
// term), and such points do not enter the workgroup's shift.
typedef __attribute__((address_space(1))) void global_void;
typedef __attribute__((address_space(3))) void lds_void;

// One 16-byte-per-lane load from global memory straight into LDS (lane l
// writes LDS byte lds + 16 l), issued as assembly: with the compiler's
// builtin for it in flight, the compiler's own waits before every LDS read
// became full drains (lgkmcnt(0), even vmcnt(0)), although no read here
// touches the buffer being filled.  Outside its view the loads count only in
// the hardware's in-order vmcnt; the stage ends wait for them explicitly
// (s_waitcnt vmcnt(0) and a barrier) before any read of that buffer, and the
// compiler's waits for its own loads stay correct because loads complete in
// issue order.  M0 (the LDS base) is set here, one wait state before the load
// reads it (the hazard the compiler covers with an s_nop for its own LDS DMA);
// nothing else in these kernels uses it.
__device__ __forceinline__ void lds_dma16(const void* src, void* lds) {
  const uint32_t base =
      (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)(lds);
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
               :
               : "v"(src), "s"(base)
               : "memory");
}

// Per-lane offsets, fixed for the whole kernel.
template <int CPL, int LOADS>
struct PipeOffsets {
  int src[LOADS];    // chunk of a stage that lands in LDS slot tid + u * 256
  int a[CPL];        // byte offset of chunk h * CPL + c of centroid row n of tile 0
  int n_store;       // byte offset of the score slot written by this thread
  int n_read;        // byte offset of the first score read by this lane (rows 4 h .. 4 h + 3)
};

// Stage = TCS centroid rows of RC 16-byte chunks, each at a power-of-two
// stride of RCP >= RC slots and XOR-swizzled within it, then TCS scores.
template <int CPL>
struct PipeLayout {
  static constexpr int TCS = CPL <= 8 ? 128 : 64, RC = 2 * CPL, TILES = TCS / 32;
  static constexpr int RCP = pow2_at_least(RC);
  static constexpr int SWZ = RCP < 16 ? RCP - 1 : 15;
  static constexpr int CHUNKS = TCS * RCP * 16;         // bytes of centroid slots
  static constexpr int STAGE = CHUNKS + TCS * 4;         // bytes per stage buffer
  static constexpr int TILE = 32 * RCP * 16;             // bytes per tile of slots
};

template <int CPL, int LOADS>
__device__ __forceinline__ void pipe_offsets(PipeOffsets<CPL, LOADS>& o, int tid, int n, int h) {
  using L = PipeLayout<CPL>;
#pragma unroll
  for (int u = 0; u < LOADS; ++u) {  // slot s holds row s / RCP, chunk (s % RCP) ^ (row & SWZ)
    const int sl = tid + u * ASSIGN_THREADS;
    const int r = sl / L::RCP, c = (sl % L::RCP) ^ (r & L::SWZ);
    // a padding slot (c >= RC) is never read: it loads the row's first chunk,
    // so every lane loads and the stage code has no branch
    o.src[u] = r * L::RC + (c < L::RC ? c : 0);
  }
#pragma unroll
  for (int c = 0; c < CPL; ++c) o.a[c] = (n * L::RCP + ((h * CPL + c) ^ (n & L::SWZ))) * 16;
  o.n_store = L::CHUNKS + (tid & (L::TCS - 1)) * 4;
  o.n_read = L::CHUNKS + 16 * h;
}

// LDS accesses at a per-lane offset plus a compile-time byte offset.
template <typename T>
__device__ __forceinline__ T& lds_at(char* base, int lane_off, int imm) {
  return *reinterpret_cast<T*>(base + lane_off + imm);
}

// Start stage `st` on its way into `buf` (complete after the wave's next
// vmcnt(0) wait and a barrier).
template <int CPL, int LOADS>
__device__ __forceinline__ void pipe_issue_dma(const u32x4* __restrict__ chat, int st, int tid,
                                               const PipeOffsets<CPL, LOADS>& o, char* buf) {
  using L = PipeLayout<CPL>;
  const u32x4* src = chat + (size_t)st * L::TCS * L::RC;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
#pragma unroll
  for (int u = 0; u < LOADS; ++u) lds_dma16(src + o.src[u], buf + (u * ASSIGN_THREADS + wave * 64) * 16);
}

// This thread's score slot of stage `st`.
template <int CPL>
__device__ __forceinline__ float pipe_score(const float* __restrict__ cinit, int st, int tid) {
  using L = PipeLayout<CPL>;
  return cinit[st * L::TCS + (tid & (L::TCS - 1))];
}

// Both: the stage's loads, then this thread's score for it.
template <int CPL, int LOADS>
__device__ __forceinline__ float pipe_issue_stage(const u32x4* __restrict__ chat,
                                                  const float* __restrict__ cinit, int st, int tid,
                                                  const PipeOffsets<CPL, LOADS>& o, char* buf) {
  pipe_issue_dma<CPL, LOADS>(chat, st, tid, o, buf);
  return pipe_score<CPL>(cinit, st, tid);
}

// Rows row0 .. row0 + TCS - 1 of X (rows past N - 1 repeat row N - 1) into
// `buf` in the stage layout: the same slots, swizzle and per-lane offsets as
// a centroid stage, so each load instruction of a wave fetches whole
// consecutive rows (coalesced) and a lane's fragments are read back with the
// stage's offsets.  Complete after the wave's next vmcnt(0) wait and a barrier.
template <int CPL, int LOADS>
__device__ __forceinline__ void pipe_issue_rows(const uint4* __restrict__ X, int row0, int N, int tid,
                                                char* buf) {
  using L = PipeLayout<CPL>;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
#pragma unroll
  for (int u = 0; u < LOADS; ++u) {
    const int sl = tid + u * ASSIGN_THREADS;
    const int r = sl / L::RCP, c = (sl % L::RCP) ^ (r & L::SWZ);
    const int row = min(row0 + r, N - 1);
    lds_dma16(X + (size_t)row * L::RC + (c < L::RC ? c : 0), buf + (u * ASSIGN_THREADS + wave * 64) * 16);
  }
}

// The MFMAs of one 32-centroid tile into acc; each chain starts from the scores' init.
template <int DT, int TILE, int CPL, int NSUB, int LOADS>
__device__ __forceinline__ void pipe_mfma_tile(f32x16 (&acc)[NSUB], const uint4 (&xr)[NSUB][CPL],
                                               char* buf, const PipeOffsets<CPL, LOADS>& o) {
  using L = PipeLayout<CPL>;
  f32x16 cin;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const f32x4 v = lds_at<f32x4>(buf, o.n_read, (TILE * 32 + 8 * q) * 4);
    cin[4 * q + 0] = v[0];
    cin[4 * q + 1] = v[1];
    cin[4 * q + 2] = v[2];
    cin[4 * q + 3] = v[3];
  }
#pragma unroll
  for (int c = 0; c < CPL; ++c) {
    const uint4 a = lds_at<uint4>(buf, o.a[c], TILE * L::TILE);
#pragma unroll
    for (int p = 0; p < NSUB; ++p) acc[p] = mfma32_chunk<DT>(a, xr[p][c], c == 0 ? cin : acc[p]);
  }
}

// Packed-key arg-max of one tile into the running (best, code) of each column
// tile.  PPQ: the scores are shifted here, by each point's own Qp.  Every
// score is negative: the shift exceeds |x|^2 / 2 by a margin far above the
// rounding, and padding rows sit at -FLT_MAX (or -inf once shifted).  For
// negative floats the larger value has the smaller bit pattern read as a
// signed integer, so the arg-max is an integer minimum over the keys (16
// distinct keys, the position in the low 4 bits: the lower position wins a
// tie of the masked scores).  A key made from -inf is a negative NaN; read as
// an integer it is larger than every finite key, so it never beats a real
// score.  The integer tree needs none of the NaN quieting a float maximum
// takes.
template <int NSUB, bool PPQ>
__device__ __forceinline__ void pipe_epilogue(const f32x16 (&acc)[NSUB], uint32_t tcode,
                                              float (&best)[NSUB], uint32_t (&code)[NSUB],
                                              const float (&Qp)[NSUB]) {
#pragma unroll
  for (int p = 0; p < NSUB; ++p) {
    int k[16];
#pragma unroll
    for (int j = 0; j < 16; ++j)
      k[j] = (int)((__float_as_uint(PPQ ? acc[p][j] - Qp[p] : acc[p][j]) & ~15u) | (uint32_t)j);
    const int t0 = min(min(k[0], k[1]), k[2]);
    const int t1 = min(min(k[3], k[4]), k[5]);
    const int t2 = min(min(k[6], k[7]), k[8]);
    const int t3 = min(min(k[9], k[10]), k[11]);
    const int t4 = min(min(k[12], k[13]), k[14]);
    const int u0 = min(min(t0, t1), t2);
    const int u1 = min(min(t3, t4), k[15]);
    const uint32_t mb = (uint32_t)min(u0, u1);
    const float mm = __uint_as_float(mb & ~15u);
    const bool gt = mm > best[p];
    best[p] = gt ? mm : best[p];
    code[p] = gt ? ((mb & 15u) | tcode) : code[p];
  }
}

// One stage in `cur`: start the next stage into `nxt`, run the stage's tiles
// (tile i on one accumulator set beside the epilogue of tile i-1 on the
// other), store the next stage's scores, then wait for the loads and sync.
// next = min(st + 1, nst - 1).  `carry` holds this thread's score of stage
// `next`, fetched one stage earlier: a score fetched in this stage would
// make the compiler wait for it before the store, and that wait (a vmcnt
// count) would wait for the stage loads issued before it as well.  The
// score of the stage after `next` is fetched here instead; the wait at the
// stage's end covers it.
template <int DT, int CPL, int NSUB, int LOADS, bool PPQ>
__device__ __forceinline__ void pipe_stage(int st, int next, int nst, float& carry,
                                           f32x16 (&accA)[NSUB], f32x16 (&accB)[NSUB],
                                           const uint4 (&xr)[NSUB][CPL], char* cur, char* nxt,
                                           const PipeOffsets<CPL, LOADS>& o, const u32x4* chat,
                                           const float* cinit, float Q,
                                           const float (&Qp)[NSUB], int tid,
                                           uint32_t& prev_code, float (&best)[NSUB],
                                           uint32_t (&code)[NSUB]) {
  using L = PipeLayout<CPL>;
  pipe_issue_dma<CPL, LOADS>(chat, next, tid, o, nxt);
  const float nn = carry;
  carry = pipe_score<CPL>(cinit, next + 1 < nst ? next + 1 : nst - 1, tid);
  // issue the prefetch first: left to the scheduler it drifts into the middle
  // of the stage and the wait at the end stalls on it
  __builtin_amdgcn_sched_barrier(0);
  const uint32_t tb = (uint32_t)(L::TILES * st);
  pipe_mfma_tile<DT, 0, CPL, NSUB, LOADS>(accB, xr, cur, o);
  pipe_epilogue<NSUB, PPQ>(accA, prev_code, best, code, Qp);
  pipe_mfma_tile<DT, 1, CPL, NSUB, LOADS>(accA, xr, cur, o);
  pipe_epilogue<NSUB, PPQ>(accB, tb << 4, best, code, Qp);
  if constexpr (L::TILES == 4) {
    pipe_mfma_tile<DT, 2, CPL, NSUB, LOADS>(accB, xr, cur, o);
    pipe_epilogue<NSUB, PPQ>(accA, (tb + 1) << 4, best, code, Qp);
    pipe_mfma_tile<DT, 3, CPL, NSUB, LOADS>(accA, xr, cur, o);
    pipe_epilogue<NSUB, PPQ>(accB, (tb + 2) << 4, best, code, Qp);
  }
  prev_code = (tb + L::TILES - 1) << 4;
  lds_at<float>(nxt, o.n_store, 0) = nn - Q;
  // interleave: the first few LDS reads, then one MFMA, a few vector
  // instructions and one LDS read, repeated
  __builtin_amdgcn_sched_group_barrier(0x100, 6, 0);
#pragma unroll
  for (int i = 0; i < L::TILES * NSUB * CPL; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x002, 4, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
  }
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
}

// Largest ratio of squared point norms within a workgroup for which one
// shift serves all its points: the 16-ulp tie window and the rounding of
// min_dist then stay below 2^-19 * 64 = 2^-13 of each point's |x|^2.  A
// workgroup with a wider spread is left to assign_pipe_wide_kernel, which
// shifts each point by its own bound.
constexpr float PIPE_WIDE_RATIO = 64.f;

// One workgroup's block of PPB points against all centroids.  PPQ = false:
// the workgroup's shift Q is folded into the stored scores (no cost per
// tile); a block whose squared norms spread by more than PIPE_WIDE_RATIO is
// only flagged (wide[blk] = 1) and left alone.  PPQ = true: each point's own
// shift, subtracted in the epilogue (16 subtractions per tile and point tile).
template <int DT, int CPL, int NSUB, bool PPQ>
__device__ __forceinline__ void pipe_block(int blk, const uint4* __restrict__ X,
                                           const u32x4* __restrict__ chat4,
                                           const float* __restrict__ cinit, int N, int nst,
                                           int32_t* __restrict__ idx, float* __restrict__ min_dist,
                                           double* __restrict__ objpart, int32_t* __restrict__ wide,
                                           char* buf0, char* buf1, float* lds_q, float* lds_qmin,
                                           double* lds_obj) {
  using L = PipeLayout<CPL>;
  constexpr int RC = L::RC;
  constexpr int PPW = 32 * NSUB;           // points per wave
  constexpr int PPB = 4 * PPW;             // points per workgroup
  constexpr int LOADS = L::TCS * L::RCP / ASSIGN_THREADS;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int n = lane & 31, h = lane >> 5;

  PipeOffsets<CPL, LOADS> o;
  pipe_offsets<CPL, LOADS>(o, tid, n, h);
  const int pbase = blk * PPB + wave * PPW;
  uint4 xr[NSUB][CPL];
  // The block's points to registers.  When they fill exactly the two stage
  // buffers, they go through LDS: loaded row-contiguous (each instruction
  // fetches whole rows), then read in the matrix-operand layout.  A lane's
  // direct fragments (16 bytes of each of 32 rows per instruction) cost about
  // as long again from cache as from memory: the loads' own cost, not the
  // latency.  The first centroid stage then follows into buf0.
  constexpr bool XLDS = PPB == 2 * L::TCS;
  float n0;
  if constexpr (XLDS) {
    pipe_issue_rows<CPL, LOADS>(X, blk * PPB, N, tid, buf0);
    pipe_issue_rows<CPL, LOADS>(X, blk * PPB + L::TCS, N, tid, buf1);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    char* xb = wave * PPW < L::TCS ? buf0 : buf1;   // the wave's rows (uniform)
    const int t0 = (wave * PPW % L::TCS) / 32;       // its first 32-row tile there
#pragma unroll
    for (int p = 0; p < NSUB; ++p)
#pragma unroll
      for (int c = 0; c < CPL; ++c) xr[p][c] = lds_at<uint4>(xb, o.a[c], (t0 + p) * L::TILE);
    __syncthreads();  // every wave has its rows before buf0 takes the first stage
    n0 = pipe_issue_stage<CPL, LOADS>(chat4, cinit, 0, tid, o, buf0);
  } else {
    n0 = pipe_issue_stage<CPL, LOADS>(chat4, cinit, 0, tid, o, buf0);
#pragma unroll
    for (int p = 0; p < NSUB; ++p) {
      const int pt = pbase + p * 32 + n;
#pragma unroll
      for (int c = 0; c < CPL; ++c)
        xr[p][c] = pt < N ? X[(size_t)pt * RC + h * CPL + c] : make_uint4(0, 0, 0, 0);
    }
  }
  float xn[NSUB];
  float xmax = 0.f, xmin = __builtin_inff();
#pragma unroll
  for (int p = 0; p < NSUB; ++p) {
    const int pt = pbase + p * 32 + n;
    const bool ok = pt < N;
    float ss = 0.f;
#pragma unroll
    for (int c = 0; c < CPL; ++c) ss = chunk_sumsq<DT>(xr[p][c], ss);
    ss += __shfl_xor(ss, 32);
    xn[p] = ss;
    // points past N and points whose norm is not finite (left unassigned) do not count
    const bool fin = ok && ss <= __FLT_MAX__;
    xmax = fin ? __builtin_fmaxf(xmax, ss) : xmax;
    xmin = fin ? __builtin_fminf(xmin, ss) : xmin;
  }
  float Q = 0.f;
  if constexpr (!PPQ) {
#pragma unroll
    for (int msk = 1; msk < 64; msk <<= 1) {
      xmax = __builtin_fmaxf(xmax, __shfl_xor(xmax, msk));
      xmin = __builtin_fminf(xmin, __shfl_xor(xmin, msk));
    }
    if (lane == 0) {
      lds_q[wave] = xmax;
      lds_qmin[wave] = xmin;
    }
    __syncthreads();
    const float wmax =
        __builtin_fmaxf(__builtin_fmaxf(lds_q[0], lds_q[1]), __builtin_fmaxf(lds_q[2], lds_q[3]));
    const float wmin = __builtin_fminf(__builtin_fminf(lds_qmin[0], lds_qmin[1]),
                                       __builtin_fminf(lds_qmin[2], lds_qmin[3]));
    // the same value in every thread (from LDS after a barrier): a uniform branch
    const bool spread = wmax > PIPE_WIDE_RATIO * wmin;
    if (tid == 0) wide[blk] = spread ? 1 : 0;
    if (spread) {
      __builtin_amdgcn_s_waitcnt(0);  // the first stage's loads into LDS complete before exit
      return;
    }
    // Q >= max |x|^2 / 2 with a relative margin of 2^-8 (far above fp32 rounding)
    Q = __builtin_fmaf(0.5f * wmax, 1.0f + 0x1p-8f, 1e-30f);
  }
  // per point: its own |x|^2 / 2 with the same margin (used when PPQ)
  float Qp[NSUB];
#pragma unroll
  for (int p = 0; p < NSUB; ++p) Qp[p] = __builtin_fmaf(0.5f * xn[p], 1.0f + 0x1p-8f, 1e-30f);

  float best[NSUB];
  uint32_t code[NSUB];
#pragma unroll
  for (int p = 0; p < NSUB; ++p) {
    best[p] = -__builtin_inff();
    code[p] = 0;
  }
  // accA holds the previous tile; before the first tile it is a dummy at the
  // most negative score, which every real score replaces
  f32x16 accA[NSUB], accB[NSUB];
#pragma unroll
  for (int p = 0; p < NSUB; ++p)
#pragma unroll
    for (int j = 0; j < 16; ++j) accA[p][j] = -0x1.fffffep127f;
  uint32_t prev_code = 0;

  lds_at<float>(buf0, o.n_store, 0) = n0 - Q;
  float carry = pipe_score<CPL>(cinit, nst > 1 ? 1 : 0, tid);  // the score of stage 1
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  int st = 0;
  for (; st + 2 <= nst; st += 2) {   // two stages per trip: each buffer is a fixed array
    pipe_stage<DT, CPL, NSUB, LOADS, PPQ>(st, st + 1, nst, carry, accA, accB, xr, buf0, buf1, o,
                                          chat4, cinit, Q, Qp, tid, prev_code, best, code);
    pipe_stage<DT, CPL, NSUB, LOADS, PPQ>(st + 1, st + 2 < nst ? st + 2 : st + 1, nst, carry, accA,
                                          accB, xr, buf1, buf0, o, chat4, cinit, Q, Qp, tid,
                                          prev_code, best, code);
  }
  if (st < nst)
    pipe_stage<DT, CPL, NSUB, LOADS, PPQ>(st, st, nst, carry, accA, accB, xr, buf0, buf1, o, chat4,
                                          cinit, Q, Qp, tid, prev_code, best, code);
  pipe_epilogue<NSUB, PPQ>(accA, prev_code, best, code, Qp);

  double obj = 0.0;
#pragma unroll
  for (int p = 0; p < NSUB; ++p) {
    float v = best[p];
    const uint32_t j = code[p] & 15u;
    int i = (int)((code[p] >> 4) * 32 + 8 * (j >> 2) + 4 * h + (j & 3));
    const float vo = __shfl_xor(v, 32);
    const int io = __shfl_xor(i, 32);
    const bool take = (vo > v) || (vo == v && io < i);
    v = take ? vo : v;
    i = take ? io : i;
    const int pt = pbase + p * 32 + n;
    if (h == 0 && pt < N) {
      // unassigned: a norm that is not finite, or no real centroid's score finite
      const bool asg = xn[p] <= __FLT_MAX__ && v > -__FLT_MAX__;
      const float md = __builtin_fmaxf(__builtin_fmaf(-2.f, v + (PPQ ? Qp[p] : Q), xn[p]), 0.f);
      idx[pt] = asg ? i : -1;
      min_dist[pt] = asg ? md : __builtin_nanf("");
      obj += asg ? (double)md : 0.0;
    }
  }
#pragma unroll
  for (int msk = 1; msk < 64; msk <<= 1) obj += __shfl_xor(obj, msk);
  if (lane == 0) lds_obj[wave] = obj;
  __syncthreads();
  if (tid == 0) objpart[blk] = ((lds_obj[0] + lds_obj[1]) + lds_obj[2]) + lds_obj[3];
}

// The assignment of one block of points per workgroup with the workgroup's
// shift; blocks whose norms spread widely are flagged in `wide` (per
// instance, one int per block) and left to assign_pipe_wide_kernel.
template <int DT, int CPL, int NSUB>
__global__ __launch_bounds__(ASSIGN_THREADS, 2) void assign_pipe_kernel(
    const uint4* __restrict__ X, const uint4* __restrict__ chat, const float* __restrict__ cinit,
    int N, int Kp, int32_t* __restrict__ idx, float* __restrict__ min_dist,
    double* __restrict__ objpart, int32_t* __restrict__ wide) {
  static_assert(DT != DT_F32, "16-bit storage types only");
  static_assert(CPL >= 2, "16-bit rows of 16 elements run on the fp32 kernel");
  using L = PipeLayout<CPL>;
  static_assert(ASSIGN_KPAD % L::TCS == 0, "K is padded to whole stages");
  static_assert(L::TCS * L::RCP / ASSIGN_THREADS * ASSIGN_THREADS == L::TCS * L::RCP,
                "stage must split evenly");
  __shared__ __attribute__((aligned(16))) char buf0[L::STAGE];
  __shared__ __attribute__((aligned(16))) char buf1[L::STAGE];
  __shared__ float lds_q[4], lds_qmin[4];
  __shared__ double lds_obj[4];
  const int b = blockIdx.y, nblk = gridDim.x;
  pipe_block<DT, CPL, NSUB, false>(
      blockIdx.x, X + (size_t)b * N * L::RC,
      reinterpret_cast<const u32x4*>(chat) + (size_t)b * Kp * L::RC, cinit + (size_t)b * Kp, N,
      Kp / L::TCS, idx + (size_t)b * N, min_dist + (size_t)b * N, objpart + (size_t)b * nblk,
      wide + (size_t)b * nblk, buf0, buf1, lds_q, lds_qmin, lds_obj);
}

// The flagged blocks, each point shifted by its own bound.  A fixed grid of
// workgroups splits the blocks into contiguous ranges; each wave reads 64
// flags of its range at once (one per lane) and the workgroup assigns the
// flagged blocks among them, so with no wide block it costs one read of the
// flags per 64 blocks.
template <int DT, int CPL, int NSUB>
__global__ __launch_bounds__(ASSIGN_THREADS, 2) void assign_pipe_wide_kernel(
    const uint4* __restrict__ X, const uint4* __restrict__ chat, const float* __restrict__ cinit,
    int N, int Kp, int nblk, int32_t* __restrict__ idx, float* __restrict__ min_dist,
    double* __restrict__ objpart, const int32_t* __restrict__ wide) {
  using L = PipeLayout<CPL>;
  __shared__ __attribute__((aligned(16))) char buf0[L::STAGE];
  __shared__ __attribute__((aligned(16))) char buf1[L::STAGE];
  __shared__ double lds_obj[4];
  const int b = blockIdx.y;
  const int32_t* wb = wide + (size_t)b * nblk;
  const int per = (nblk + gridDim.x - 1) / gridDim.x;
  const int r0 = blockIdx.x * per, r1 = min(r0 + per, nblk);
  for (int g0 = r0; g0 < r1; g0 += 64) {
    const int bl = g0 + (threadIdx.x & 63);
    // every wave reads the same 64 flags, so the mask is the same in all of them
    uint64_t m = __ballot(bl < r1 && wb[bl] != 0);
    while (m != 0) {
      const int blk = g0 + __builtin_ctzll(m);
      m &= m - 1;
      pipe_block<DT, CPL, NSUB, true>(
          blk, X + (size_t)b * N * L::RC,
          reinterpret_cast<const u32x4*>(chat) + (size_t)b * Kp * L::RC, cinit + (size_t)b * Kp, N,
          Kp / L::TCS, idx + (size_t)b * N, min_dist + (size_t)b * N, objpart + (size_t)b * nblk,
          nullptr, buf0, buf1, nullptr, nullptr, lds_obj);
      __syncthreads();  // every wave is done with the stage buffers before the next block
    }
  }
}

// Workgroups of the wide-block pass, over all instances: enough to cover a
// few flagged blocks per CU, few enough that reading the flags is cheap when
// none is set.
constexpr int64_t PIPE_WIDE_GRID = 512;

template <int DT, int CPL, int NSUB>
hipError_t launch_pipe(const void* X, const Workspace& w, int64_t B, int64_t N,
                              int32_t* idx, float* min_dist, hipStream_t s) {
  const dim3 grid((unsigned)w.n_assign_blocks, (unsigned)B), block(ASSIGN_THREADS);
  assign_pipe_kernel<DT, CPL, NSUB><<<grid, block, 0, s>>>(
      (const uint4*)X, (const uint4*)w.chat, w.cinit, (int)N, (int)w.Kp, idx, min_dist, w.objpart,
      w.wide);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t per = (PIPE_WIDE_GRID + B - 1) / B;  // workgroups per instance
  const int64_t nw = w.n_assign_blocks < per ? w.n_assign_blocks : per;
  assign_pipe_wide_kernel<DT, CPL, NSUB><<<dim3((unsigned)nw, (unsigned)B), block, 0, s>>>(
      (const uint4*)X, (const uint4*)w.chat, w.cinit, (int)N, (int)w.Kp, (int)w.n_assign_blocks,
      idx, min_dist, w.objpart, w.wide);
  return hipGetLastError();
}

// CPL = D / 16 chunks per lane (2 .. 16: 16-bit rows of 16 run as fp32);
// NSUB must agree with assign_nsub16(D).
template <int DT>
hipError_t launch_pipe_dt(const void* X, const Workspace& w, int64_t B, int64_t N,
                                 int64_t D, int32_t* idx, float* min_dist, hipStream_t s) {
  if (D % 16 != 0) return hipErrorInvalidValue;
  switch (D / 16) {
    case 2: return launch_pipe<DT, 2, 4>(X, w, B, N, idx, min_dist, s);
    case 3: return launch_pipe<DT, 3, 4>(X, w, B, N, idx, min_dist, s);
    case 4: return launch_pipe<DT, 4, 4>(X, w, B, N, idx, min_dist, s);
    case 5: return launch_pipe<DT, 5, 2>(X, w, B, N, idx, min_dist, s);
    case 6: return launch_pipe<DT, 6, 2>(X, w, B, N, idx, min_dist, s);
    case 7: return launch_pipe<DT, 7, 2>(X, w, B, N, idx, min_dist, s);
    case 8: return launch_pipe<DT, 8, 2>(X, w, B, N, idx, min_dist, s);
    case 9: return launch_pipe<DT, 9, 1>(X, w, B, N, idx, min_dist, s);
    case 10: return launch_pipe<DT, 10, 1>(X, w, B, N, idx, min_dist, s);
    case 11: return launch_pipe<DT, 11, 1>(X, w, B, N, idx, min_dist, s);
    case 12: return launch_pipe<DT, 12, 1>(X, w, B, N, idx, min_dist, s);
    case 13: return launch_pipe<DT, 13, 1>(X, w, B, N, idx, min_dist, s);
    case 14: return launch_pipe<DT, 14, 1>(X, w, B, N, idx, min_dist, s);
    case 15: return launch_pipe<DT, 15, 1>(X, w, B, N, idx, min_dist, s);
    case 16: return launch_pipe<DT, 16, 1>(X, w, B, N, idx, min_dist, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace fkm
