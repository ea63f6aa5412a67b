// assign.hip -- the assignment step of the Lloyd iteration (paper Section 5:
// squared Euclidean distance of each point to all K centroids, then the
// arg-min), fused so that the N x K distance matrix is never stored.  This
// file holds the centroid preparation, the fp32 kernel, the row-width copies
// and the dispatch; the bf16/fp16 kernels are in assign_pipe.h (D <= 256),
// assign_smallk.h (small K) and assign_tiled.hip (wider rows).
//
// For point x and centroid c the kernels maximise
//     s(x, c) = <x, c^> - |c^|^2 / 2
// which orders the centroids exactly as |x - c^|^2 = |x|^2 - 2 s(x, c) does
// (|x|^2 is common to all of them).  c^ is the centroid rounded once to the
// storage type of x; <x, c^> runs on the matrix cores with fp32 accumulation,
// and -|c^|^2 / 2 enters as the accumulator's initial value.
//
// fp32 kernel layout, one 16x16x4 MFMA tile: 16 centroids (A rows) x 16
// points (B columns).  Lane l = 16 g + m supplies centroid row m and point
// column m for the k-slice g (the k-to-lane map is the same for A and B, so
// any fixed split of the D dimensions over the four lane groups gives the same
// contraction); it receives accumulator rows 4 g .. 4 g + 3 of column m.  A
// lane therefore keeps a running best over its own quarter of the centroids
// of one point, and the four quarters are merged once at the end.
#include "fkm_device.h"

namespace fkm {

// ---------------------------------------------------------------------------
// prep: c^ = round(c) to the storage type and cinit = -|c^|^2 / 2 (fp32),
// one wave per centroid row; the squared norm is summed lane-strided and then
// by a fixed xor butterfly, so every lane (and every call) gets the same bits.
// Rows K..Kp-1 of each instance are padding: zero, with cinit = -FLT_MAX.
template <int DT>
__global__ __launch_bounds__(256) void prep_kernel(const float* __restrict__ C, int64_t B, int K,
                                                   int Kp, int D, void* __restrict__ chat,
                                                   float* __restrict__ cinit) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= B * Kp) return;
  const int64_t b = row / Kp;
  const int k = (int)(row % Kp);
  const bool pad = k >= K;
  prep_row<DT>(C + (b * K + (pad ? 0 : k)) * D, pad, D, lane,
               (char*)chat + row * D * (DT == DT_F32 ? 4 : 2), cinit + row);
}

// ---------------------------------------------------------------------------
// Resident-X assignment.  CPL = 16-byte chunks of one point held by one lane
// (the point's row is split over the four lane groups), NSUB = 16-point MFMA
// column tiles per wave.  A centroid row of RC chunks sits in LDS at a
// power-of-two stride RCP >= RC, XOR-swizzled within it.
template <int DT, int CPL, int NSUB>
__global__ __launch_bounds__(ASSIGN_THREADS, 2) void assign_resident_kernel(
    const uint4* __restrict__ X, const uint4* __restrict__ chat, const float* __restrict__ cinit,
    int N, int K, int Kp, int32_t* __restrict__ idx, float* __restrict__ min_dist,
    double* __restrict__ objpart) {
  constexpr int RC = 4 * CPL;              // 16-byte chunks per row
  constexpr int RCP = pow2_at_least(RC);   // chunk slots per LDS row
  constexpr int SWZ = RCP < 16 ? RCP - 1 : 15;
  constexpr int TCS = ASSIGN_TCS;
  constexpr int PPW = 16 * NSUB;           // points per wave
  constexpr int PPB = 4 * PPW;             // points per workgroup
  constexpr int LOADS = TCS * RC / ASSIGN_THREADS;  // chunks per thread per stage
  static_assert(LOADS * ASSIGN_THREADS == TCS * RC, "stage must split evenly");

  __shared__ uint4 lds_c[2][TCS * RCP];
  __shared__ __attribute__((aligned(16))) float lds_n[2][TCS];
  __shared__ double lds_obj[4];

  const int b = blockIdx.y;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int m = lane & 15, g = lane >> 4;
  X += (size_t)b * N * RC;
  chat += (size_t)b * Kp * RC;
  cinit += (size_t)b * Kp;
  idx += (size_t)b * N;
  min_dist += (size_t)b * N;

  // ---- this lane's slices of its NSUB points, and their squared norms
  const int pbase = blockIdx.x * PPB + wave * PPW;
  uint4 xr[NSUB][CPL];
  float xn[NSUB];
#pragma unroll
  for (int p = 0; p < NSUB; ++p) {
    const int pt = pbase + p * 16 + m;
    const bool ok = pt < N;
    float ss = 0.f;
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
      xr[p][c] = ok ? X[(size_t)pt * RC + g * CPL + c] : make_uint4(0, 0, 0, 0);
      ss = chunk_sumsq<DT>(xr[p][c], ss);
    }
    ss += __shfl_xor(ss, 16);
    ss += __shfl_xor(ss, 32);
    xn[p] = ss;
  }

  // ---- centroid stages through LDS (double-buffered)
  const int nst = (K + TCS - 1) / TCS;
  uint4 pre[LOADS];
  float pren = 0.f;
  auto load_stage = [&](int st) {
    const int kb = st * TCS;
#pragma unroll
    for (int u = 0; u < LOADS; ++u) {
      const int q = tid + u * ASSIGN_THREADS;
      const int r = q / RC, c = q % RC;
      pre[u] = (kb + r < K) ? chat[(size_t)(kb + r) * RC + c] : make_uint4(0, 0, 0, 0);
    }
    if (tid < TCS) pren = (kb + tid < K) ? cinit[kb + tid] : -__builtin_inff();
  };
  auto store_stage = [&](int buf) {
#pragma unroll
    for (int u = 0; u < LOADS; ++u) {
      const int q = tid + u * ASSIGN_THREADS;
      const int r = q / RC, c = q % RC;
      lds_c[buf][r * RCP + (c ^ (r & SWZ))] = pre[u];
    }
    if (tid < TCS) lds_n[buf][tid] = pren;
  };

  float best[NSUB];
  int code[NSUB];
#pragma unroll
  for (int p = 0; p < NSUB; ++p) {
    best[p] = -__builtin_inff();
    code[p] = 0;
  }

  load_stage(0);
  store_stage(0);
  __syncthreads();
  for (int st = 0; st < nst; ++st) {
    const int buf = st & 1;
    if (st + 1 < nst) load_stage(st + 1);
#pragma unroll 1
    for (int tile = 0; tile < TCS / 16; ++tile) {
      const int row = tile * 16 + m;
      const f32x4 cin = *reinterpret_cast<const f32x4*>(&lds_n[buf][tile * 16 + 4 * g]);
      uint4 a[CPL];
#pragma unroll
      for (int c = 0; c < CPL; ++c) a[c] = lds_c[buf][row * RCP + ((g * CPL + c) ^ (row & SWZ))];
      const int kcode = st * TCS + tile * 16;  // + 4 g + j is the centroid index
#pragma unroll
      for (int p = 0; p < NSUB; ++p) {
        f32x4 acc = cin;
#pragma unroll
        for (int c = 0; c < CPL; ++c) acc = mfma_chunk<DT>(a[c], xr[p][c], acc);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const bool gt = acc[j] > best[p];
          best[p] = gt ? acc[j] : best[p];
          code[p] = gt ? kcode + j : code[p];
        }
      }
    }
    if (st + 1 < nst) store_stage(buf ^ 1);
    __syncthreads();
  }

  // ---- merge the four centroid quarters of each point; ties -> lower index
  double obj = 0.0;
#pragma unroll
  for (int p = 0; p < NSUB; ++p) {
    float v = best[p];
    int i = code[p] + 4 * g;
#pragma unroll
    for (int msk = 16; msk <= 32; msk <<= 1) {
      const float vo = __shfl_xor(v, msk);
      const int io = __shfl_xor(i, msk);
      const bool take = (vo > v) || (vo == v && io < i);
      v = take ? vo : v;
      i = take ? io : i;
    }
    const int pt = pbase + p * 16 + m;
    if (g == 0 && pt < N) {
      // unassigned: a norm that is not finite, or no real centroid's score finite
      const bool asg = xn[p] <= __FLT_MAX__ && v > -__FLT_MAX__;
      const float md = __builtin_fmaxf(__builtin_fmaf(-2.f, v, xn[p]), 0.f);
      idx[pt] = asg ? i : -1;
      min_dist[pt] = asg ? md : __builtin_nanf("");
      obj += asg ? (double)md : 0.0;
    }
  }
#pragma unroll
  for (int msk = 1; msk < 64; msk <<= 1) obj += __shfl_xor(obj, msk);
  if (lane == 0) lds_obj[wave] = obj;
  __syncthreads();
  if (tid == 0)
    objpart[(size_t)b * gridDim.x + blockIdx.x] = ((lds_obj[0] + lds_obj[1]) + lds_obj[2]) + lds_obj[3];
}


// ---------------------------------------------------------------------------
hipError_t launch_prep(const float* C, int dt, int64_t B, int64_t K, int64_t Kp, int64_t D,
                       void* chat, float* cinit, hipStream_t s) {
  const dim3 grid((unsigned)((B * Kp + 3) / 4)), block(256);
  if (dt == DT_BF16)
    prep_kernel<DT_BF16><<<grid, block, 0, s>>>(C, B, (int)K, (int)Kp, (int)D, chat, cinit);
  else if (dt == DT_F16)
    prep_kernel<DT_F16><<<grid, block, 0, s>>>(C, B, (int)K, (int)Kp, (int)D, chat, cinit);
  else
    prep_kernel<DT_F32><<<grid, block, 0, s>>>(C, B, (int)K, (int)Kp, (int)D, chat, cinit);
  return hipGetLastError();
}

// NSUB as assign_nsub32 gives it: the D-dependent value, or 2 for small problems.
template <int DT, int CPL>
static hipError_t launch_resident(const void* X, const Workspace& w, int64_t B, int64_t N,
                                  int64_t K, int32_t* idx, float* min_dist, hipStream_t s) {
  constexpr int BASE = CPL <= 4 ? 8 : (CPL <= 8 ? 4 : 2);
  const dim3 grid((unsigned)w.n_assign_blocks, (unsigned)B), block(ASSIGN_THREADS);
  const uint4* Xv = (const uint4*)X;
  const uint4* ch = (const uint4*)w.chat;
  if (assign_nsub32(16 * CPL, B * N) == BASE)
    assign_resident_kernel<DT, CPL, BASE><<<grid, block, 0, s>>>(
        Xv, ch, w.cinit, (int)N, (int)K, (int)w.Kp, idx, min_dist, w.objpart);
  else
    assign_resident_kernel<DT, CPL, 2><<<grid, block, 0, s>>>(
        Xv, ch, w.cinit, (int)N, (int)K, (int)w.Kp, idx, min_dist, w.objpart);
  return hipGetLastError();
}

template <int DT>
static hipError_t launch_resident_dt(const void* X, const Workspace& w, int64_t B, int64_t N,
                                     int64_t D, int64_t K, int32_t* idx, float* min_dist,
                                     hipStream_t s) {
  if (D % 16 != 0) return hipErrorInvalidValue;
  switch (D / 16) {  // chunks per lane
    case 1: return launch_resident<DT, 1>(X, w, B, N, K, idx, min_dist, s);
    case 2: return launch_resident<DT, 2>(X, w, B, N, K, idx, min_dist, s);
    case 3: return launch_resident<DT, 3>(X, w, B, N, K, idx, min_dist, s);
    case 4: return launch_resident<DT, 4>(X, w, B, N, K, idx, min_dist, s);
    case 5: return launch_resident<DT, 5>(X, w, B, N, K, idx, min_dist, s);
    case 6: return launch_resident<DT, 6>(X, w, B, N, K, idx, min_dist, s);
    case 7: return launch_resident<DT, 7>(X, w, B, N, K, idx, min_dist, s);
    case 8: return launch_resident<DT, 8>(X, w, B, N, K, idx, min_dist, s);
    case 9: return launch_resident<DT, 9>(X, w, B, N, K, idx, min_dist, s);
    case 10: return launch_resident<DT, 10>(X, w, B, N, K, idx, min_dist, s);
    case 11: return launch_resident<DT, 11>(X, w, B, N, K, idx, min_dist, s);
    case 12: return launch_resident<DT, 12>(X, w, B, N, K, idx, min_dist, s);
    case 13: return launch_resident<DT, 13>(X, w, B, N, K, idx, min_dist, s);
    case 14: return launch_resident<DT, 14>(X, w, B, N, K, idx, min_dist, s);
    case 15: return launch_resident<DT, 15>(X, w, B, N, K, idx, min_dist, s);
    case 16: return launch_resident<DT, 16>(X, w, B, N, K, idx, min_dist, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_assign(const void* X, int dt, const Workspace& w, int64_t B, int64_t N,
                         int64_t D, int64_t K, int32_t* idx, float* min_dist, hipStream_t s) {
  if (assign_tiled(dt, D)) return launch_assign_tiled(X, dt, w, B, N, D, idx, min_dist, s);
  if (!assign_resident_ok(dt, D)) return hipErrorInvalidValue;
  // small K: the kernel of the fused step, without the sums (the same bits)
  if (sums_ok(dt, D, K)) return launch_sums(X, dt, w, B, N, D, K, SUMS_ASSIGN, idx, min_dist, s);
  if (dt == DT_BF16) return launch_pipe_bf16(X, w, B, N, D, idx, min_dist, s);
  if (dt == DT_F16) return launch_pipe_f16(X, w, B, N, D, idx, min_dist, s);
  return launch_resident_dt<DT_F32>(X, w, B, N, D, K, idx, min_dist, s);
}

// Row width change for rows whose width the kernels do not take: each block
// copies PAD_ROWS rows of width Din into rows of width Dout (zeros past Din).
constexpr int PAD_ROWS = 64;
template <typename T>
__global__ __launch_bounds__(256) void pad_rows_kernel(const T* __restrict__ src, int64_t rows,
                                                       int Din, int Dout, T* __restrict__ dst) {
  const int64_t r0 = (int64_t)blockIdx.x * PAD_ROWS;
  const int64_t left = rows - r0;
  const int nr = left < PAD_ROWS ? (int)left : PAD_ROWS;
  src += r0 * Din;
  dst += r0 * Dout;
  const unsigned total = (unsigned)nr * (unsigned)Dout;
  for (unsigned j = threadIdx.x; j < total; j += 256) {
    const unsigned r = j / (unsigned)Dout, d = j - r * (unsigned)Dout;
    dst[j] = (int)d < Din ? src[(size_t)r * Din + d] : T(0);
  }
}

hipError_t launch_pad_rows(const void* src, int64_t rows, int64_t D, int64_t Dk, int elem_bytes,
                           void* dst, hipStream_t s) {
  const dim3 grid((unsigned)((rows + PAD_ROWS - 1) / PAD_ROWS));
  if (elem_bytes == 2)
    pad_rows_kernel<uint16_t><<<grid, 256, 0, s>>>((const uint16_t*)src, rows, (int)D, (int)Dk,
                                                   (uint16_t*)dst);
  else
    pad_rows_kernel<uint32_t><<<grid, 256, 0, s>>>((const uint32_t*)src, rows, (int)D, (int)Dk,
                                                   (uint32_t*)dst);
  return hipGetLastError();
}

template <int DT>
__global__ __launch_bounds__(256) void widen_rows_kernel(const uint16_t* __restrict__ src,
                                                         int64_t rows, int Din, int Dout,
                                                         float* __restrict__ dst) {
  const int64_t r0 = (int64_t)blockIdx.x * PAD_ROWS;
  const int64_t left = rows - r0;
  const int nr = left < PAD_ROWS ? (int)left : PAD_ROWS;
  src += r0 * Din;
  dst += r0 * Dout;
  const unsigned total = (unsigned)nr * (unsigned)Dout;
  for (unsigned j = threadIdx.x; j < total; j += 256) {
    const unsigned r = j / (unsigned)Dout, d = j - r * (unsigned)Dout;
    dst[j] = (int)d < Din ? Elem<DT>::widen(src[(size_t)r * Din + d]) : 0.f;
  }
}

hipError_t launch_widen_rows(const void* src, int dt, int64_t rows, int64_t D, int64_t Dk,
                             float* dst, hipStream_t s) {
  const dim3 grid((unsigned)((rows + PAD_ROWS - 1) / PAD_ROWS));
  if (dt == DT_BF16)
    widen_rows_kernel<DT_BF16><<<grid, 256, 0, s>>>((const uint16_t*)src, rows, (int)D, (int)Dk, dst);
  else if (dt == DT_F16)
    widen_rows_kernel<DT_F16><<<grid, 256, 0, s>>>((const uint16_t*)src, rows, (int)D, (int)Dk, dst);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_unpad_rows(const float* src, int64_t rows, int64_t Dk, int64_t D, float* dst,
                             hipStream_t s) {
  const dim3 grid((unsigned)((rows + PAD_ROWS - 1) / PAD_ROWS));
  pad_rows_kernel<uint32_t><<<grid, 256, 0, s>>>((const uint32_t*)src, rows, (int)Dk, (int)D,
                                                 (uint32_t*)dst);
  return hipGetLastError();
}

hipError_t launch_sums(const void* X, int dt, const Workspace& w, int64_t B, int64_t N, int64_t D,
                       int64_t K, int mode, int32_t* idx, float* min_dist, hipStream_t s) {
  if (dt == DT_BF16) return launch_sums_bf16(X, w, B, N, D, K, mode, idx, min_dist, s);
  if (dt == DT_F16) return launch_sums_f16(X, w, B, N, D, K, mode, idx, min_dist, s);
  return hipErrorInvalidValue;
}


}  // namespace fkm
