// calib.hip -- microbenchmark kernels of libfkm_calib.so (declared in
// include/fkm_calib.h): the matrix-core, streaming-read and row-gather
// ceilings that a benchmark measures in its own run.
#include <hip/hip_runtime.h>

#include "../../include/fkm_calib.h"

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ uint32_t mix(uint32_t x) {
  x ^= x >> 16;
  x *= 0x7feb352du;
  x ^= x >> 15;
  x *= 0x846ca68bu;
  x ^= x >> 16;
  return x;
}

// 8 bf16 values in +-[1, 2) with random mantissas and signs
__device__ u32x4 random_operand(uint32_t seed) {
  u32x4 r;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t a = mix(seed * 4 + i);
    const uint32_t lo = 0x3f80u | (a & 0x7fu) | (((a >> 7) & 1u) << 15);
    const uint32_t hi = 0x3f80u | ((a >> 8) & 0x7fu) | (((a >> 15) & 1u) << 15);
    r[i] = lo | (hi << 16);
  }
  return r;
}

constexpr int SETS = 8, CHAINS = 4;

__global__ __launch_bounds__(256, 2) void mfma_loop_kernel(float* __restrict__ out, int iters) {
  u32x4 a[SETS], b[SETS];
#pragma unroll
  for (int j = 0; j < SETS; ++j) {
    a[j] = random_operand(threadIdx.x * 131u + j * 7u + blockIdx.x * 977u);
    b[j] = random_operand(threadIdx.x * 17u + j * 1001u + 5u);
  }
  f32x16 acc[CHAINS];
#pragma unroll
  for (int p = 0; p < CHAINS; ++p)
#pragma unroll
    for (int i = 0; i < 16; ++i) acc[p][i] = 0.f;
  for (int it = 0; it < iters; ++it)
#pragma unroll
    for (int j = 0; j < SETS; ++j)
#pragma unroll
      for (int p = 0; p < CHAINS; ++p)
        acc[p] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a[j]),
                                                         __builtin_bit_cast(bf16x8, b[(j + p) % SETS]),
                                                         acc[p], 0, 0, 0);
  float s = 0.f;
#pragma unroll
  for (int p = 0; p < CHAINS; ++p) s += acc[p][0] + acc[p][15];
  out[blockIdx.x * 256 + threadIdx.x] = s;
}

// Each workgroup streams one contiguous range, 8 loads of 4 KB per workgroup
// in flight, with the non-temporal hint: on the MI355X this reads ~25% faster
// than a grid-stride loop of ordinary loads (whose waves touch 8 scattered
// 1 KB pieces per step), so it is the fairer ceiling for a streaming read.
__global__ __launch_bounds__(256) void read_kernel(const u32x4* __restrict__ x, size_t n,
                                                   uint32_t* __restrict__ out) {
  constexpr int U = 8;
  uint32_t acc = 0;
  const size_t per = (n + gridDim.x - 1) / gridDim.x;
  const size_t b0 = (size_t)blockIdx.x * per;
  const size_t b1 = b0 + per < n ? b0 + per : n;
  size_t i = b0 + threadIdx.x;
  for (; i + (U - 1) * 256 < b1; i += U * 256) {
    u32x4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = __builtin_nontemporal_load(&x[i + u * 256]);
#pragma unroll
    for (int u = 0; u < U; ++u) acc ^= v[u][0] + v[u][1] + v[u][2] + v[u][3];
  }
  for (; i < b1; i += 256) {
    const u32x4 v = x[i];
    acc ^= v[0] + v[3];
  }
  out[blockIdx.x * 256 + threadIdx.x] = acc;
}

// LPR lanes per row (one 16-byte chunk each; rows of rc <= LPR chunks, lanes
// past the row's end idle), 64 / LPR rows per wave step, 8 steps in flight.
// Row indices are clamped to [0, src_rows).
template <int LPR>
__global__ __launch_bounds__(256) void gather_kernel(const u32x4* __restrict__ x, int64_t src_rows,
                                                     int rc, const int32_t* __restrict__ rows,
                                                     int64_t nrows, uint32_t* __restrict__ out) {
  constexpr int RPW = 64 / LPR, U = 8;
  const int lane = threadIdx.x & 63;
  const int64_t w = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int64_t nw = (int64_t)gridDim.x * 4;
  const int r = lane / LPR, q = lane % LPR;
  uint32_t acc = 0;
  for (int64_t j0 = w * RPW * U; j0 < nrows; j0 += nw * RPW * U) {
    u32x4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t j = j0 + u * RPW + r;
      int64_t row = j < nrows ? rows[j] : 0;
      row = row < 0 ? 0 : (row >= src_rows ? src_rows - 1 : row);
      v[u] = (j < nrows && q < rc) ? x[(size_t)row * rc + q] : u32x4{0, 0, 0, 0};
    }
#pragma unroll
    for (int u = 0; u < U; ++u) acc ^= v[u][0] + v[u][2];
  }
  out[blockIdx.x * 256 + threadIdx.x] = acc;
}

}  // namespace

extern "C" {

int fkm_calib_mfma(float* out, int blocks, int iters, void* stream) {
  if (!out || blocks < 1 || iters < 1) return -1;
  mfma_loop_kernel<<<blocks, 256, 0, (hipStream_t)stream>>>(out, iters);
  return hipGetLastError() == hipSuccess ? 0 : -4;
}

int fkm_calib_read(const void* src, size_t bytes, uint32_t* out, int blocks, void* stream) {
  if (!src || !out || blocks < 1 || bytes % 16 != 0 || ((uintptr_t)src & 15)) return -1;
  read_kernel<<<blocks, 256, 0, (hipStream_t)stream>>>((const u32x4*)src, bytes / 16, out);
  return hipGetLastError() == hipSuccess ? 0 : -4;
}

int fkm_calib_gather(const void* src, int64_t src_rows, int row_bytes, const int32_t* rows,
                     int64_t nrows, uint32_t* out, int blocks, void* stream) {
  if (!src || !rows || !out || blocks < 1 || src_rows < 1 || nrows < 0 || row_bytes < 16 ||
      row_bytes > 1024 || row_bytes % 16 != 0 || ((uintptr_t)src & 15))
    return -1;
  const int rc = row_bytes / 16;
  hipStream_t s = (hipStream_t)stream;
  const u32x4* x = (const u32x4*)src;
  if (rc <= 4)
    gather_kernel<4><<<blocks, 256, 0, s>>>(x, src_rows, rc, rows, nrows, out);
  else if (rc <= 16)
    gather_kernel<16><<<blocks, 256, 0, s>>>(x, src_rows, rc, rows, nrows, out);
  else
    gather_kernel<64><<<blocks, 256, 0, s>>>(x, src_rows, rc, rows, nrows, out);
  return hipGetLastError() == hipSuccess ? 0 : -4;
}

}  // extern "C"
