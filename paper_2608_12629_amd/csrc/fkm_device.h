// fkm_device.h -- device helpers shared by the assignment kernels: element
// conversions, squared norms of 16-byte chunks, and the MFMA calls.
#pragma once

#include "fkm_internal.h"

namespace fkm {

// ---------------------------------------------------------------------------
// element helpers
template <int DT> struct Elem;
template <> struct Elem<DT_BF16> {
  static constexpr int per16 = 8;  // elements in 16 bytes
  __device__ static float widen(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }
  __device__ static uint16_t narrow(float f) {
    __bf16 b = (__bf16)f;  // round to nearest even
    return __builtin_bit_cast(uint16_t, b);
  }
};
template <> struct Elem<DT_F16> {
  static constexpr int per16 = 8;
  __device__ static float widen(uint16_t h) { return (float)__builtin_bit_cast(_Float16, h); }
  __device__ static uint16_t narrow(float f) {
    _Float16 b = (_Float16)f;  // round to nearest even
    return __builtin_bit_cast(uint16_t, b);
  }
};
template <> struct Elem<DT_F32> {
  static constexpr int per16 = 4;
};

// Sum of squares of the elements of one 16-byte chunk, widened to fp32,
// accumulated in element order.
template <int DT>
__device__ inline float chunk_sumsq(const uint4& q, float acc) {
  if constexpr (DT == DT_F32) {
    const float v[4] = {__uint_as_float(q.x), __uint_as_float(q.y), __uint_as_float(q.z),
                        __uint_as_float(q.w)};
#pragma unroll
    for (int e = 0; e < 4; ++e) acc = __builtin_fmaf(v[e], v[e], acc);
  } else {
    const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float lo = Elem<DT>::widen((uint16_t)(w[e] & 0xffffu));
      const float hi = Elem<DT>::widen((uint16_t)(w[e] >> 16));
      acc = __builtin_fmaf(lo, lo, acc);
      acc = __builtin_fmaf(hi, hi, acc);
    }
  }
  return acc;
}

// One centroid row for the assignment: c^ = round(c) to the storage type
// into out (D elements) and -|c^|^2 / 2 into *cinit (a padding row: zeros and
// -FLT_MAX), by one wave: the squares are summed lane-strided and then by a
// fixed xor butterfly, so wherever this runs the bits are the same.  A row
// whose |c^|^2 is not finite (a NaN or infinite coordinate) is written as a
// padding row, so it is never chosen and the kernels' scores stay finite or
// NaN-free (an infinite score with position bits in its low mantissa would
// become a signalling NaN in the arg-max tree).
template <int DT>
__device__ inline void prep_row(const float* c, bool pad, int D, int lane, void* out,
                                float* cinit) {
  auto rounded = [&](int d) -> float {
    if constexpr (DT == DT_F32) return c[d];
    else return Elem<DT>::widen(Elem<DT>::narrow(c[d]));
  };
  float ss = 0.f;
  if (!pad) {
    for (int d = lane; d < D; d += 64) {
      const float v = rounded(d);
      ss = __builtin_fmaf(v, v, ss);
    }
  }
#pragma unroll
  for (int m = 1; m < 64; m <<= 1) ss += __shfl_xor(ss, m);
  const bool zero = pad || !(ss <= __FLT_MAX__);  // the same in every lane
  if constexpr (DT == DT_F32) {
    float* o = (float*)out;
    for (int d = lane; d < D; d += 64) o[d] = zero ? 0.f : c[d];
  } else {
    uint16_t* o = (uint16_t*)out;
    for (int d = lane; d < D; d += 64) o[d] = zero ? (uint16_t)0 : Elem<DT>::narrow(c[d]);
  }
  if (lane == 0) *cinit = zero ? -0x1.fffffep127f : -0.5f * ss;
}

// acc += A-chunk x B-chunk over the k-slice these two 16-byte chunks carry.
template <int DT>
__device__ inline f32x4 mfma_chunk(const uint4& a, const uint4& b, f32x4 acc) {
  if constexpr (DT == DT_BF16) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), acc, 0, 0, 0);
  } else if constexpr (DT == DT_F16) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a),
                                                  __builtin_bit_cast(f16x8, b), acc, 0, 0, 0);
  } else {
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), acc, 0, 0, 0);
    return acc;
  }
}


// acc += A-chunk x B-chunk on a 32x32x16 tile (16-bit storage types).
template <int DT>
__device__ inline f32x16 mfma32_chunk(const uint4& a, const uint4& b, f32x16 acc) {
  if constexpr (DT == DT_BF16) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), acc, 0, 0, 0);
  } else {
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a),
                                                  __builtin_bit_cast(f16x8, b), acc, 0, 0, 0);
  }
}

}  // namespace fkm
