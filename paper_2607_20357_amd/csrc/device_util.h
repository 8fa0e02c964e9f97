// Small device helpers shared by the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace svl {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t h) {
  return __uint_as_float(h << 16);
}

// Round-to-nearest-even float -> bf16 bits (NaN stays NaN).
__device__ __forceinline__ uint16_t f32_to_bf16_bits(float f) {
  __bf16 b = static_cast<__bf16>(f);
  return __builtin_bit_cast(uint16_t, b);
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return (uint32_t)f32_to_bf16_bits(lo) | ((uint32_t)f32_to_bf16_bits(hi) << 16);
}

// Index of the group whose first tile is the largest tile0 <= t (groups are
// sorted by tile0, group 0 starts at 0).
template <class G>
__device__ __forceinline__ int find_group(const G* groups, int ngroups, int t) {
  int lo = 0, hi = ngroups - 1;
  while (lo < hi) {
    int mid = (lo + hi + 1) >> 1;
    if (groups[mid].tile0 <= t) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// Workgroup index -> tile index such that consecutive tiles land on the same
// XCD.  The hardware hands workgroup i to XCD i % 8; tiles that share a
// weight slice (M tiles and split-K pieces of one N tile) are consecutive in
// tile order, so they run on one XCD at about the same time and share the
// slice through that XCD's L2.  gridDim.x is a multiple of 8.
__device__ __forceinline__ int xcd_tile_index() {
  const int per = gridDim.x >> 3;
  return (int)(blockIdx.x & 7) * per + (int)(blockIdx.x >> 3);
}

__device__ __forceinline__ float warp_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

}  // namespace svl

namespace svl {

typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));

// Float -> 16-bit activation bits (fp16 or bf16, round to nearest even).
template <bool F16>
__device__ __forceinline__ uint16_t f32_to_act_bits(float f) {
  if constexpr (F16) {
    _Float16 h = static_cast<_Float16>(f);
    return __builtin_bit_cast(uint16_t, h);
  } else {
    return f32_to_bf16_bits(f);
  }
}

template <bool F16>
__device__ __forceinline__ float act_bits_to_f32(uint32_t h) {
  if constexpr (F16) {
    return static_cast<float>(__builtin_bit_cast(_Float16, (uint16_t)h));
  } else {
    return bf16_bits_to_f32(h);
  }
}

template <bool F16>
__device__ __forceinline__ uint32_t pack_act2(float lo, float hi) {
  if constexpr (F16) {
    // one packed conversion, rounding to nearest even as the scalar one does
    typedef float f32x2_t __attribute__((ext_vector_type(2)));
    typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{lo, hi}, f16x2_t));
  } else {
    return (uint32_t)f32_to_act_bits<false>(lo) | ((uint32_t)f32_to_act_bits<false>(hi) << 16);
  }
}

// Low bf16 parts of two values whose high parts are the bf16 word `hi`
// (pack_act2<false>(lo_val, hi_val)): bf16(v - bf16(v)) each, so the two
// words together carry v to about 16 significant bits.
__device__ __forceinline__ uint32_t bf16_low2(float v0, float v1, uint32_t hi) {
  return pack_bf16x2(v0 - bf16_bits_to_f32(hi & 0xffffu), v1 - bf16_bits_to_f32(hi >> 16));
}

// Two bf16 values (one 32-bit word) -> the same two values as fp16.  Exact
// for magnitudes in [2^-14, 65504]; smaller ones become fp16 subnormals
// (absolute error at most 2^-25).
__device__ __forceinline__ uint32_t bf16x2_to_f16x2(uint32_t w) {
  const float lo = __uint_as_float(w << 16), hi = __uint_as_float(w & 0xffff0000u);
  return pack_act2<true>(lo, hi);
}

// 16 x 16 x 32 MFMA on 8-element fragments of 16-bit activations.
template <bool F16>
__device__ __forceinline__ floatx4 mfma16x16x32(const uint4& a, const uint4& b, const floatx4& c) {
  if constexpr (F16) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8_t, a),
                                                  __builtin_bit_cast(f16x8_t, b), c, 0, 0, 0);
  } else {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                   __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
  }
}

}  // namespace svl
