// Lane exchanges inside a 16-lane DPP row (gfx950 data-parallel primitives):
// the value of lane (lane ^ x) for x in {1, 2, 4, 8}, and butterfly
// all-reductions over the 16 lanes.  In a butterfly every lane adds (or
// maxes) the same two operands at every stage, only swapped, so all 16 lanes
// end with bit-identical results.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mixfp4 {

template <int kCtrl>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, kCtrl, 0xF, 0xF, false);
}

// Value of lane (lane ^ kX) within a 16-lane row, kX in {1, 2, 4, 8}.
template <int kX>
__device__ __forceinline__ uint32_t xor_u32(uint32_t v) {
  if constexpr (kX == 1) return dpp_u32<0xB1>(v);                    // quad_perm [1,0,3,2]
  if constexpr (kX == 2) return dpp_u32<0x4E>(v);                    // quad_perm [2,3,0,1]
  if constexpr (kX == 4) return dpp_u32<0x1B>(dpp_u32<0x141>(v));    // half mirror, quad reverse
  return dpp_u32<0x128>(v);                                           // row_ror:8
}

template <int kX>
__device__ __forceinline__ float xor_f32(float v) {
  return __uint_as_float(xor_u32<kX>(__float_as_uint(v)));
}

template <int kX>
__device__ __forceinline__ double xor_f64(double v) {
  const uint64_t u = __builtin_bit_cast(uint64_t, v);
  const uint32_t lo = xor_u32<kX>((uint32_t)u), hi = xor_u32<kX>((uint32_t)(u >> 32));
  return __builtin_bit_cast(double, ((uint64_t)hi << 32) | lo);
}

// All-reductions over the 16 lanes of a DPP row (every lane active).
__device__ __forceinline__ float row16_max(float v) {
  v = fmaxf(v, xor_f32<1>(v));
  v = fmaxf(v, xor_f32<2>(v));
  v = fmaxf(v, xor_f32<4>(v));
  return fmaxf(v, xor_f32<8>(v));
}
__device__ __forceinline__ float row16_sum(float v) {
  v += xor_f32<1>(v);
  v += xor_f32<2>(v);
  v += xor_f32<4>(v);
  return v + xor_f32<8>(v);
}
__device__ __forceinline__ uint32_t row16_sum(uint32_t v) {
  v += xor_u32<1>(v);
  v += xor_u32<2>(v);
  v += xor_u32<4>(v);
  return v + xor_u32<8>(v);
}
__device__ __forceinline__ double row16_sum(double v) {
  v += xor_f64<1>(v);
  v += xor_f64<2>(v);
  v += xor_f64<4>(v);
  return v + xor_f64<8>(v);
}

}  // namespace mixfp4
