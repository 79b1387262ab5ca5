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

// In-register transpose of a 16 x 16 matrix of 4-bit values held by the 16
// lanes of a DPP row: on entry lane i holds row i (value j in bits 4j..4j+3
// of the 64-bit pair (lo, hi)), on exit column i in the same order.  The
// usual recursive block transpose: at distance d = 8, 4, 2, 1 the lanes i and
// i ^ d swap the off-diagonal d x d blocks of their 2d x 2d block (words,
// 16-bit halves, bytes, nibbles), one exchanged word per stage.  Every lane
// of the row must be active.
struct Transpose16 {
  uint32_t send4, keep4x, keep4y, send2, keep2x, keep2y, shl1, shr1, mask1;
  bool low8;
};

__device__ __forceinline__ Transpose16 transpose16_setup(int i) {
  const bool l4 = !(i & 4), l2 = !(i & 2), l1 = !(i & 1);
  Transpose16 t;
  t.low8 = !(i & 8);
  // byte selectors of v_perm_b32(S0, S1): 0-3 pick bytes of S1, 4-7 of S0
  t.send4 = l4 ? 0x07060302u : 0x05040100u;
  t.keep4x = l4 ? 0x05040100u : 0x03020504u;
  t.keep4y = l4 ? 0x07060100u : 0x03020706u;
  t.send2 = l2 ? 0x07050301u : 0x06040200u;
  t.keep2x = l2 ? 0x05020400u : 0x03050104u;
  t.keep2y = l2 ? 0x07020600u : 0x03070106u;
  t.shl1 = l1 ? 4u : 0u;
  t.shr1 = l1 ? 0u : 4u;
  t.mask1 = l1 ? 0x0F0F0F0Fu : 0xF0F0F0F0u;
  return t;
}

__device__ __forceinline__ void transpose16_nibbles(const Transpose16& t, uint32_t& lo, uint32_t& hi) {
  uint32_t x = lo, y = hi, r;
  r = xor_u32<8>(t.low8 ? y : x);                 // 8 x 8 blocks: whole words
  x = t.low8 ? x : r;
  y = t.low8 ? r : y;
  r = xor_u32<4>(__builtin_amdgcn_perm(y, x, t.send4));   // 4 x 4: 16-bit halves
  x = __builtin_amdgcn_perm(r, x, t.keep4x);
  y = __builtin_amdgcn_perm(r, y, t.keep4y);
  r = xor_u32<2>(__builtin_amdgcn_perm(y, x, t.send2));   // 2 x 2: bytes
  x = __builtin_amdgcn_perm(r, x, t.keep2x);
  y = __builtin_amdgcn_perm(r, y, t.keep2y);
  // 1 x 1: nibbles; the even lane sends its high nibbles, the odd its low ones
  r = xor_u32<1>(((x >> t.shl1) & 0x0F0F0F0Fu) | ((y << t.shr1) & 0xF0F0F0F0u));
  lo = (x & t.mask1) | ((r << t.shl1) & ~t.mask1);
  hi = (y & t.mask1) | ((r >> t.shr1) & ~t.mask1);
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
