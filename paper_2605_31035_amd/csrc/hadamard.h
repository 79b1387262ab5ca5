// Block-diagonal (random) Hadamard transform of bf16 data along K, exact
// then rounded once to bf16 (the rotation the paper applies before MixFP4
// quantization: the RHT of the training recipe, Sec. 3.2 / Fig. 7, and the
// "+RHT" rows of Sec. 4.2):
//   y[c b + j] = sum_i s_i x[c b + i] H_b[i, j] / sqrt(b),
// H_b the Sylvester matrix ((-1)^popcount(i & j)), s a vector of b signs.
//
// Layout: a lane holds one 16-element quantization block, so a Hadamard
// block of b = 16 L elements spans L consecutive lanes (L = 1..16, within
// one DPP row).  The fast Walsh-Hadamard butterflies run in fp64: four
// stages inside the lane, then log2 L stages across lanes through DPP lane
// exchanges (xor 1, 2: quad permutes; xor 4: half-row mirror then quad
// reverse; xor 8: row rotate by 8).
//
// Exactness: a bf16 value is a multiple of 2^(e-7) below 2^(e+1), so a block
// sum of b of them is exact in fp64 when the nonzero inputs of the block span
// at most 2^(45 - log2 b) in magnitude (2^37 for b = 256).  Then the sum S is
// exact, S / sqrt(b) is exact for b a power of 4 and within 2^-52 (relative)
// otherwise, and the result is rounded to bf16 once: to fp32 with round to
// odd (which keeps the correct final rounding, fp32 having 16 more bits),
// then to bf16 with ties to even.  For b = 2 * 4^m, a value whose fp32 image
// sits on a bf16 rounding midpoint is settled exactly: y > M iff
// S^2 > b M^2, with S^2 held exactly as p + e (fma) and p - b M^2 exact
// (Sterbenz).  An exactly zero result is +0.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "internal.h"
#include "lanes.h"

namespace mixfp4 {

// One butterfly stage across lanes: the lane with bit kX clear keeps
// own + partner, the other partner - own (fma with +-1: one rounding, exact
// whenever the sum is).
template <int kX>
__device__ __forceinline__ void cross_stage(double (&v)[16], int lane) {
  const double sg = (lane & kX) ? -1.0 : 1.0;
#pragma unroll
  for (int j = 0; j < 16; ++j) v[j] = __builtin_fma(v[j], sg, xor_f64<kX>(v[j]));
}

// Round y = S * scale to bf16 (see the header comment); returns the bits.
__device__ __forceinline__ uint32_t round_to_bf16(double S, const HadamardParams& hp) {
  const double y = __builtin_fma(S, hp.scale, 0.0);   // S * scale, and -0 -> +0
  const float f = (float)y;
  uint32_t fb = __float_as_uint(f);
  if (hp.odd && (fb & 0xFFFFu) - 0x7FFFu <= 2u) {
    // fp32 image within an ulp of the bf16 midpoint M: decide y > M exactly
    const uint32_t upper = fb & 0xFFFF0000u;
    const double M = (double)__uint_as_float((upper & 0x7FFFFFFFu) | 0x8000u);
    const double p = S * S;
    const double e = __builtin_fma(S, S, -p);
    const double diff = (p - M * M * hp.b) + e;
    return (upper >> 16) + (diff > 0.0 ? 1u : 0u);
  }
  const double back = (double)f;
  if (__builtin_fabs(back) > __builtin_fabs(y)) fb -= 1u;   // truncate toward zero
  if (back != y) fb |= 1u;                                  // round to odd
  return (fb + 0x7FFFu + ((fb >> 16) & 1u)) >> 16;
}

// Per-thread xor masks flipping the bf16 sign bits of the 16 elements of a
// lane at position `pos` within its Hadamard block (pos = lane % L).
struct SignMasks {
  uint32_t m[8];
};

__device__ __forceinline__ SignMasks load_sign_masks(const HadamardParams& hp, int pos) {
  SignMasks s;
#pragma unroll
  for (int i = 0; i < 8; ++i) s.m[i] = 0u;
  if (hp.signs) {
    const int8_t* p = hp.signs + 16 * pos;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const uint32_t a = (uint32_t)(uint8_t)p[2 * i] >> 7, b = (uint32_t)(uint8_t)p[2 * i + 1] >> 7;
      s.m[i] = (a << 15) | (b << 31);
    }
  }
  return s;
}

// Rotate the lane's 16 bf16 values (v0: elements 0-7, v1: 8-15) in place.
// Every lane of a Hadamard block must be active.
__device__ __forceinline__ void hadamard_rotate(uint4& v0, uint4& v1, const SignMasks& sm,
                                                const HadamardParams& hp) {
  const uint32_t w[8] = {v0.x ^ sm.m[0], v0.y ^ sm.m[1], v0.z ^ sm.m[2], v0.w ^ sm.m[3],
                         v1.x ^ sm.m[4], v1.y ^ sm.m[5], v1.z ^ sm.m[6], v1.w ^ sm.m[7]};
  double v[16];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    v[2 * i] = (double)__uint_as_float(w[i] << 16);
    v[2 * i + 1] = (double)__uint_as_float(w[i] & 0xFFFF0000u);
  }
#pragma unroll
  for (int h = 1; h < 16; h <<= 1) {
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      if (j & h) continue;
      const double a = v[j], c = v[j + h];
      v[j] = a + c;
      v[j + h] = a - c;
    }
  }
  const int lane = (int)(threadIdx.x & 63u);
  if (hp.lanes_log2 >= 1) cross_stage<1>(v, lane);
  if (hp.lanes_log2 >= 2) cross_stage<2>(v, lane);
  if (hp.lanes_log2 >= 3) cross_stage<4>(v, lane);
  if (hp.lanes_log2 >= 4) cross_stage<8>(v, lane);
  uint32_t o[8];
#pragma unroll
  for (int i = 0; i < 8; ++i)
    o[i] = round_to_bf16(v[2 * i], hp) | (round_to_bf16(v[2 * i + 1], hp) << 16);
  v0 = make_uint4(o[0], o[1], o[2], o[3]);
  v1 = make_uint4(o[4], o[5], o[6], o[7]);
}

}  // namespace mixfp4
