// Device-side bit-level helpers for the MixFP4 number formats.
//
// E4M3 is OCP E4M3FN (bias 7, max 448 = code 0x7E, no Inf, 0x7F = NaN); the
// paper names 448 and 384 as E4M3 values (Algorithm 1).  E2M1 magnitudes are
// {0,.5,1,1.5,2,3,4,6} and E1M2 magnitudes after the x2 remap are {0,...,7}
// (Sec. 3.1 Table 1, App. B.2).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mixfp4 {

// bf16 bit pattern (low / high half of a dword) -> fp32, exact.
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// Value of a 7-bit E4M3 magnitude code (bit 7 must already be cleared).
__device__ __forceinline__ float e4m3_value(uint32_t c) {
  const uint32_t e = c >> 3, m = c & 7u;
  // normal: 2^(e-7) * (1 + m/8) -> fp32 exponent field e + 120, mantissa m << 20
  const float normal = __uint_as_float(((e + 120u) << 23) | (m << 20));
  const float sub = (float)m * 0x1p-9f;   // subnormal: m * 2^-9
  return e ? normal : sub;
}

// Round v >= 0 (finite fp32) to the nearest E4M3 value, ties to the even
// code, saturating at 448; returns the 7-bit magnitude code.  Branch-free.
__device__ __forceinline__ uint32_t e4m3_code(float v) {
  uint32_t b = __float_as_uint(v);
  b += 0x7FFFFu + ((b >> 20) & 1u);                      // RNE to 3 mantissa bits
  const uint32_t normal = (b >> 20) - (120u << 3);        // rebias exponent 127 -> 7
  const uint32_t sub = (uint32_t)rintf(v * 512.0f);       // m * 2^-9, m in 0..8
  const uint32_t c = v < 0x1p-6f ? sub : normal;
  return (v < 448.0f && c < 0x7Eu) ? c : 0x7Eu;
}

// E2M1 magnitude of a 3-bit code (App. B.2: e = p2p1, m = p0, bias 1).
__device__ __forceinline__ float e2m1_value(uint32_t c) {
  const float normal = __uint_as_float((((c >> 1) + 126u) << 23) | ((c & 1u) << 22));
  return c >= 2u ? normal : 0.5f * (float)c;
}

}  // namespace mixfp4
