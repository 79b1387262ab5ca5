// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel Random Numbers: As
// Easy as 1, 2, 3", SC 2011): a counter-based generator, so every 16-element
// block draws its own random bits from its index with no state.
//
// One round maps counter (c0, c1, c2, c3) under key (k0, k1) to
//   (hi(M1 c2) ^ c1 ^ k0, lo(M1 c2), hi(M0 c0) ^ c3 ^ k1, lo(M0 c0))
// with the 64-bit products of M0 = 0xD2511F53 and M1 = 0xCD9E8D57; the key
// advances by (0x9E3779B9, 0xBB67AE85) between rounds; ten rounds.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "internal.h"

namespace mixfp4 {

__device__ __forceinline__ uint4 philox4x32_10(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3,
                                               uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint64_t p0 = (uint64_t)0xD2511F53u * c0;
    const uint64_t p1 = (uint64_t)0xCD9E8D57u * c2;
    const uint32_t n0 = (uint32_t)(p1 >> 32) ^ c1 ^ k0;
    const uint32_t n2 = (uint32_t)(p0 >> 32) ^ c3 ^ k1;
    c1 = (uint32_t)p1;
    c3 = (uint32_t)p0;
    c0 = n0;
    c2 = n2;
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  return make_uint4(c0, c1, c2, c3);
}

// Stochastic-rounding draws (SrParams): key = the 64-bit seed, counter =
// (block index, 64-bit offset).  Element j of the block takes byte j % 4 of
// word j / 4.
__device__ __forceinline__ uint4 block_draws(int64_t g, const SrParams& p) {
  return philox4x32_10((uint32_t)g, (uint32_t)((uint64_t)g >> 32), p.off_lo, p.off_hi, p.seed_lo,
                       p.seed_hi);
}

}  // namespace mixfp4
