// Decoding MixFP4 elements to exact fp16 values s8 * v (Sec. 3.3, App. B.5):
// shared by the GEMM kernels and the operand decode pass.
//
// Every unscaled unified value (E2M1 {0,.5,1,1.5,2,3,4,6}, E1M2 x2 = INT4
// {0..7}) has a zero low byte in fp16, so the 8 magnitudes of a codebook are
// one 8-byte constant of high bytes.  A code dword (8 nibbles) decodes with
// v_perm_b32 byte lookups into that constant (picked by T), the nibble sign
// bit is OR-ed in, two more perms place the bytes as fp16 pairs, and
// v_pk_mul_f16 multiplies by s8.  s8 has at most 4 significant bits and v at
// most 3, so s8 * v has at most 7 and lies in [2^-10, 3136]: exact in fp16.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mixfp4 {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));

// High bytes of the fp16 values of magnitudes 0..7 (bytes 0-3 in the low
// dword): E2M1 {0, .5, 1, 1.5, 2, 3, 4, 6} and E1M2 x2 = INT4 {0, ..., 7}.
constexpr uint32_t kE2M1Lo = 0x3E3C3800u, kE2M1Hi = 0x46444240u;
constexpr uint32_t kInt4Lo = 0x42403C00u, kInt4Hi = 0x47464544u;

// Decoding constants of one block from its scale byte: the codebook's high
// bytes (by T = bit 7) and s8 = E4M3(bits 6:0) as an fp16 pair.  E4M3 ->
// fp32 is exact (hardware converter) and so is fp32 -> fp16 (4 significant
// bits, 2^-9 .. 448), whatever the rounding mode of the packing conversion.
struct BlockDec {
  uint32_t lo, hi;
  f16x2 s8;
};
__device__ __forceinline__ BlockDec block_dec(uint32_t sb) {
  BlockDec d;
  const bool t1 = (sb & 0x80u) != 0;
  d.lo = t1 ? kInt4Lo : kE2M1Lo;
  d.hi = t1 ? kInt4Hi : kE2M1Hi;
  const float s8 = __builtin_amdgcn_cvt_f32_fp8((int)(sb & 0x7Fu), 0);
  d.s8 = __builtin_bit_cast(f16x2, __builtin_amdgcn_cvt_pkrtz(s8, s8));
  return d;
}

// The four blocks of a scale dword (byte b = block b): T selects each
// block's codebook; E4M3 -> fp16 by the hardware converter at scale 1, which
// is exact (every E4M3 value is an fp16 normal; the converter applies only
// the exponent of its fp32 scale, here 2^0).  Two conversions serve four
// blocks, against three instructions per block for block_dec.
__device__ __forceinline__ void block_dec4(uint32_t sw, BlockDec (&d)[4]) {
  const uint32_t m = sw & 0x7F7F7F7Fu;
  const f16x2 s01 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(m, 1.0f, false);
  const f16x2 s23 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(m, 1.0f, true);
#pragma unroll
  for (int b = 0; b < 4; ++b) {
    const bool t1 = ((sw >> (8 * b + 7)) & 1u) != 0;
    d[b].lo = t1 ? kInt4Lo : kE2M1Lo;
    d[b].hi = t1 ? kInt4Hi : kE2M1Hi;
    const _Float16 s = b == 0 ? s01.x : b == 1 ? s01.y : b == 2 ? s23.x : s23.y;
    d[b].s8 = f16x2{s, s};
  }
}

__device__ __forceinline__ uint32_t scale_pair(uint32_t v, f16x2 s8) {
  return __builtin_bit_cast(uint32_t, __builtin_bit_cast(f16x2, v) * s8);
}

// Decode one code dword (8 nibbles, element 2j in the low nibble of byte j)
// of a block into 8 fp16 s8 * v in the order [e0 e2 e4 e6 e1 e3 e5 e7].
__device__ __forceinline__ uint4 decode8(uint32_t c, const BlockDec& d) {
  const uint32_t me = c & 0x07070707u;
  const uint32_t mo = (c >> 4) & 0x07070707u;
  const uint32_t he = __builtin_amdgcn_perm(d.hi, d.lo, me) | ((c << 4) & 0x80808080u);
  const uint32_t ho = __builtin_amdgcn_perm(d.hi, d.lo, mo) | (c & 0x80808080u);
  // selector byte 0x0C yields a zero byte: fp16 pairs {0, hi_a, 0, hi_b}
  uint4 r;
  r.x = scale_pair(__builtin_amdgcn_perm(he, he, 0x010C000Cu), d.s8);   // e0 e2
  r.y = scale_pair(__builtin_amdgcn_perm(he, he, 0x030C020Cu), d.s8);   // e4 e6
  r.z = scale_pair(__builtin_amdgcn_perm(ho, ho, 0x010C000Cu), d.s8);   // e1 e3
  r.w = scale_pair(__builtin_amdgcn_perm(ho, ho, 0x030C020Cu), d.s8);   // e5 e7
  return r;
}

}  // namespace mixfp4
