// Per-block device code of the MixFP4 quantizer (Algorithm 1), shared by the
// 1D kernels (one lane per 16-element block) and the 2D kernels (16 lanes per
// 16 x 16 tile).  See quantize.hip for the numerics of each step.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "formats.h"
#include "internal.h"
#include "lanes.h"

namespace mixfp4 {

// max(|X|) bits over 8 bf16 in a 16-byte vector
__device__ __forceinline__ uint32_t absmax8(uint4 v) {
  const uint32_t m0 = max(max(v.x & 0x7FFFu, (v.x >> 16) & 0x7FFFu), max(v.y & 0x7FFFu, (v.y >> 16) & 0x7FFFu));
  const uint32_t m1 = max(max(v.z & 0x7FFFu, (v.z >> 16) & 0x7FFFu), max(v.w & 0x7FFFu, (v.w >> 16) & 0x7FFFu));
  return max(m0, m1);
}

__device__ __forceinline__ float tensor_scale_of(uint32_t amax_bf16_bits) {
  const float amax = __uint_as_float(amax_bf16_bits << 16);
  return amax > 0.0f ? amax / 2688.0f : 1.0f;       // Algorithm 1, first step
}

// A block-scale divisor s with its two-term reciprocal: rh = 1 / s rounded
// toward zero and rl = fl32((1 - rh s) / s) >= 0 (the residual 1 - rh s is
// exact: one fma).  rh + rl equals 1 / s to about 2^-48 relative.
struct alignas(16) ScaleRecip {
  float s, rh, rl, unused;
};

__device__ __forceinline__ ScaleRecip scale_recip(float s) {
  float rh = __fdiv_rn(1.0f, s);
  float e = __builtin_fmaf(-rh, s, 1.0f);
  if (e < 0.0f) {
    rh = __uint_as_float(__float_as_uint(rh) - 1u);
    e = __builtin_fmaf(-rh, s, 1.0f);
  }
  return ScaleRecip{s, rh, __fdiv_rn(e, s), 0.0f};
}

// The divisor and two-term reciprocal of every 7-bit E4M3 code (all zero for
// the zero scale and the NaN code), built by the first 128 threads; the
// caller synchronizes before use.
__device__ __forceinline__ void fill_scale_table(ScaleRecip* tab) {
  if (threadIdx.x < 128) {
    const bool ok = threadIdx.x > 0 && threadIdx.x < 127;
    tab[threadIdx.x] = ok ? scale_recip(e4m3_value(threadIdx.x)) : ScaleRecip{0.0f, 0.0f, 0.0f, 0.0f};
  }
}

typedef float f32x2 __attribute__((ext_vector_type(2)));

// fl32(a / s) given r = fl32(1 / s): q0 = a r is within an ulp of the
// quotient, the fma residual q0 s - a is exact, and q0 minus residual * r is
// the correctly rounded quotient (Markstein's division step).  Verified
// exhaustively for every fp32 a against every divisor with at most 4
// significant bits, and for every bf16 a against every fp32 divisor, with all
// three results in the normal range.  The residual is taken as q0 s - a
// (not a - q0 s) so that a zero a keeps its sign: both fmas then add two
// zeros of the sign of a.  A zero divisor with r = 0 returns a zero with the
// sign of a.
__device__ __forceinline__ float div_rn(float a, float s, float r) {
  const float q0 = a * r;
  return __builtin_fmaf(-__builtin_fmaf(q0, s, -a), r, q0);
}

// fl32(a / s) for a divisor s with at most 4 significant bits (the E4M3
// block scales, 6 and 7) from its two-term reciprocal: a rh + fl32(a rl) is
// within about 2^-47 of a / s, while a / s with a in fp32 lies at least
// 2^-29 (relative) away from every rounding boundary of fp32, so the one
// rounding of the fma is the correctly rounded quotient.  Verified
// exhaustively for every fp32 a against every such divisor, results and
// a * rl in the normal range; both addends carry the sign of a (rl >= 0), so
// zeros keep their sign, also with the zero scale (rh = rl = 0).
__device__ __forceinline__ float div_scale(float a, float rh, float rl) {
  return __builtin_fmaf(a, rh, a * rl);
}

typedef short s16x2 __attribute__((ext_vector_type(2)));

// x = fl32(X / s32) for the 16 elements of a block, signed (Algorithm 1, FP8
// domain).  X is first multiplied by xmul (a power of two, exact) when
// kScaled, and divided by sx = s32 * xmul with rx = fl32(1 / sx).
template <bool kScaled>
__device__ __forceinline__ void to_fp8_domain(uint4 v0, uint4 v1, float xmul, float sx, float rx,
                                              float (&xs)[16]) {
  const uint32_t w[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const float lo = kScaled ? bf16_lo(w[i]) * xmul : bf16_lo(w[i]);
    const float hi = kScaled ? bf16_hi(w[i]) * xmul : bf16_hi(w[i]);
    xs[2 * i] = div_rn(lo, sx, rx);
    xs[2 * i + 1] = div_rn(hi, sx, rx);
  }
}

// x = fl32(X / s32) for the 16 elements of a block from the two-term
// reciprocal of s32 (div_scale).  s32 has 24 significant bits, so this is
// exact only for tensor scales that pass the per-launch check in
// quantize_kernel: every one of the 128 bf16 mantissas divided this way
// gives Markstein's (exact) quotient.  Scaling X by a power of two scales
// both steps exactly while x and X * rl stay normal, which covers every x
// at or above 2^-78; smaller elements receive zero codes with X's sign (kept:
// rl >= 0) whatever their exact value, and contribute nothing to the errors.
__device__ __forceinline__ void to_fp8_domain_two_term(uint4 v0, uint4 v1, float rh, float rl,
                                                       float (&xs)[16]) {
  const uint32_t w[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    xs[2 * i] = div_scale(bf16_lo(w[i]), rh, rl);
    xs[2 * i + 1] = div_scale(bf16_hi(w[i]), rh, rl);
  }
}

// Elements J, J+1 (J even) of a block, E2M1 branch: y = fl32(x / s_F)
// rounded by the gfx950 FP4 converter (scale 1: nearest, ties to the even
// code, saturating at 6, sign kept) into nibble pair (J%8)/2 of pf[J/8].
template <int J>
__device__ __forceinline__ void encode_f_pair(const float (&xs)[16], const ScaleRecip& f,
                                              uint32_t (&pf)[2]) {
  const float yf0 = div_scale(xs[J], f.rh, f.rl), yf1 = div_scale(xs[J + 1], f.rh, f.rl);
  pf[J >> 3] = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(pf[J >> 3], yf0, yf1, 1.0f, (J & 7) >> 1);
}

// Elements J, J+1 (J even), E1M2 (x2 = INT4) branch: q = rint(fl32(|x| /
// s_I)) (round half to even), an exact small integer, inserted as a byte:
// element J into byte (J%8)/2 of pe[J/8], element J+1 into the same byte of
// po[J/8] (the nibbles are interleaved afterwards).  With kErr, ai[J/2 % 2]
// += |x| * q.
template <int J, bool kErr>
__device__ __forceinline__ void encode_i_pair(const float (&xs)[16], const ScaleRecip& i,
                                              uint32_t (&pe)[2], uint32_t (&po)[2],
                                              float (&ai)[2]) {
  const float a0 = fabsf(xs[J]), a1 = fabsf(xs[J + 1]);
  const float q0 = __builtin_rintf(div_scale(a0, i.rh, i.rl));
  const float q1 = __builtin_rintf(div_scale(a1, i.rh, i.rl));
  if (kErr) {
    float& acc = ai[(J >> 1) & 1];
    acc = __builtin_fmaf(a0, q0, acc);
    acc = __builtin_fmaf(a1, q1, acc);
  }
  pe[J >> 3] = __builtin_amdgcn_cvt_pk_u8_f32(q0, (J & 7) >> 1, pe[J >> 3]);
  po[J >> 3] = __builtin_amdgcn_cvt_pk_u8_f32(q1, (J & 7) >> 1, po[J >> 3]);
}

typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));

// E2M1 error sums of elements J, J+1 from the decoded codes, in two chains:
//   af += x * q_F (same signs, so every term is >= 0),  bf += q_F^2.
// The pair is decoded to two fp16 values (exact: E2M1 magnitudes have at
// most two significant bits); x * q_F + af is one fp32 fma with the fp16
// operand widened exactly (v_fma_mix), and q_F^2 summed by one dot2: its
// terms are multiples of 1/4 below 2^6, so the sum is exact in fp32.
template <int J>
__device__ __forceinline__ void error_pair(const float (&xs)[16], const uint32_t (&pf)[2],
                                           float (&af)[2], float (&bf)[2]) {
  const f16x2 qf = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(pf[J >> 3], 1.0f, (J & 7) >> 1);
  constexpr int c = (J >> 1) & 1;
  af[c] = __builtin_fmaf(xs[J], (float)qf.x, af[c]);
  af[c] = __builtin_fmaf(xs[J + 1], (float)qf.y, af[c]);
  bf[c] = __builtin_amdgcn_fdot2(qf, qf, bf[c], false);
}

// Exact contribution of elements J, J+1 to Err_E2M1 - Err_E1M2 in fp64:
//   (D_I - D_F) (2|x| - D_F - D_I),  D_T = s_T q_T.
// D_F, D_I are exact fp32 products; an element contributes only when
// D_I != D_F, and then |x| >= min(s_F, s_I) / 4, so every term and every
// partial sum of a block is exact in fp64 and the total is exact.
template <int J>
__device__ __forceinline__ void exact_pair(const float (&xs)[16], const uint32_t (&pf)[2],
                                           const uint32_t (&pi)[2], float sf, float si, double& d) {
  const f32x2 qf = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(pf[J >> 3], 1.0f, (J & 7) >> 1);
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const double ax = (double)fabsf(xs[J + h]);
    const double df = (double)(fabsf(h ? qf.y : qf.x) * sf);
    const uint32_t ci = (pi[(J + h) >> 3] >> (4 * ((J + h) & 7))) & 7u;
    const double di = (double)((float)ci * si);
    d += (di - df) * ((2.0 * ax - df) - di);
  }
}

// Nibbles of v (eight 4-bit codes) with a nonzero 3-bit magnitude, as one
// bit per nibble (bit 4k for nibble k).
__device__ __forceinline__ uint32_t nonzero_nibbles(uint32_t v) {
  return (v | (v >> 1) | (v >> 2)) & 0x11111111u;
}

// The 3-bit magnitude of the only nonzero code among two words (the others
// are zero).
__device__ __forceinline__ uint32_t only_code(uint32_t w0, uint32_t w1) {
  uint32_t w = (w0 | w1) & 0x77777777u;
  w |= w >> 16;
  w |= w >> 8;
  w |= w >> 4;
  return w & 7u;
}

// Err_A - Err_B of a block in which at most one element has a nonzero code
// under either candidate A (E2M1 codes pa) or B (E1M2 codes pb, or E2M1
// codes when kFF): every other element quantizes to 0 in both and adds
// (|x| - 0)^2 to both errors, and the nonzero one is the block maximum
// (|x| = bm: the element at bm always gets a nonzero code under a nonzero
// scale).  The single term (D_B - D_A)(2 bm - D_A - D_B) is exact in fp64
// (D_A, D_B have at most 7 significant bits).  In blocks dominated by one
// element this is the common way for both candidates to tie, and it costs
// a few instructions instead of the 16-element fp64 sum.
template <bool kFF>
__device__ __forceinline__ double single_element_delta(const uint32_t (&pa)[2],
                                                       const uint32_t (&pb)[2], float sa,
                                                       float sb, float bm) {
  const uint32_t ca = only_code(pa[0], pa[1]), cb = only_code(pb[0], pb[1]);
  const double da = (double)(e2m1_value(ca) * sa);
  const double db = (double)((kFF ? e2m1_value(cb) : (float)cb) * sb);
  return (db - da) * ((2.0 * (double)bm - da) - db);
}

// Number of elements of a block with a nonzero code under A or B.
__device__ __forceinline__ uint32_t nonzero_elements(const uint32_t (&pa)[2],
                                                     const uint32_t (&pb)[2]) {
  return __builtin_popcount(nonzero_nibbles(pa[0] & 0x77777777u) | nonzero_nibbles(pb[0] & 0x77777777u)) +
         __builtin_popcount(nonzero_nibbles(pa[1] & 0x77777777u) | nonzero_nibbles(pb[1] & 0x77777777u));
}

// Format modes: MixFP4 selection (Algorithm 1), or one branch for every
// block (E2M1 = NVFP4, E1M2 = INT4); T records the branch either way.
// kFourSix: the candidate set {E2M1 under max/6, E2M1 under max/4} (the 4/6
// baseline the paper compares against), T = 0.
constexpr int kSelect = 0, kForceE2M1 = 1, kForceE1M2 = 2, kFourSix = 3;

// Exact contribution of elements J, J+1 to Err(max/6) - Err(max/4) in fp64,
// both branches E2M1: (D_4 - D_6) (2|x| - D_6 - D_4), exact for the same
// reasons as exact_pair.
template <int J>
__device__ __forceinline__ void exact_pair_ff(const float (&xs)[16], const uint32_t (&p6)[2],
                                              const uint32_t (&p4)[2], float s6, float s4,
                                              double& d) {
  const f32x2 q6 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(p6[J >> 3], 1.0f, (J & 7) >> 1);
  const f32x2 q4 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(p4[J >> 3], 1.0f, (J & 7) >> 1);
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const double ax = (double)fabsf(xs[J + h]);
    const double d6 = (double)(fabsf(h ? q6.y : q6.x) * s6);
    const double d4 = (double)(fabsf(h ? q4.y : q4.x) * s4);
    d += (d4 - d6) * ((2.0 * ax - d6) - d4);
  }
}

// E1M2 codes of the 16 elements with saturation at 7 (a subnormal or
// saturated s_I admits codes above 7; rare path): codes into pi, with kErr
// also sum |x| q_I into ai.
template <bool kErr>
__device__ __forceinline__ void encode_i_saturated(const float (&xs)[16], const ScaleRecip& i,
                                                   uint32_t (&pi)[2], float (&ai)[2]) {
  pi[0] = pi[1] = 0u;
  ai[0] = ai[1] = 0.0f;
  for (int j = 0; j < 16; ++j) {
    const float q = fminf(rintf(div_scale(fabsf(xs[j]), i.rh, i.rl)), 7.0f);
    if (kErr) ai[j & 1] = __builtin_fmaf(fabsf(xs[j]), q, ai[j & 1]);
    pi[j >> 3] |= (uint32_t)q << (4 * (j & 7));
  }
}

// Stochastic rounding (App. D) of the block onto the chosen grid: y =
// fl32(|x| / s) (the same quotient round-to-nearest takes), and between its
// grid neighbours lo <= y < lo + d the rule round(y + (eps - 1/2) d) with
// eps = (u + 1/2) / 256, u the element's draw (255 - u for a negative X,
// which turns App. D's signed rule into this magnitude rule).  In units of
// the local spacing, w = 512 (y - lo) / d is exact in fp32 and the rule
// reads: up iff w > 511 - 2u, ties (w == 511 - 2u) to the even code.  y at
// or above the largest magnitude clamps to code 7.  E2M1 spacing: 1/2 below
// 2, 1 below 4, 2 up to 6; E1M2 (x2): 1 everywhere.
__device__ __forceinline__ uint2 sr_codes(const float (&xs)[16], const ScaleRecip& sc, bool int4,
                                          uint4 rnd) {
  const uint32_t words[4] = {rnd.x, rnd.y, rnd.z, rnd.w};
  // Branch-free lattice choice (a per-lane select, not control flow): E2M1
  // spacing 2^(t-1) with t = clamp(exponent of y, 0, 2), so z = y 2^(1-t)
  // exactly and the lattice point below y is code floor(z) + 2t; E1M2 (x2)
  // spacing 1, z = y, code floor(z).
  const int keep = int4 ? 0 : -1;                    // all ones on the E2M1 lattice
  const float top = int4 ? 7.0f : 6.0f;
  uint32_t o[2] = {0u, 0u};
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    const uint32_t xb = __float_as_uint(xs[j]);
    const uint32_t neg = xb >> 31;
    const float y = div_scale(__uint_as_float(xb & 0x7FFFFFFFu), sc.rh, sc.rl);
    const int e = (int)(__float_as_uint(y) >> 23) - 127;
    const int t = min(max(e, 0), 2);
    const float z = __builtin_ldexpf(y, (1 - t) & keep);
    const float lat = floorf(z);
    const float w = (z - lat) * 512.0f;
    const uint32_t u = ((words[j >> 2] >> (8 * (j & 3))) & 0xFFu) ^ (0xFFu & (0u - neg));
    const float thr = (float)(511 - 2 * (int)u);
    uint32_t code = (uint32_t)lat + (uint32_t)((2 * t) & keep);
    code += ((uint32_t)(w > thr) | ((uint32_t)(w == thr) & code)) & 1u;
    code = y >= top ? 7u : code;
    o[j >> 3] |= (code | (neg << 3)) << (4 * (j & 7));
  }
  return make_uint2(o[0], o[1]);
}

// 4/6: both candidates are E2M1, under E4M3(bm/6) and E4M3(bm/4) (bm/4 is
// exact in fp32); the squared errors are compared as in Algorithm 1's
// selection (bounded fp32 estimate, exact fp64 sum inside the bound); /4 is
// kept only where its error is strictly smaller.  T = 0.
template <bool kSR, bool kTile>
__device__ __forceinline__ void quantize_four_six(const float (&xs)[16], float bm, float bm_lane,
                                                  const ScaleRecip* __restrict__ tab, uint2& out,
                                                  uint32_t& scale_byte, uint4 rnd) {
  const ScaleRecip d6 = scale_recip(6.0f);
  const float cand6 = fminf(div_scale(bm, d6.rh, d6.rl), 448.0f);
  const float cand4 = fminf(bm * 0.25f, 448.0f);
  const s16x2 sc = __builtin_amdgcn_cvt_scalef32_pk_fp8_f32(s16x2{0, 0}, cand6, cand4, 1.0f, false);
  const uint32_t scw = __builtin_bit_cast(uint32_t, sc);
  const uint32_t c6 = scw & 0x7Fu, c4 = (scw >> 8) & 0x7Fu;
  const ScaleRecip e6 = tab[c6], e4 = tab[c4];
  const float s6 = e6.s, s4 = e4.s;
  uint32_t p6[2] = {0u, 0u}, p4[2] = {0u, 0u};
  float a6[2] = {0.0f, 0.0f}, b6[2] = {0.0f, 0.0f}, a4[2] = {0.0f, 0.0f}, b4[2] = {0.0f, 0.0f};
#define MIXFP4_PAIR(J)                    \
  encode_f_pair<J>(xs, e6, p6);           \
  encode_f_pair<J>(xs, e4, p4);           \
  error_pair<J>(xs, p6, a6, b6);          \
  error_pair<J>(xs, p4, a4, b4);
  MIXFP4_PAIR(0) MIXFP4_PAIR(2) MIXFP4_PAIR(4) MIXFP4_PAIR(6)
  MIXFP4_PAIR(8) MIXFP4_PAIR(10) MIXFP4_PAIR(12) MIXFP4_PAIR(14)
#undef MIXFP4_PAIR
  float a6s = a6[0] + a6[1], b6s = b6[0] + b6[1], a4s = a4[0] + a4[1], b4s = b4[0] + b4[1];
  if constexpr (kTile) {
    a6s = row16_sum(a6s);
    b6s = row16_sum(b6s);
    a4s = row16_sum(a4s);
    b4s = row16_sum(b4s);
  }
  // Err6 - Err4 = (s6^2 b6 - s4^2 b4) + 2 (s4 a4 - s6 a6); same error bound
  // as the MixFP4 selection (both cross sums have non-negative terms).
  const float s62b = (s6 * s6) * b6s, s42b = (s4 * s4) * b4s;
  const float t6 = s6 * a6s, t4 = s4 * a4s;
  const float est = (s62b - s42b) + 2.0f * (t4 - t6);
  const float tau = kTile ? 0x1p-18f * (t6 + t4) + 0x1p-21f * (s62b + s42b)
                          : 0x1p-19f * (t6 + t4) + 0x1p-22f * (s62b + s42b);
  bool use4;
  uint32_t nz = 0;
  if (!(c6 != 0u && c4 != 0u && fabsf(est) > tau)) {
    nz = nonzero_elements(p6, p4);
    if constexpr (kTile) nz = row16_sum(nz);
  }
  if (c6 != 0u && c4 != 0u && fabsf(est) > tau) {
    use4 = est > 0.0f;
  } else if (nz <= 1u) {
    double d = single_element_delta<true>(p6, p4, s6, s4, bm_lane);
    if constexpr (kTile) d = row16_sum(d);
    use4 = d > 0.0;
  } else {
    double d = 0.0;
    exact_pair_ff<0>(xs, p6, p4, s6, s4, d);
    exact_pair_ff<2>(xs, p6, p4, s6, s4, d);
    exact_pair_ff<4>(xs, p6, p4, s6, s4, d);
    exact_pair_ff<6>(xs, p6, p4, s6, s4, d);
    exact_pair_ff<8>(xs, p6, p4, s6, s4, d);
    exact_pair_ff<10>(xs, p6, p4, s6, s4, d);
    exact_pair_ff<12>(xs, p6, p4, s6, s4, d);
    exact_pair_ff<14>(xs, p6, p4, s6, s4, d);
    if constexpr (kTile) d = row16_sum(d);
    use4 = d > 0.0;
  }
  if constexpr (kSR)
    out = sr_codes(xs, use4 ? e4 : e6, false, rnd);
  else
    out = use4 ? make_uint2(p4[0], p4[1]) : make_uint2(p6[0], p6[1]);
  scale_byte = use4 ? c4 : c6;
}

// Codes and scale byte of one block from x (Algorithm 1 after the tensor
// scale).  With kSR the chosen branch's codes are written by stochastic
// rounding with the draws in `rnd`; scales and the format choice stay those
// of round-to-nearest.
//
// kTile: the block is a 16 x 16 tile held by the 16 lanes of a DPP row (this
// lane's xs is one row of it).  The block maximum and the four error sums
// are then all-reduced over the row with butterflies, which leave identical
// values in every lane, so all 16 lanes take the same decision.
template <int kMode, bool kSR, bool kTile = false>
__device__ __forceinline__ void quantize_xs(const float (&xs)[16], const ScaleRecip* __restrict__ tab,
                                            uint2& out, uint32_t& scale_byte, uint4 rnd) {
  // fl32 rounding is monotonic, so bm is also fl32(max|X| / s32).
  float bm = 0.0f;
#pragma unroll
  for (int j = 0; j < 16; ++j) bm = fmaxf(bm, fabsf(xs[j]));
  const float bm_lane = bm;          // this lane's 16 elements (a tile row)
  if constexpr (kTile) bm = row16_max(bm);
  if constexpr (kMode == kFourSix) {
    quantize_four_six<kSR, kTile>(xs, bm, bm_lane, tab, out, scale_byte, rnd);
    return;
  }
  // Candidate block scales E4M3(bm/6), E4M3(bm/7): the exactly rounded
  // quotients, clamped at 448 (saturation), through the gfx950 E4M3
  // converter (scale 1: nearest, ties to the even code; checked against the
  // software rounding on every fp32 value in [0, 448]).
  const ScaleRecip d6 = scale_recip(6.0f), d7 = scale_recip(7.0f);
  const float cand6 = kMode == kForceE1M2 ? 0.0f : fminf(div_scale(bm, d6.rh, d6.rl), 448.0f);
  const float cand7 = kMode == kForceE2M1 ? 0.0f : fminf(div_scale(bm, d7.rh, d7.rl), 448.0f);
  const s16x2 sc = __builtin_amdgcn_cvt_scalef32_pk_fp8_f32(s16x2{0, 0}, cand6, cand7, 1.0f, false);
  const uint32_t scw = __builtin_bit_cast(uint32_t, sc);
  const uint32_t cf = scw & 0x7Fu, ci = (scw >> 8) & 0x7Fu;
  const ScaleRecip ef = tab[cf], ei = tab[ci];
  const float sf = ef.s, si = ei.s;

  uint32_t pf[2] = {0u, 0u}, pi[2] = {0u, 0u};
  float af[2] = {0.0f, 0.0f}, bf[2] = {0.0f, 0.0f}, ai[2] = {0.0f, 0.0f};
  if constexpr (kMode != kForceE1M2) {
    encode_f_pair<0>(xs, ef, pf);
    encode_f_pair<2>(xs, ef, pf);
    encode_f_pair<4>(xs, ef, pf);
    encode_f_pair<6>(xs, ef, pf);
    encode_f_pair<8>(xs, ef, pf);
    encode_f_pair<10>(xs, ef, pf);
    encode_f_pair<12>(xs, ef, pf);
    encode_f_pair<14>(xs, ef, pf);
  }
  if constexpr (kMode == kForceE2M1) {
    out = kSR ? sr_codes(xs, ef, false, rnd) : make_uint2(pf[0], pf[1]);
    scale_byte = cf;
    return;
  }
  constexpr bool kErr = kMode == kSelect;
  {
    uint32_t pe[2] = {0u, 0u}, po[2] = {0u, 0u};
    encode_i_pair<0, kErr>(xs, ei, pe, po, ai);
    encode_i_pair<2, kErr>(xs, ei, pe, po, ai);
    encode_i_pair<4, kErr>(xs, ei, pe, po, ai);
    encode_i_pair<6, kErr>(xs, ei, pe, po, ai);
    encode_i_pair<8, kErr>(xs, ei, pe, po, ai);
    encode_i_pair<10, kErr>(xs, ei, pe, po, ai);
    encode_i_pair<12, kErr>(xs, ei, pe, po, ai);
    encode_i_pair<14, kErr>(xs, ei, pe, po, ai);
    pi[0] = pe[0] | (po[0] << 4);
    pi[1] = pe[1] | (po[1] << 4);
  }
  // INT4 codes cannot exceed 7 when s_I is a normal E4M3 value below the
  // maximum (then max|x| / s_I < 7.47); other blocks redo the branch with
  // saturation (rare path).
  if (ci < 8u || ci >= 0x7Eu) encode_i_saturated<kErr>(xs, ei, pi, ai);
  if constexpr (kMode == kForceE1M2) {
    // sign of X into bit 3 of every nibble
    uint32_t sg[2] = {0u, 0u};
#pragma unroll
    for (int j = 0; j < 16; ++j) sg[j >> 3] |= (__float_as_uint(xs[j]) >> 31) << (4 * (j & 7) + 3);
    out = kSR ? sr_codes(xs, ei, true, rnd) : make_uint2(pi[0] | sg[0], pi[1] | sg[1]);
    scale_byte = 0x80u | ci;
    return;
  }
  error_pair<0>(xs, pf, af, bf);
  error_pair<2>(xs, pf, af, bf);
  error_pair<4>(xs, pf, af, bf);
  error_pair<6>(xs, pf, af, bf);
  error_pair<8>(xs, pf, af, bf);
  error_pair<10>(xs, pf, af, bf);
  error_pair<12>(xs, pf, af, bf);
  error_pair<14>(xs, pf, af, bf);
  uint32_t bi = __builtin_amdgcn_udot8(pi[0], pi[0], __builtin_amdgcn_udot8(pi[1], pi[1], 0u, false),
                                       false);
  // Err_F - Err_I with Err_T = sum x^2 - 2 s_T sum |x| q_T + s_T^2 sum q_T^2
  // (the sum of x^2 cancels):  est = (sf^2 bf - si^2 bi) + 2 (si ai - sf af).
  // bf and bi are exact (multiples of 1/4, integers) and so are sf^2 bf and
  // si^2 bi (at most 20 significant bits).  af and ai are sums of
  // non-negative terms in two chains of 8 fmas plus one add: relative error
  // at most 9u (u = 2^-24); with the four roundings that follow, |est - Err_F
  // + Err_I| <= 24u (tf + ti) + 2u (sf^2 bf + si^2 bi) to first order, which
  // tau bounds with margin.  Products x q with q != 0 are at least 2^-12
  // (|x| >= s/4 >= 2^-11), so nothing underflows.  Inside tau, or when
  // either candidate scale is zero (that branch's error is then sum x^2,
  // which the estimate does not model), the exact fp64 sum decides.
  //
  // For a tile (kTile) the sums run over 256 elements: bf (multiples of 1/4
  // up to 9216) and bi stay exact, s_F^2 bf has at most 24 significant bits,
  // and af, ai gain four butterfly additions (relative error at most 13u), so
  // the bound becomes 30u (tf + ti) + 2u (...), which the doubled tau covers.
  float afs = af[0] + af[1], ais = ai[0] + ai[1], bfs = bf[0] + bf[1];
  if constexpr (kTile) {
    afs = row16_sum(afs);
    ais = row16_sum(ais);
    bfs = row16_sum(bfs);
    bi = row16_sum(bi);
  }
  const float sf2b = (sf * sf) * bfs, si2b = (si * si) * (float)bi;
  const float tf = sf * afs, ti = si * ais;
  const float est = (sf2b - si2b) + 2.0f * (ti - tf);
  const float tau = kTile ? 0x1p-18f * (tf + ti) + 0x1p-21f * (sf2b + si2b)
                          : 0x1p-19f * (tf + ti) + 0x1p-22f * (sf2b + si2b);
  bool t1;
  uint32_t nz = 0;
  if (!(cf != 0u && ci != 0u && fabsf(est) > tau)) {
    nz = nonzero_elements(pf, pi);
    if constexpr (kTile) nz = row16_sum(nz);
  }
  if (cf != 0u && ci != 0u && fabsf(est) > tau) {
    t1 = !(est < 0.0f);
  } else if (nz <= 1u) {
    double d = single_element_delta<false>(pf, pi, sf, si, bm_lane);
    if constexpr (kTile) d = row16_sum(d);     // one nonzero term in the tile: exact
    t1 = !(d < 0.0);
  } else {
    double d = 0.0;
    exact_pair<0>(xs, pf, pi, sf, si, d);
    exact_pair<2>(xs, pf, pi, sf, si, d);
    exact_pair<4>(xs, pf, pi, sf, si, d);
    exact_pair<6>(xs, pf, pi, sf, si, d);
    exact_pair<8>(xs, pf, pi, sf, si, d);
    exact_pair<10>(xs, pf, pi, sf, si, d);
    exact_pair<12>(xs, pf, pi, sf, si, d);
    exact_pair<14>(xs, pf, pi, sf, si, d);
    // a tile's 256 contributions still span at most ~49 bits: exact in any order
    if constexpr (kTile) d = row16_sum(d);
    t1 = !(d < 0.0);
  }
  // Sign of X into bit 3 of every nibble: the E2M1 codes already carry it.
  if constexpr (kSR) {
    out = sr_codes(xs, t1 ? ei : ef, t1, rnd);
  } else {
    out.x = t1 ? (pi[0] | (pf[0] & 0x88888888u)) : pf[0];
    out.y = t1 ? (pi[1] | (pf[1] & 0x88888888u)) : pf[1];
  }
  scale_byte = t1 ? (0x80u | ci) : cf;
}

}  // namespace mixfp4
