// MixFP4 tensor scale and block quantizer (Algorithm 1) for gfx950.
//
// Tensor scale (Algorithm 1, first step): s32 = max|X| / 2688, where
// 2688 = 6 * 448 = 7 * 384 makes the block holding the tensor maximum land on
// the largest E4M3 scales.  Computed on the device in three short launches:
// clear -> per-workgroup max + one atomic max of the fp32 bit pattern (order
// free, so deterministic) -> finalize in place.
//
// Quantizer: one lane owns one 16-element block (App. B.1, V = 16): two
// 16-byte loads, no cross-lane traffic, one 8-byte code store and one scale
// byte.  Codes, scales and the format bit are exactly those of Algorithm 1:
//   * x = fl32(X / s32) is computed as fl32(X * fl64(1/s32)); X has 8
//     significant bits, so the exact quotient is never within 2^-50 of an
//     fp32 rounding boundary while the fp64 product is within 2^-52.
//   * y = fl32(x / s8) likewise as fl32(x * fl64(1/s8)) (s8 has 4
//     significant bits); rounding y to a grid equals rounding the exact
//     quotient, because |x| sits more than half an fp32 ulp of y away from
//     every grid midpoint * s8 unless it is exactly on it.
//   * E2M1 rounding uses the gfx950 FP4 converter with scale 1 (round to
//     nearest even onto the E2M1 grid, ties to the even code, saturating,
//     sign kept); INT4 rounding adds 2^23 (round half to even).
//   * The format choice: an fp32 estimate s_F^2 sum r_F^2 - s_I^2 sum r_I^2
//     (r = y - grid value) decides when it is farther from zero than its
//     proven error bound; otherwise the exact fp64 sum
//     sum_i (D_I - D_F)(2|x| - D_F - D_I) decides (every term exact, only
//     elements whose two dequantized values differ contribute, so the sum
//     is exact in any order).
#include <cmath>

#include "formats.h"
#include "hadamard.h"
#include "internal.h"
#include "philox.h"

namespace mixfp4 {
namespace {

constexpr int kThreads = 256;

__global__ void clear_u32(uint32_t* p) { *p = 0u; }

// max(|X|) bits over 8 bf16 in a 16-byte vector
__device__ __forceinline__ uint32_t absmax8(uint4 v) {
  const uint32_t m0 = max(max(v.x & 0x7FFFu, (v.x >> 16) & 0x7FFFu), max(v.y & 0x7FFFu, (v.y >> 16) & 0x7FFFu));
  const uint32_t m1 = max(max(v.z & 0x7FFFu, (v.z >> 16) & 0x7FFFu), max(v.w & 0x7FFFu, (v.w >> 16) & 0x7FFFu));
  return max(m0, m1);
}

// Per-workgroup max of |X| over a [rows, k] bf16 matrix (row pitch ldx) as
// bf16 magnitude bits.  Each thread keeps four 16-byte loads in flight.
// With `partials` the result of workgroup b goes to partials[b]; otherwise it
// is folded into *out with an atomic max of the fp32 bit pattern.
__global__ __launch_bounds__(kThreads) void amax_kernel(const uint16_t* __restrict__ x,
                                                         int64_t rows, int64_t k, int64_t ldx,
                                                         uint32_t* __restrict__ partials,
                                                         uint32_t* __restrict__ out) {
  const int64_t vec_per_row = k >> 3;               // 8 bf16 per 16-byte vector
  const int64_t total = rows * vec_per_row;
  auto vec_ptr = [&](int64_t i) -> const uint4* {
    if (ldx == k) return reinterpret_cast<const uint4*>(x) + i;
    const int64_t r = i / vec_per_row;
    return reinterpret_cast<const uint4*>(x + r * ldx) + (i - r * vec_per_row);
  };
  uint32_t m = 0u;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  for (; i + 3 * stride < total; i += 4 * stride) {
    const uint4 a = *vec_ptr(i), b = *vec_ptr(i + stride);
    const uint4 c = *vec_ptr(i + 2 * stride), d = *vec_ptr(i + 3 * stride);
    m = max(m, max(max(absmax8(a), absmax8(b)), max(absmax8(c), absmax8(d))));
  }
  for (; i < total; i += stride) m = max(m, absmax8(*vec_ptr(i)));
  for (int off = 32; off > 0; off >>= 1) m = max(m, (uint32_t)__shfl_xor((int)m, off));
  __shared__ uint32_t wave_max[kThreads / 64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) wave_max[wave] = m;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t r = wave_max[0];
    for (int w = 1; w < kThreads / 64; ++w) r = max(r, wave_max[w]);
    if (partials) partials[blockIdx.x] = r;
    else if (r) atomicMax(out, r << 16);            // bf16 bits -> fp32 bits
  }
}

__device__ __forceinline__ float tensor_scale_of(uint32_t amax_bf16_bits) {
  const float amax = __uint_as_float(amax_bf16_bits << 16);
  return amax > 0.0f ? amax / 2688.0f : 1.0f;       // Algorithm 1, first step
}

// One workgroup: fold the per-workgroup maxima and write s32.
__global__ __launch_bounds__(kThreads) void reduce_scale(const uint32_t* __restrict__ partials,
                                                          int count, float* __restrict__ out) {
  uint32_t m = 0u;
  for (int i = threadIdx.x; i < count; i += kThreads) m = max(m, partials[i]);
  for (int off = 32; off > 0; off >>= 1) m = max(m, (uint32_t)__shfl_xor((int)m, off));
  __shared__ uint32_t wave_max[kThreads / 64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) wave_max[wave] = m;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t r = wave_max[0];
    for (int w = 1; w < kThreads / 64; ++w) r = max(r, wave_max[w]);
    *out = tensor_scale_of(r);
  }
}

// In place: fp32 bits of max|X| -> s32 = fl32(amax / 2688), or 1.0 if zero.
__global__ void finalize_scale(uint32_t* p) {
  *reinterpret_cast<float*>(p) = tensor_scale_of(*p >> 16);
}

typedef float f32x2 __attribute__((ext_vector_type(2)));

// sum_{j<8} (0x4B000000 << 4j) mod 2^32: the constant part of the INT4 code
// accumulator below (every term is the bit pattern of 2^23 + code).
constexpr uint32_t kMagicPack = 0x4B000000u + (0x4B000000u << 4) + (0x4B000000u << 8) +
                                (0x4B000000u << 12) + (0x4B000000u << 16) + (0x4B000000u << 20) +
                                (0x4B000000u << 24) + (0x4B000000u << 28);

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

// Elements J, J+1 (J even) of a block, E2M1 branch: y = fl32(x / s_F)
// rounded by the gfx950 FP4 converter (scale 1: nearest, ties to the even
// code, saturating at 6, sign kept) into nibble pair (J%8)/2 of pf[J/8].
template <int J>
__device__ __forceinline__ void encode_f_pair(const float (&xs)[16], float sf, float rf,
                                              uint32_t (&pf)[2]) {
  const float yf0 = div_rn(xs[J], sf, rf), yf1 = div_rn(xs[J + 1], sf, rf);
  pf[J >> 3] = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(pf[J >> 3], yf0, yf1, 1.0f, (J & 7) >> 1);
}

// Elements J, J+1 (J even), E1M2 (x2 = INT4) branch: y = fl32(|x| / s_I);
// adding 2^23 rounds it to an integer (ties to even) held in the low mantissa
// bits, accumulated into pi[J/8] at nibble J%8 together with a constant
// removed afterwards.  With kErr, ai[J/2 % 2] += |x| * q_I.
template <int J, bool kErr>
__device__ __forceinline__ void encode_i_pair(const float (&xs)[16], float si, float ri,
                                              uint32_t (&pi)[2], float (&ai)[2]) {
  const float a0 = fabsf(xs[J]), a1 = fabsf(xs[J + 1]);
  const uint32_t b0 = __float_as_uint(div_rn(a0, si, ri) + 0x1p23f);
  const uint32_t b1 = __float_as_uint(div_rn(a1, si, ri) + 0x1p23f);
  if (kErr) {
    float& acc = ai[(J >> 1) & 1];
    acc = __builtin_fmaf(a0, __uint_as_float(b0) - 0x1p23f, acc);
    acc = __builtin_fmaf(a1, __uint_as_float(b1) - 0x1p23f, acc);
  }
  pi[J >> 3] += b0 << (4 * (J & 7));
  pi[J >> 3] += b1 << (4 * ((J + 1) & 7));
}

// E2M1 error sums of elements J, J+1 from the decoded codes, in two chains:
//   af += x * q_F (same signs, so every term is >= 0),  bf += q_F^2.
template <int J>
__device__ __forceinline__ void error_pair(const float (&xs)[16], const uint32_t (&pf)[2],
                                           float (&af)[2], float (&bf)[2]) {
  const f32x2 qf = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(pf[J >> 3], 1.0f, (J & 7) >> 1);
  constexpr int c = (J >> 1) & 1;
  af[c] = __builtin_fmaf(xs[J], qf.x, af[c]);
  af[c] = __builtin_fmaf(xs[J + 1], qf.y, af[c]);
  bf[c] = __builtin_fmaf(qf.x, qf.x, bf[c]);
  bf[c] = __builtin_fmaf(qf.y, qf.y, bf[c]);
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

// Format modes: MixFP4 selection (Algorithm 1), or one branch for every
// block (E2M1 = NVFP4, E1M2 = INT4); T records the branch either way.
constexpr int kSelect = 0, kForceE2M1 = 1, kForceE1M2 = 2;

// E1M2 codes of the 16 elements with saturation at 7 (a subnormal or
// saturated s_I admits codes above 7; rare path): codes into pi, with kErr
// also sum |x| q_I into ai.
template <bool kErr>
__device__ __forceinline__ void encode_i_saturated(const float (&xs)[16], float si, float ri,
                                                   uint32_t (&pi)[2], float (&ai)[2]) {
  pi[0] = pi[1] = 0u;
  ai[0] = ai[1] = 0.0f;
  for (int j = 0; j < 16; ++j) {
    const float q = fminf(rintf(div_rn(fabsf(xs[j]), si, ri)), 7.0f);
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
__device__ __forceinline__ uint2 sr_codes(const float (&xs)[16], float s, float r, bool int4,
                                          uint4 rnd) {
  const uint32_t words[4] = {rnd.x, rnd.y, rnd.z, rnd.w};
  uint32_t o[2] = {0u, 0u};
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    const uint32_t xb = __float_as_uint(xs[j]);
    const uint32_t neg = xb >> 31;
    const float y = div_rn(__uint_as_float(xb & 0x7FFFFFFFu), s, r);
    const uint32_t u = ((words[j >> 2] >> (8 * (j & 3))) & 0xFFu) ^ (neg ? 0xFFu : 0u);
    const float thr = (float)(511 - 2 * (int)u);
    const float inv_d = int4 ? 1.0f : (y < 2.0f ? 2.0f : (y < 4.0f ? 1.0f : 0.5f));
    const uint32_t base = int4 ? 0u : (y < 2.0f ? 0u : (y < 4.0f ? 2u : 4u));
    const float z = y * inv_d;
    const float lat = floorf(z);
    const float w = (z - lat) * 512.0f;
    uint32_t code = (uint32_t)lat + base;
    code += (w > thr || (w == thr && (code & 1u))) ? 1u : 0u;
    code = y >= (int4 ? 7.0f : 6.0f) ? 7u : code;
    o[j >> 3] |= (code | (neg << 3)) << (4 * (j & 7));
  }
  return make_uint2(o[0], o[1]);
}

// Codes and scale byte of one block from x (Algorithm 1 after the tensor
// scale).  With kSR the chosen branch's codes are written by stochastic
// rounding with the draws in `rnd`; scales and the format choice stay those
// of round-to-nearest.
template <int kMode, bool kSR>
__device__ __forceinline__ void quantize_xs(const float (&xs)[16], const float2* __restrict__ tab,
                                            uint2& out, uint32_t& scale_byte, uint4 rnd) {
  // fl32 rounding is monotonic, so bm is also fl32(max|X| / s32).
  float bm = 0.0f;
#pragma unroll
  for (int j = 0; j < 16; ++j) bm = fmaxf(bm, fabsf(xs[j]));
  // Candidate block scales E4M3(bm/6), E4M3(bm/7): the exactly rounded
  // quotients, clamped at 448 (saturation), through the gfx950 E4M3
  // converter (scale 1: nearest, ties to the even code; checked against the
  // software rounding on every fp32 value in [0, 448]).
  constexpr float kR6 = 1.0f / 6.0f, kR7 = 1.0f / 7.0f;
  const float cand6 = kMode == kForceE1M2 ? 0.0f : fminf(div_rn(bm, 6.0f, kR6), 448.0f);
  const float cand7 = kMode == kForceE2M1 ? 0.0f : fminf(div_rn(bm, 7.0f, kR7), 448.0f);
  const s16x2 sc = __builtin_amdgcn_cvt_scalef32_pk_fp8_f32(s16x2{0, 0}, cand6, cand7, 1.0f, false);
  const uint32_t scw = __builtin_bit_cast(uint32_t, sc);
  const uint32_t cf = scw & 0x7Fu, ci = (scw >> 8) & 0x7Fu;
  const float2 ef = tab[cf], ei = tab[ci];
  const float sf = ef.x, rf = ef.y, si = ei.x, ri = ei.y;

  uint32_t pf[2] = {0u, 0u}, pi[2] = {0u, 0u};
  float af[2] = {0.0f, 0.0f}, bf[2] = {0.0f, 0.0f}, ai[2] = {0.0f, 0.0f};
  if constexpr (kMode != kForceE1M2) {
    encode_f_pair<0>(xs, sf, rf, pf);
    encode_f_pair<2>(xs, sf, rf, pf);
    encode_f_pair<4>(xs, sf, rf, pf);
    encode_f_pair<6>(xs, sf, rf, pf);
    encode_f_pair<8>(xs, sf, rf, pf);
    encode_f_pair<10>(xs, sf, rf, pf);
    encode_f_pair<12>(xs, sf, rf, pf);
    encode_f_pair<14>(xs, sf, rf, pf);
  }
  if constexpr (kMode == kForceE2M1) {
    out = kSR ? sr_codes(xs, sf, rf, false, rnd) : make_uint2(pf[0], pf[1]);
    scale_byte = cf;
    return;
  }
  constexpr bool kErr = kMode == kSelect;
  encode_i_pair<0, kErr>(xs, si, ri, pi, ai);
  encode_i_pair<2, kErr>(xs, si, ri, pi, ai);
  encode_i_pair<4, kErr>(xs, si, ri, pi, ai);
  encode_i_pair<6, kErr>(xs, si, ri, pi, ai);
  encode_i_pair<8, kErr>(xs, si, ri, pi, ai);
  encode_i_pair<10, kErr>(xs, si, ri, pi, ai);
  encode_i_pair<12, kErr>(xs, si, ri, pi, ai);
  encode_i_pair<14, kErr>(xs, si, ri, pi, ai);
  pi[0] -= kMagicPack;
  pi[1] -= kMagicPack;
  // INT4 codes cannot exceed 7 when s_I is a normal E4M3 value below the
  // maximum (then max|x| / s_I < 7.47); other blocks redo the branch with
  // saturation (rare path).
  if (ci < 8u || ci >= 0x7Eu) encode_i_saturated<kErr>(xs, si, ri, pi, ai);
  if constexpr (kMode == kForceE1M2) {
    // sign of X into bit 3 of every nibble
    uint32_t sg[2] = {0u, 0u};
#pragma unroll
    for (int j = 0; j < 16; ++j) sg[j >> 3] |= (__float_as_uint(xs[j]) >> 31) << (4 * (j & 7) + 3);
    out = kSR ? sr_codes(xs, si, ri, true, rnd) : make_uint2(pi[0] | sg[0], pi[1] | sg[1]);
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
  const uint32_t bi = __builtin_amdgcn_udot8(pi[0], pi[0], __builtin_amdgcn_udot8(pi[1], pi[1], 0u, false),
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
  const float afs = af[0] + af[1], ais = ai[0] + ai[1], bfs = bf[0] + bf[1];
  const float sf2b = (sf * sf) * bfs, si2b = (si * si) * (float)bi;
  const float tf = sf * afs, ti = si * ais;
  const float est = (sf2b - si2b) + 2.0f * (ti - tf);
  const float tau = 0x1p-19f * (tf + ti) + 0x1p-22f * (sf2b + si2b);
  bool t1;
  if (cf != 0u && ci != 0u && fabsf(est) > tau) {
    t1 = !(est < 0.0f);
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
    t1 = !(d < 0.0);
  }
  // Sign of X into bit 3 of every nibble: the E2M1 codes already carry it.
  if constexpr (kSR) {
    out = sr_codes(xs, t1 ? si : sf, t1 ? ri : rf, t1, rnd);
  } else {
    out.x = t1 ? (pi[0] | (pf[0] & 0x88888888u)) : pf[0];
    out.y = t1 ? (pi[1] | (pf[1] & 0x88888888u)) : pf[1];
  }
  scale_byte = t1 ? (0x80u | ci) : cf;
}

// Grid-stride walk over the blocks.  The next block of this thread is
// loaded as soon as the current one has been turned into x, so its load
// overlaps this block's arithmetic (measured: a second block in flight, or
// more waves per SIMD, gains nothing; the kernel is bound by VALU issue).
//
// kSR: stochastic rounding with Philox draws per block (its global index).
// kHad: each block is first rotated (block-diagonal Hadamard across the
// L = b / 16 lanes holding one Hadamard block; the grid stride is a multiple
// of 256, so a thread keeps its position in its Hadamard block and every
// Hadamard block is processed by lanes of one wave in one iteration).
template <bool kContig, bool kScaled, int kMode, bool kSR, bool kHad>
__device__ __forceinline__ void quantize_loop(const uint16_t* __restrict__ x, int64_t nbk,
                                              int64_t ldx, int64_t nblocks,
                                              uint8_t* __restrict__ codes,
                                              uint8_t* __restrict__ scales, float xmul, float sx,
                                              float rx, const float2* tab, const SrParams& sr,
                                              const HadamardParams& hp) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  // Loads are unconditional (a block index past the end reads the last
  // block, whose data is then never used), so they need no branch and no
  // register copies.
  auto load = [&](int64_t gi, uint4& p, uint4& q) {
    gi = gi < nblocks ? gi : nblocks - 1;
    const uint16_t* src;
    if (kContig) {
      src = x + (gi << 4);
    } else {
      const int64_t r = gi / nbk;
      src = x + r * ldx + ((gi - r * nbk) << 4);
    }
    p = *reinterpret_cast<const uint4*>(src);
    q = *reinterpret_cast<const uint4*>(src + 8);
  };
  int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  SignMasks sm;
  if constexpr (kHad) sm = load_sign_masks(hp, (int)(threadIdx.x & ((1u << hp.lanes_log2) - 1u)));
  uint4 a0, a1;
  load(g, a0, a1);
  for (; g < nblocks; g += stride) {
    float xs[16];
    if constexpr (kHad) {
      uint4 r0 = a0, r1 = a1;
      hadamard_rotate(r0, r1, sm, hp);
      to_fp8_domain<kScaled>(r0, r1, xmul, sx, rx, xs);
    } else {
      to_fp8_domain<kScaled>(a0, a1, xmul, sx, rx, xs);
    }
    load(g + stride, a0, a1);
    uint2 out;
    uint32_t sb;
    quantize_xs<kMode, kSR>(xs, tab, out, sb, kSR ? block_draws(g, sr) : make_uint4(0, 0, 0, 0));
    *reinterpret_cast<uint2*>(codes + (g << 3)) = out;
    scales[g] = (uint8_t)sb;
  }
}

// {E4M3(c), fl32(1 / E4M3(c))} for every 7-bit code ({0, 0} for the zero
// scale and the NaN code), built by the first 128 threads; the caller
// synchronizes before use.
__device__ __forceinline__ void fill_scale_table(float2* tab) {
  if (threadIdx.x < 128) {
    const float v = e4m3_value(threadIdx.x);
    const bool ok = threadIdx.x > 0 && threadIdx.x < 127;
    tab[threadIdx.x] = ok ? make_float2(v, __fdiv_rn(1.0f, v)) : make_float2(0.0f, 0.0f);
  }
}

// Quantize blocks [this thread's grid-stride share] with tensor scale s32.
// The division steps stay in the normal range for every element that can get
// a nonzero code when 2^-90 <= s32 <= 2^120; beyond that both X and s32 are
// rescaled by 2^64 or 2^-64 first.
template <bool kContig, int kMode, bool kSR, bool kHad>
__device__ __forceinline__ void quantize_all(const uint16_t* __restrict__ x, int64_t nbk,
                                             int64_t ldx, int64_t nblocks,
                                             uint8_t* __restrict__ codes,
                                             uint8_t* __restrict__ scales, float s32,
                                             const float2* tab, const SrParams& sr,
                                             const HadamardParams& hp) {
  if (s32 >= 0x1p-90f && s32 <= 0x1p120f) {
    quantize_loop<kContig, false, kMode, kSR, kHad>(x, nbk, ldx, nblocks, codes, scales, 1.0f,
                                                    s32, __fdiv_rn(1.0f, s32), tab, sr, hp);
  } else {
    const float xmul = s32 < 1.0f ? 0x1p64f : 0x1p-64f;
    const float sx = s32 * xmul;
    quantize_loop<kContig, true, kMode, kSR, kHad>(x, nbk, ldx, nblocks, codes, scales, xmul, sx,
                                                   __fdiv_rn(1.0f, sx), tab, sr, hp);
  }
}

template <bool kContig, int kMode, bool kSR, bool kHad>
__global__ __launch_bounds__(kThreads) void quantize_kernel(
    const uint16_t* __restrict__ x, int64_t nbk, int64_t ldx, int64_t nblocks,
    uint8_t* __restrict__ codes, uint8_t* __restrict__ scales,
    const float* __restrict__ tensor_scale, SrParams sr, HadamardParams hp) {
  __shared__ float2 tab[128];
  fill_scale_table(tab);
  __syncthreads();
  quantize_all<kContig, kMode, kSR, kHad>(x, nbk, ldx, nblocks, codes, scales, *tensor_scale, tab,
                                          sr, hp);
}

// Small tensors with the tensor scale computed (at most kSmallElems
// elements): one launch, at most one block per thread.  Every workgroup reads
// the whole tensor for max|X| (a few hundred KB, from L2 after the first), so
// all of them hold the same s32 without talking to each other; workgroup 0
// stores it.  The read walks blocks in the order of the quantize assignment
// (block w * kSmallThreads + t of workgroup w goes to its thread t), so each
// thread keeps its own block from that pass and quantizes it without a
// second read.  The maximum is order-independent: the result is the
// two-pass one, bit for bit.
constexpr int kSmallThreads = 1024;
constexpr int64_t kSmallElems = int64_t(1) << 18;

template <bool kContig, int kMode, bool kSR>
__global__ __launch_bounds__(kSmallThreads) void quantize_small_kernel(
    const uint16_t* __restrict__ x, int64_t nbk, int64_t ldx, int64_t nblocks,
    uint8_t* __restrict__ codes, uint8_t* __restrict__ scales, float* __restrict__ tensor_scale,
    SrParams sr) {
  __shared__ float2 tab[128];
  __shared__ uint32_t wave_max[kSmallThreads / 64];
  fill_scale_table(tab);
  auto block_ptr = [&](int64_t g) -> const uint16_t* {
    if (kContig) return x + (g << 4);
    const int64_t r = g / nbk;
    return x + r * ldx + ((g - r * nbk) << 4);
  };
  // max|X| as bf16 magnitude bits; eight blocks in flight per thread
  constexpr int kInFlight = 8;
  const int64_t rounds = (nblocks + kSmallThreads - 1) / kSmallThreads;
  const int64_t mine = blockIdx.x;                  // round holding this thread's block
  uint32_t mx = 0u;
  uint4 k0 = make_uint4(0, 0, 0, 0), k1 = k0;
  for (int64_t r0 = 0; r0 < rounds; r0 += kInFlight) {
    uint4 v0[kInFlight], v1[kInFlight];
#pragma unroll
    for (int j = 0; j < kInFlight; ++j) {
      int64_t g = (r0 + j) * kSmallThreads + threadIdx.x;
      g = g < nblocks ? g : nblocks - 1;           // past the end: re-read the last block
      const uint16_t* src = block_ptr(g);
      v0[j] = *reinterpret_cast<const uint4*>(src);
      v1[j] = *reinterpret_cast<const uint4*>(src + 8);
    }
#pragma unroll
    for (int j = 0; j < kInFlight; ++j) {
      mx = max(mx, max(absmax8(v0[j]), absmax8(v1[j])));
      if (r0 + j == mine) {
        k0 = v0[j];
        k1 = v1[j];
      }
    }
  }
  for (int off = 32; off > 0; off >>= 1) mx = max(mx, (uint32_t)__shfl_xor((int)mx, off));
  if ((threadIdx.x & 63) == 0) wave_max[threadIdx.x >> 6] = mx;
  __syncthreads();                                  // also publishes the scale table
  uint32_t r = wave_max[0];
#pragma unroll
  for (int w = 1; w < kSmallThreads / 64; ++w) r = max(r, wave_max[w]);
  const float s32 = tensor_scale_of(r);
  if (blockIdx.x == 0 && threadIdx.x == 0) *tensor_scale = s32;

  const int64_t g = mine * kSmallThreads + threadIdx.x;
  if (g >= nblocks) return;
  const bool direct = s32 >= 0x1p-90f && s32 <= 0x1p120f;
  float xs[16];
  if (direct) {
    to_fp8_domain<false>(k0, k1, 1.0f, s32, __fdiv_rn(1.0f, s32), xs);
  } else {
    const float xmul = s32 < 1.0f ? 0x1p64f : 0x1p-64f;
    const float sx = s32 * xmul;
    to_fp8_domain<true>(k0, k1, xmul, sx, __fdiv_rn(1.0f, sx), xs);
  }
  uint2 out;
  uint32_t sb;
  quantize_xs<kMode, kSR>(xs, tab, out, sb, kSR ? block_draws(g, sr) : make_uint4(0, 0, 0, 0));
  *reinterpret_cast<uint2*>(codes + (g << 3)) = out;
  scales[g] = (uint8_t)sb;
}

// Per-workgroup max|Y| of the rotated tensor (bf16 magnitude bits of the
// rounded results), same lane-per-block walk as the quantizer so that every
// Hadamard block sits in consecutive lanes of one wave.  Results go to
// partials[blockIdx.x] or, without partials, into *out by atomic max.
template <bool kContig>
__global__ __launch_bounds__(kThreads) void amax_rotated_kernel(
    const uint16_t* __restrict__ x, int64_t nbk, int64_t ldx, int64_t nblocks, HadamardParams hp,
    uint32_t* __restrict__ partials, uint32_t* __restrict__ out) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const SignMasks sm = load_sign_masks(hp, (int)(threadIdx.x & ((1u << hp.lanes_log2) - 1u)));
  uint32_t m = 0u;
  for (int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; g < nblocks; g += stride) {
    const uint16_t* src;
    if (kContig) {
      src = x + (g << 4);
    } else {
      const int64_t r = g / nbk;
      src = x + r * ldx + ((g - r * nbk) << 4);
    }
    uint4 v0 = *reinterpret_cast<const uint4*>(src);
    uint4 v1 = *reinterpret_cast<const uint4*>(src + 8);
    hadamard_rotate(v0, v1, sm, hp);
    m = max(m, max(absmax8(v0), absmax8(v1)));
  }
  for (int off = 32; off > 0; off >>= 1) m = max(m, (uint32_t)__shfl_xor((int)m, off));
  __shared__ uint32_t wave_max[kThreads / 64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) wave_max[wave] = m;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t r = wave_max[0];
    for (int w = 1; w < kThreads / 64; ++w) r = max(r, wave_max[w]);
    if (partials) partials[blockIdx.x] = r;
    else if (r) atomicMax(out, r << 16);
  }
}

// Standalone rotation: y[g] = rotated block g (y contiguous [rows, k]).
template <bool kContig>
__global__ __launch_bounds__(kThreads) void hadamard_kernel(const uint16_t* __restrict__ x,
                                                            int64_t nbk, int64_t ldx,
                                                            int64_t nblocks, HadamardParams hp,
                                                            uint16_t* __restrict__ y) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const SignMasks sm = load_sign_masks(hp, (int)(threadIdx.x & ((1u << hp.lanes_log2) - 1u)));
  for (int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; g < nblocks; g += stride) {
    const uint16_t* src;
    if (kContig) {
      src = x + (g << 4);
    } else {
      const int64_t r = g / nbk;
      src = x + r * ldx + ((g - r * nbk) << 4);
    }
    uint4 v0 = *reinterpret_cast<const uint4*>(src);
    uint4 v1 = *reinterpret_cast<const uint4*>(src + 8);
    hadamard_rotate(v0, v1, sm, hp);
    uint4* dst = reinterpret_cast<uint4*>(y + (g << 4));
    dst[0] = v0;
    dst[1] = v1;
  }
}

// Workgroups of kThreads that the device keeps resident at once for
// `kernel` (occupancy per CU x CU count); `cache` holds one value per device.
template <typename Kernel>
int64_t resident_groups(Kernel kernel, int64_t (&cache)[64]) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 1024;
  if (!cache[dev]) {
    int per_cu = 0, cus = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, kThreads, 0) != hipSuccess ||
        per_cu <= 0)
      per_cu = 4;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        cus <= 0)
      cus = 256;
    cache[dev] = (int64_t)per_cu * cus;
  }
  return cache[dev];
}

int grid_for(int64_t work, int per_thread) {
  int64_t g = (work + (int64_t)kThreads * per_thread - 1) / ((int64_t)kThreads * per_thread);
  if (g < 1) g = 1;
  if (g > 65536) g = 65536;
  return (int)g;
}

// Per-workgroup maxima: to the caller's scratch (the scale-byte output, which
// the quantize kernel overwrites afterwards) when it holds at least 16 slots,
// else an atomic on *tensor_scale.  `run(grid, partials, out)` launches the
// maximum kernel; `grid` is capped by the slots.
template <typename Run>
hipError_t tensor_scale_with(int64_t work, int grid, uint8_t* scratch, int64_t scratch_bytes,
                             float* tensor_scale, hipStream_t stream, Run run) {
  const uintptr_t base = reinterpret_cast<uintptr_t>(scratch);
  const uintptr_t aligned = (base + 3u) & ~uintptr_t(3);
  const int64_t slots = scratch ? (scratch_bytes - (int64_t)(aligned - base)) / 4 : 0;
  if (work > 0 && slots >= 16) {
    if (grid > slots) grid = (int)slots;
    uint32_t* partials = reinterpret_cast<uint32_t*>(aligned);
    run(grid, partials, (uint32_t*)nullptr);
    reduce_scale<<<1, kThreads, 0, stream>>>(partials, grid, tensor_scale);
    return hipGetLastError();
  }
  uint32_t* p = reinterpret_cast<uint32_t*>(tensor_scale);
  clear_u32<<<1, 1, 0, stream>>>(p);
  if (work > 0) run(grid, (uint32_t*)nullptr, p);
  finalize_scale<<<1, 1, 0, stream>>>(p);
  return hipGetLastError();
}

}  // namespace

HadamardParams hadamard_params(int b, const int8_t* signs) {
  HadamardParams hp{};
  int level = 0;
  while ((1 << level) < b) ++level;
  hp.signs = signs;
  hp.lanes_log2 = level - 4;
  hp.odd = level & 1;
  // 1 / sqrt(b) = 2^-(level / 2) (times the fp64 sqrt(1/2) for odd levels)
  hp.scale = std::ldexp(hp.odd ? 0.70710678118654752440 : 1.0, -(level / 2));
  hp.b = (double)b;
  return hp;
}

hipError_t launch_tensor_scale(const uint16_t* x, int64_t rows, int64_t k, int64_t ldx,
                               uint8_t* scratch, int64_t scratch_bytes, float* tensor_scale,
                               hipStream_t stream) {
  const int64_t total = rows * (k >> 3);
  // up to 1024 workgroups x 256 threads x 4 loads of 16 B keeps ~16 MB in flight
  int g = grid_for(total, 4);
  if (g > 1024) g = 1024;
  return tensor_scale_with(total, g, scratch, scratch_bytes, tensor_scale, stream,
                           [&](int grid, uint32_t* partials, uint32_t* out) {
                             amax_kernel<<<grid, kThreads, 0, stream>>>(x, rows, k, ldx, partials,
                                                                         out);
                           });
}

hipError_t launch_tensor_scale_rotated(const uint16_t* x, int64_t rows, int64_t k, int64_t ldx,
                                       const HadamardParams& hp, uint8_t* scratch,
                                       int64_t scratch_bytes, float* tensor_scale,
                                       hipStream_t stream) {
  const int64_t nbk = k / kBlock, nblocks = rows * nbk;
  static int64_t cache_c[64], cache_s[64];
  const int64_t resident = ldx == k ? resident_groups(amax_rotated_kernel<true>, cache_c)
                                    : resident_groups(amax_rotated_kernel<false>, cache_s);
  const int64_t wanted = (nblocks + kThreads - 1) / kThreads;
  int g = (int)(wanted < resident ? wanted : resident);
  if (g < 1) g = 1;
  return tensor_scale_with(nblocks, g, scratch, scratch_bytes, tensor_scale, stream,
                           [&](int grid, uint32_t* partials, uint32_t* out) {
                             if (ldx == k)
                               amax_rotated_kernel<true><<<grid, kThreads, 0, stream>>>(
                                   x, nbk, ldx, nblocks, hp, partials, out);
                             else
                               amax_rotated_kernel<false><<<grid, kThreads, 0, stream>>>(
                                   x, nbk, ldx, nblocks, hp, partials, out);
                           });
}

namespace {

template <int kMode, bool kSR>
hipError_t launch_small_mode(const uint16_t* x, int64_t rows, int64_t k, int64_t ldx,
                             uint8_t* codes, uint8_t* scales, float* tensor_scale,
                             const SrParams& sr, hipStream_t stream) {
  const int64_t nbk = k / kBlock, nblocks = rows * nbk;
  const int64_t g = (nblocks + kSmallThreads - 1) / kSmallThreads;   // one block per thread
  if (ldx == k)
    quantize_small_kernel<true, kMode, kSR><<<(unsigned)g, kSmallThreads, 0, stream>>>(
        x, nbk, ldx, nblocks, codes, scales, tensor_scale, sr);
  else
    quantize_small_kernel<false, kMode, kSR><<<(unsigned)g, kSmallThreads, 0, stream>>>(
        x, nbk, ldx, nblocks, codes, scales, tensor_scale, sr);
  return hipGetLastError();
}

template <int kMode, bool kSR, bool kHad>
hipError_t launch_mode(const uint16_t* x, int64_t rows, int64_t k, int64_t ldx, uint8_t* codes,
                       uint8_t* scales, const float* tensor_scale, const QuantOptions& opt,
                       hipStream_t stream) {
  const int64_t nbk = k / kBlock;
  const int64_t nblocks = rows * nbk;
  // One wave of resident workgroups (occupancy x CUs) walks all blocks, so
  // no partial second wave is left at the end; fewer if the tensor is small.
  static int64_t cache_c[64], cache_s[64];
  const int64_t wanted = (nblocks + kThreads - 1) / kThreads;
  const int64_t resident =
      ldx == k ? resident_groups(quantize_kernel<true, kMode, kSR, kHad>, cache_c)
               : resident_groups(quantize_kernel<false, kMode, kSR, kHad>, cache_s);
  const int g = (int)(wanted < resident ? wanted : resident);
  if (ldx == k)
    quantize_kernel<true, kMode, kSR, kHad><<<g, kThreads, 0, stream>>>(
        x, nbk, ldx, nblocks, codes, scales, tensor_scale, opt.srp, opt.hp);
  else
    quantize_kernel<false, kMode, kSR, kHad><<<g, kThreads, 0, stream>>>(
        x, nbk, ldx, nblocks, codes, scales, tensor_scale, opt.srp, opt.hp);
  return hipGetLastError();
}

template <int kMode>
hipError_t launch_mode_opts(const uint16_t* x, int64_t rows, int64_t k, int64_t ldx,
                            uint8_t* codes, uint8_t* scales, const float* tensor_scale,
                            const QuantOptions& opt, hipStream_t stream) {
  if (opt.sr)
    return opt.had ? launch_mode<kMode, true, true>(x, rows, k, ldx, codes, scales, tensor_scale,
                                                    opt, stream)
                   : launch_mode<kMode, true, false>(x, rows, k, ldx, codes, scales,
                                                     tensor_scale, opt, stream);
  return opt.had ? launch_mode<kMode, false, true>(x, rows, k, ldx, codes, scales, tensor_scale,
                                                   opt, stream)
                 : launch_mode<kMode, false, false>(x, rows, k, ldx, codes, scales, tensor_scale,
                                                    opt, stream);
}

template <int kMode>
hipError_t launch_small_opts(const uint16_t* x, int64_t rows, int64_t k, int64_t ldx,
                             uint8_t* codes, uint8_t* scales, float* tensor_scale,
                             const QuantOptions& opt, hipStream_t stream) {
  return opt.sr ? launch_small_mode<kMode, true>(x, rows, k, ldx, codes, scales, tensor_scale,
                                                 opt.srp, stream)
                : launch_small_mode<kMode, false>(x, rows, k, ldx, codes, scales, tensor_scale,
                                                  opt.srp, stream);
}

}  // namespace

hipError_t launch_quantize_small(const uint16_t* x, int64_t rows, int64_t k, int64_t ldx,
                                 uint8_t* codes, uint8_t* scales, float* tensor_scale,
                                 const QuantOptions& opt, hipStream_t stream) {
  if (opt.mode == kForceE2M1)
    return launch_small_opts<kForceE2M1>(x, rows, k, ldx, codes, scales, tensor_scale, opt, stream);
  if (opt.mode == kForceE1M2)
    return launch_small_opts<kForceE1M2>(x, rows, k, ldx, codes, scales, tensor_scale, opt, stream);
  return launch_small_opts<kSelect>(x, rows, k, ldx, codes, scales, tensor_scale, opt, stream);
}

bool quantize_is_small(int64_t rows, int64_t k) { return rows * k <= kSmallElems; }

hipError_t launch_quantize(const uint16_t* x, int64_t rows, int64_t k, int64_t ldx,
                           uint8_t* codes, uint8_t* scales, const float* tensor_scale,
                           const QuantOptions& opt, hipStream_t stream) {
  if (rows * (k / kBlock) == 0) return hipSuccess;
  if (opt.mode == kForceE2M1)
    return launch_mode_opts<kForceE2M1>(x, rows, k, ldx, codes, scales, tensor_scale, opt, stream);
  if (opt.mode == kForceE1M2)
    return launch_mode_opts<kForceE1M2>(x, rows, k, ldx, codes, scales, tensor_scale, opt, stream);
  return launch_mode_opts<kSelect>(x, rows, k, ldx, codes, scales, tensor_scale, opt, stream);
}

hipError_t launch_hadamard(const uint16_t* x, int64_t rows, int64_t k, int64_t ldx,
                           const HadamardParams& hp, uint16_t* y, hipStream_t stream) {
  const int64_t nbk = k / kBlock, nblocks = rows * nbk;
  if (nblocks == 0) return hipSuccess;
  static int64_t cache_c[64], cache_s[64];
  const int64_t resident = ldx == k ? resident_groups(hadamard_kernel<true>, cache_c)
                                    : resident_groups(hadamard_kernel<false>, cache_s);
  const int64_t wanted = (nblocks + kThreads - 1) / kThreads;
  const int g = (int)(wanted < resident ? wanted : resident);
  if (ldx == k)
    hadamard_kernel<true><<<g, kThreads, 0, stream>>>(x, nbk, ldx, nblocks, hp, y);
  else
    hadamard_kernel<false><<<g, kThreads, 0, stream>>>(x, nbk, ldx, nblocks, hp, y);
  return hipGetLastError();
}

}  // namespace mixfp4
