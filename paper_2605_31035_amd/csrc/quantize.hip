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
#include "formats.h"
#include "internal.h"

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

// Codes and scale byte of one block from x (Algorithm 1 after the tensor
// scale).
template <int kMode>
__device__ __forceinline__ void quantize_xs(const float (&xs)[16], const float2* __restrict__ tab,
                                            uint2& out, uint32_t& scale_byte) {
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
    out = make_uint2(pf[0], pf[1]);
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
    out = make_uint2(pi[0] | sg[0], pi[1] | sg[1]);
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
  out.x = t1 ? (pi[0] | (pf[0] & 0x88888888u)) : pf[0];
  out.y = t1 ? (pi[1] | (pf[1] & 0x88888888u)) : pf[1];
  scale_byte = t1 ? (0x80u | ci) : cf;
}

// Grid-stride walk over the blocks.  The next block of this thread is
// loaded as soon as the current one has been turned into x, so its load
// overlaps this block's arithmetic (measured: a second block in flight, or
// more waves per SIMD, gains nothing; the kernel is bound by VALU issue).
template <bool kContig, bool kScaled, int kMode>
__device__ __forceinline__ void quantize_loop(const uint16_t* __restrict__ x, int64_t nbk,
                                              int64_t ldx, int64_t nblocks,
                                              uint8_t* __restrict__ codes,
                                              uint8_t* __restrict__ scales, float xmul, float sx,
                                              float rx, const float2* tab) {
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
  uint4 a0, a1;
  load(g, a0, a1);
  for (; g < nblocks; g += stride) {
    float xs[16];
    to_fp8_domain<kScaled>(a0, a1, xmul, sx, rx, xs);
    load(g + stride, a0, a1);
    uint2 out;
    uint32_t sb;
    quantize_xs<kMode>(xs, tab, out, sb);
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
template <bool kContig, int kMode>
__device__ __forceinline__ void quantize_all(const uint16_t* __restrict__ x, int64_t nbk,
                                             int64_t ldx, int64_t nblocks,
                                             uint8_t* __restrict__ codes,
                                             uint8_t* __restrict__ scales, float s32,
                                             const float2* tab) {
  if (s32 >= 0x1p-90f && s32 <= 0x1p120f) {
    quantize_loop<kContig, false, kMode>(x, nbk, ldx, nblocks, codes, scales, 1.0f, s32,
                                  __fdiv_rn(1.0f, s32), tab);
  } else {
    const float xmul = s32 < 1.0f ? 0x1p64f : 0x1p-64f;
    const float sx = s32 * xmul;
    quantize_loop<kContig, true, kMode>(x, nbk, ldx, nblocks, codes, scales, xmul, sx,
                                 __fdiv_rn(1.0f, sx), tab);
  }
}

template <bool kContig, int kMode>
__global__ __launch_bounds__(kThreads) void quantize_kernel(
    const uint16_t* __restrict__ x, int64_t nbk, int64_t ldx, int64_t nblocks,
    uint8_t* __restrict__ codes, uint8_t* __restrict__ scales,
    const float* __restrict__ tensor_scale) {
  __shared__ float2 tab[128];
  fill_scale_table(tab);
  __syncthreads();
  quantize_all<kContig, kMode>(x, nbk, ldx, nblocks, codes, scales, *tensor_scale, tab);
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

template <bool kContig, int kMode>
__global__ __launch_bounds__(kSmallThreads) void quantize_small_kernel(
    const uint16_t* __restrict__ x, int64_t nbk, int64_t ldx, int64_t nblocks,
    uint8_t* __restrict__ codes, uint8_t* __restrict__ scales, float* __restrict__ tensor_scale) {
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
  quantize_xs<kMode>(xs, tab, out, sb);
  *reinterpret_cast<uint2*>(codes + (g << 3)) = out;
  scales[g] = (uint8_t)sb;
}

// Workgroups of kThreads that the device keeps resident at once for
// quantize_kernel<kContig, kMode> (occupancy per CU x CU count), cached per
// device.
template <bool kContig, int kMode>
int64_t resident_groups() {
  static int64_t cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 1024;
  if (!cached[dev]) {
    int per_cu = 0, cus = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, quantize_kernel<kContig, kMode>, kThreads,
                                                     0) != hipSuccess ||
        per_cu <= 0)
      per_cu = 4;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        cus <= 0)
      cus = 256;
    cached[dev] = (int64_t)per_cu * cus;
  }
  return cached[dev];
}

int grid_for(int64_t work, int per_thread) {
  int64_t g = (work + (int64_t)kThreads * per_thread - 1) / ((int64_t)kThreads * per_thread);
  if (g < 1) g = 1;
  if (g > 65536) g = 65536;
  return (int)g;
}

}  // namespace

hipError_t launch_tensor_scale(const uint16_t* x, int64_t rows, int64_t k, int64_t ldx,
                               uint8_t* scratch, int64_t scratch_bytes, float* tensor_scale,
                               hipStream_t stream) {
  const int64_t total = rows * (k >> 3);
  // Per-workgroup maxima go to the caller's scale-byte output, which the
  // quantize kernel overwrites afterwards; tiny outputs use an atomic instead.
  const uintptr_t base = reinterpret_cast<uintptr_t>(scratch);
  const uintptr_t aligned = (base + 3u) & ~uintptr_t(3);
  const int64_t slots = scratch ? (scratch_bytes - (int64_t)(aligned - base)) / 4 : 0;
  // up to 1024 workgroups x 256 threads x 4 loads of 16 B keeps ~16 MB in flight
  int g = grid_for(total, 4);
  if (g > 1024) g = 1024;
  if (total > 0 && slots >= 16) {
    if (g > slots) g = (int)slots;
    uint32_t* partials = reinterpret_cast<uint32_t*>(aligned);
    amax_kernel<<<g, kThreads, 0, stream>>>(x, rows, k, ldx, partials, nullptr);
    reduce_scale<<<1, kThreads, 0, stream>>>(partials, g, tensor_scale);
    return hipGetLastError();
  }
  uint32_t* p = reinterpret_cast<uint32_t*>(tensor_scale);
  clear_u32<<<1, 1, 0, stream>>>(p);
  if (total > 0) amax_kernel<<<g, kThreads, 0, stream>>>(x, rows, k, ldx, nullptr, p);
  finalize_scale<<<1, 1, 0, stream>>>(p);
  return hipGetLastError();
}

namespace {

template <int kMode>
hipError_t launch_small_mode(const uint16_t* x, int64_t rows, int64_t k, int64_t ldx,
                             uint8_t* codes, uint8_t* scales, float* tensor_scale,
                             hipStream_t stream) {
  const int64_t nbk = k / kBlock, nblocks = rows * nbk;
  const int64_t g = (nblocks + kSmallThreads - 1) / kSmallThreads;   // one block per thread
  if (ldx == k)
    quantize_small_kernel<true, kMode><<<(unsigned)g, kSmallThreads, 0, stream>>>(
        x, nbk, ldx, nblocks, codes, scales, tensor_scale);
  else
    quantize_small_kernel<false, kMode><<<(unsigned)g, kSmallThreads, 0, stream>>>(
        x, nbk, ldx, nblocks, codes, scales, tensor_scale);
  return hipGetLastError();
}

template <int kMode>
hipError_t launch_mode(const uint16_t* x, int64_t rows, int64_t k, int64_t ldx, uint8_t* codes,
                       uint8_t* scales, const float* tensor_scale, hipStream_t stream) {
  const int64_t nbk = k / kBlock;
  const int64_t nblocks = rows * nbk;
  // One wave of resident workgroups (occupancy x CUs) walks all blocks, so
  // no partial second wave is left at the end; fewer if the tensor is small.
  const int64_t wanted = (nblocks + kThreads - 1) / kThreads;
  const int64_t resident = ldx == k ? resident_groups<true, kMode>() : resident_groups<false, kMode>();
  const int g = (int)(wanted < resident ? wanted : resident);
  if (ldx == k)
    quantize_kernel<true, kMode><<<g, kThreads, 0, stream>>>(x, nbk, ldx, nblocks, codes, scales,
                                                              tensor_scale);
  else
    quantize_kernel<false, kMode><<<g, kThreads, 0, stream>>>(x, nbk, ldx, nblocks, codes,
                                                               scales, tensor_scale);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_quantize_small(const uint16_t* x, int64_t rows, int64_t k, int64_t ldx,
                                 uint8_t* codes, uint8_t* scales, float* tensor_scale, int mode,
                                 hipStream_t stream) {
  if (mode == kForceE2M1)
    return launch_small_mode<kForceE2M1>(x, rows, k, ldx, codes, scales, tensor_scale, stream);
  if (mode == kForceE1M2)
    return launch_small_mode<kForceE1M2>(x, rows, k, ldx, codes, scales, tensor_scale, stream);
  return launch_small_mode<kSelect>(x, rows, k, ldx, codes, scales, tensor_scale, stream);
}

bool quantize_is_small(int64_t rows, int64_t k) { return rows * k <= kSmallElems; }

hipError_t launch_quantize(const uint16_t* x, int64_t rows, int64_t k, int64_t ldx,
                           uint8_t* codes, uint8_t* scales, const float* tensor_scale, int mode,
                           hipStream_t stream) {
  if (rows * (k / kBlock) == 0) return hipSuccess;
  if (mode == kForceE2M1)
    return launch_mode<kForceE2M1>(x, rows, k, ldx, codes, scales, tensor_scale, stream);
  if (mode == kForceE1M2)
    return launch_mode<kForceE1M2>(x, rows, k, ldx, codes, scales, tensor_scale, stream);
  return launch_mode<kSelect>(x, rows, k, ldx, codes, scales, tensor_scale, stream);
}

}  // namespace mixfp4
