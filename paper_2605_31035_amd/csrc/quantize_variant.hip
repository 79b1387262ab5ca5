// Block-wise format selection over other FP4 candidate sets and block sizes
// (Sec. 2.3-2.4, Fig. 3; Table 5): Algorithm 1 with blocks of g = 8, 16, 32
// or 64 consecutive K elements and any non-empty subset of {E2M1, E1M2 x2,
// E3M0} as candidates, and its decode.  MixFP4 itself is the set
// {E2M1, E1M2} at g = 16; its fast kernels live in quantize.hip.
//
// Per block (one lane per block), exactly as Algorithm 1 does for its pair:
//   x = fl32(X / s32) by Markstein's division step (div_rn, exact);
//   per candidate f: s_f = FP8_E4M3(fl32(bm / Q_f)), Q = 6, 7, 16 (the
//   quotient by 6 or 7 through the exact two-term step, by 16 an exact
//   multiply; the gfx950 E4M3 converter rounds to nearest even, after a
//   clamp at 448); codes from y = fl32(|x| / s_f) (exact two-term step):
//   E2M1 by the gfx950 FP4 converter, E1M2 x2 by rint with a clamp at 7,
//   E3M0 by comparing y with the midpoints 1.5 * 2^e of its power-of-two
//   grid (exact on the fp32 bits; ties to the even code, saturating at 16);
//   the candidate with the smaller exact sum of squared errors replaces the
//   current best, ties going to the later candidate in the order E2M1, E1M2,
//   E3M0 (Algorithm 1's rule for its pair).
// The comparison of candidates b and j is the sign of
//   Err_b - Err_j = sum (D_j - D_b) (2|x| - D_b - D_j),  D = s * v,
// with every D exact in fp32 (at most 7 significant bits).  When no
// candidate scale was clamped at 448 (always so with the tensor scale
// computed: bm <= 2688), every factor, product and partial sum is exact in
// fp64 for blocks of up to 64 elements: D is a multiple of s_min / 64 below
// 1.07 bm, an element contributes only if |x| >= s_min / 8 (so its last bit
// is at least s_min 2^-27), and s_min >= bm / 17, so a term needs at most
// 44 bits and the block sum at most 50.  A clamped scale (a tensor scale
// far below max|X| / 2688 given by the caller) lets |x| outrun the scales;
// the sum is then formed from the exact split terms 2 |x| (D_j - D_b) and
// (D_j - D_b) (D_b + D_j) with error-free transformations (TwoSum into a
// compensated pair), which decides as the exact sum does unless that lies
// within about 2^-100 of zero relative to its terms.
#include "formats.h"
#include "internal.h"
#include "quant_block.h"

namespace mixfp4 {
namespace {

constexpr int kVThreads = 256;
constexpr int kFmtE2M1 = 0, kFmtE1M2 = 1, kFmtE3M0 = 2;

// E3M0 code of y >= 0: nearest of {0, 2^-2, ..., 2^4} (code p > 0 is
// 2^(p - 3)), ties to the even code, saturating at 16.  On [2^e, 2^(e+1))
// the midpoint is 1.5 * 2^e, i.e. mantissa bits 0x400000; below 1/4 the
// only candidates are 0 and 1/4, with the midpoint 1/8.
__device__ __forceinline__ uint32_t e3m0_code(float y) {
  const uint32_t b = __float_as_uint(y);
  const int e = (int)(b >> 23) - 127;
  const uint32_t m = b & 0x7FFFFFu;
  if (e < -3) return 0u;
  if (e == -3) return m != 0u ? 1u : 0u;            // (1/8, 1/4) -> 1/4; 1/8 ties to 0
  if (e >= 4) return 7u;
  const uint32_t lo = (uint32_t)(e + 3);
  const bool up = m > 0x400000u || (m == 0x400000u && (lo & 1u) != 0u);
  return lo + (up ? 1u : 0u);
}

__device__ __forceinline__ float e3m0_value(uint32_t c) {
  return c ? __uint_as_float((c + 124u) << 23) : 0.0f;   // 2^(c - 3)
}

__device__ __forceinline__ float fmt_value(int fmt, uint32_t c) {
  return fmt == kFmtE2M1 ? e2m1_value(c) : (fmt == kFmtE1M2 ? (float)c : e3m0_value(c));
}

template <int kFmt>
__device__ __forceinline__ uint32_t fmt_code(float y) {
  if constexpr (kFmt == kFmtE2M1)
    return __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(0u, y, 0.0f, 1.0f, 0) & 0xFu;
  else if constexpr (kFmt == kFmtE1M2)
    return (uint32_t)fminf(__builtin_rintf(y), 7.0f);
  else
    return e3m0_code(y);
}

// Candidate i (0-based) of the set mask: E2M1 (bit 0), E1M2 (bit 1), E3M0
// (bit 2), in that order.
template <unsigned kSet>
struct CandSet {
  static constexpr int count = (int)((kSet & 1u) + ((kSet >> 1) & 1u) + ((kSet >> 2) & 1u));
  static constexpr int fmt(int i) {
    int seen = 0;
    for (int f = 0; f < 3; ++f)
      if (kSet & (1u << f)) {
        if (seen == i) return f;
        ++seen;
      }
    return -1;
  }
};

__device__ __forceinline__ void two_sum(double a, double b, double& s, double& e) {
  s = a + b;
  const double bb = s - a;
  e = (a - (s - bb)) + (b - bb);
}

template <int kG, unsigned kSet>
__global__ __launch_bounds__(kVThreads) void quantize_variant_kernel(
    const uint16_t* __restrict__ x, int64_t nbk, int64_t ldx, int64_t nblocks,
    uint8_t* __restrict__ codes, uint8_t* __restrict__ scales, uint8_t* __restrict__ fmt_out,
    const float* __restrict__ tensor_scale) {
  using CS = CandSet<kSet>;
  constexpr int C = CS::count;
  constexpr int kW = kG / 8;                        // nibble words per block
  __shared__ ScaleRecip tab[128];
  fill_scale_table(tab);
  const float s32 = *tensor_scale;
  const bool direct = s32 >= 0x1p-90f && s32 <= 0x1p120f;
  const float xmul = direct ? 1.0f : (s32 < 1.0f ? 0x1p64f : 0x1p-64f);
  const float sx = s32 * xmul, rx = __fdiv_rn(1.0f, sx);
  const ScaleRecip d6 = scale_recip(6.0f), d7 = scale_recip(7.0f);
  __syncthreads();
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; g < nblocks; g += stride) {
    const int64_t r = g / nbk;
    const uint16_t* src = x + r * ldx + (g - r * nbk) * kG;
    float xs[kG];
    uint32_t sgn[kW];
#pragma unroll
    for (int h = 0; h < (kG + 15) / 16; ++h) {
      const uint4 v0 = *reinterpret_cast<const uint4*>(src + 16 * h);
      const uint4 v1 = kG >= 16 ? *reinterpret_cast<const uint4*>(src + 16 * h + 8)
                                : make_uint4(0, 0, 0, 0);
      float t[16];
      if (direct)
        to_fp8_domain<false>(v0, v1, 1.0f, sx, rx, t);
      else
        to_fp8_domain<true>(v0, v1, xmul, sx, rx, t);
#pragma unroll
      for (int i = 0; i < 16 && 16 * h + i < kG; ++i) xs[16 * h + i] = t[i];
      const uint32_t w[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
#pragma unroll
      for (int q = 0; q < 2 && 2 * h + q < kW; ++q) {
        uint32_t sbits = 0u;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const uint32_t wi = w[4 * q + i];
          sbits |= ((wi >> 15) & 1u) << (8 * i + 3);          // element 2i: nibble 2i, bit 3
          sbits |= (wi >> 31) << (8 * i + 7);                 // element 2i+1
        }
        sgn[2 * h + q] = sbits;
      }
    }
    float bm = 0.0f;
#pragma unroll
    for (int i = 0; i < kG; ++i) bm = fmaxf(bm, fabsf(xs[i]));

    // every candidate's scale code, scale and codes
    uint32_t sc[C];
    float sv[C];
    uint32_t cw[C][kW];
    bool clamped = false;
#pragma unroll
    for (int c = 0; c < C; ++c) {
      const int f = CS::fmt(c);
      float cand = f == kFmtE3M0 ? bm * 0.0625f
                                 : div_scale(bm, f == kFmtE2M1 ? d6.rh : d7.rh,
                                             f == kFmtE2M1 ? d6.rl : d7.rl);
      clamped |= cand > 448.0f;
      cand = fminf(cand, 448.0f);
      const s16x2 cv = __builtin_amdgcn_cvt_scalef32_pk_fp8_f32(s16x2{0, 0}, cand, 0.0f, 1.0f, false);
      sc[c] = __builtin_bit_cast(uint32_t, cv) & 0x7Fu;
      const ScaleRecip e = tab[sc[c]];
      sv[c] = e.s;
#pragma unroll
      for (int q = 0; q < kW; ++q) cw[c][q] = 0u;
#pragma unroll
      for (int i = 0; i < kG; ++i) {
        const float y = div_scale(fabsf(xs[i]), e.rh, e.rl);
        uint32_t code;
        if (f == kFmtE2M1)
          code = fmt_code<kFmtE2M1>(y);
        else if (f == kFmtE1M2)
          code = fmt_code<kFmtE1M2>(y);
        else
          code = fmt_code<kFmtE3M0>(y);
        cw[c][i >> 3] |= code << (4 * (i & 7));
      }
    }

    // the selection: the later candidate replaces the best unless it is
    // strictly worse
    int best = 0;
#pragma unroll
    for (int j = 1; j < C; ++j) {
      const int fj = CS::fmt(j);
      double hi = 0.0, lo = 0.0;
#pragma unroll
      for (int i = 0; i < kG; ++i) {
        uint32_t cb = 0u;
        float sb = 0.0f;
        int fbest = 0;
#pragma unroll
        for (int c = 0; c < C; ++c)
          if (c == best) {
            cb = (cw[c][i >> 3] >> (4 * (i & 7))) & 7u;
            sb = sv[c];
            fbest = CS::fmt(c);
          }
        const uint32_t cj = (cw[j][i >> 3] >> (4 * (i & 7))) & 7u;
        const double db = (double)(fmt_value(fbest, cb) * sb);
        const double dj = (double)(fmt_value(fj, cj) * sv[j]);
        const double f1 = dj - db;
        if (!clamped) {
          hi += f1 * ((2.0 * (double)fabsf(xs[i]) - db) - dj);
        } else {
          double s, e;
          two_sum(hi, f1 * (2.0 * (double)fabsf(xs[i])), s, e);
          lo += e;
          double s2, e2;
          two_sum(s, -(f1 * (db + dj)), s2, e2);
          lo += e2;
          hi = s2;
        }
      }
      const double delta = hi + lo;                   // Err_best - Err_j
      if (!(delta < 0.0)) best = j;
    }

    uint32_t out[kW];
    uint32_t scale_byte = 0u;
#pragma unroll
    for (int c = 0; c < C; ++c)
      if (c == best) {
#pragma unroll
        for (int q = 0; q < kW; ++q) out[q] = cw[c][q] | sgn[q];
        scale_byte = sc[c];
      }
    if (C == 2) scale_byte |= (uint32_t)best << 7;
    uint8_t* dst = codes + g * (kG / 2);
    if constexpr (kG == 8) {
      *reinterpret_cast<uint32_t*>(dst) = out[0];
    } else if constexpr (kG == 16) {
      *reinterpret_cast<uint2*>(dst) = make_uint2(out[0], out[1]);
    } else {
#pragma unroll
      for (int q = 0; q < kW; q += 4)
        *reinterpret_cast<uint4*>(dst + 4 * q) = make_uint4(out[q], out[q + 1], out[q + 2], out[q + 3]);
    }
    scales[g] = (uint8_t)scale_byte;
    if (fmt_out) fmt_out[g] = (uint8_t)best;
  }
}

// out = fl32(s32 * (s8 * v)) with v from the block's chosen candidate
// (fmt[g], else bit 7 of the scale byte for two candidates, else the only
// one); the three candidate formats in set order are packed in `fmts`.
template <int kG>
__global__ __launch_bounds__(kVThreads) void dequantize_variant_kernel(
    const uint8_t* __restrict__ codes, const uint8_t* __restrict__ scales,
    const uint8_t* __restrict__ fmt_in, const float* __restrict__ tensor_scale, int64_t nblocks,
    int ncand, int fmts, float* __restrict__ out) {
  const float s32 = tensor_scale ? *tensor_scale : 1.0f;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; g < nblocks; g += stride) {
    const uint32_t sb = scales[g];
    const int idx = fmt_in ? (int)fmt_in[g] : (ncand == 2 ? (int)(sb >> 7) : 0);
    const int f = (fmts >> (4 * idx)) & 0xF;
    const float s8 = e4m3_value(sb & 0x7Fu);
    const uint8_t* c = codes + g * (kG / 2);
    float* o = out + g * kG;
#pragma unroll
    for (int q = 0; q < kG / 8; ++q) {
      const uint32_t w = *reinterpret_cast<const uint32_t*>(c + 4 * q);
      float v[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const uint32_t nib = (w >> (4 * i)) & 0xFu;
        const float a = s32 * (s8 * fmt_value(f, nib & 7u));
        v[i] = (nib & 8u) ? -a : a;
      }
      *reinterpret_cast<float4*>(o + 8 * q) = make_float4(v[0], v[1], v[2], v[3]);
      *reinterpret_cast<float4*>(o + 8 * q + 4) = make_float4(v[4], v[5], v[6], v[7]);
    }
  }
}

unsigned grid_for(int64_t nblocks) {
  const int64_t cap = compute_units() * 8;
  int64_t g = (nblocks + kVThreads - 1) / kVThreads;
  return (unsigned)(g < cap ? g : cap);
}

template <int kG>
hipError_t launch_g(const uint16_t* x, int64_t rows, int64_t k, int64_t ldx, unsigned set,
                    uint8_t* codes, uint8_t* scales, uint8_t* fmt, const float* ts,
                    hipStream_t stream) {
  const int64_t nbk = k / kG, nblocks = rows * nbk;
  const unsigned grid = grid_for(nblocks);
#define MIXFP4_QV(S)                                                                      \
  case S:                                                                                 \
    quantize_variant_kernel<kG, S><<<grid, kVThreads, 0, stream>>>(x, nbk, ldx, nblocks, \
                                                                 codes, scales, fmt, ts); \
    break;
  switch (set) {
    MIXFP4_QV(1u) MIXFP4_QV(2u) MIXFP4_QV(3u) MIXFP4_QV(4u) MIXFP4_QV(5u) MIXFP4_QV(6u)
    MIXFP4_QV(7u)
    default: return hipErrorInvalidValue;
  }
#undef MIXFP4_QV
  return hipGetLastError();
}

}  // namespace

hipError_t launch_quantize_variant(const uint16_t* x, int64_t rows, int64_t k, int64_t ldx,
                                   int block, unsigned set, uint8_t* codes, uint8_t* scales,
                                   uint8_t* fmt, const float* tensor_scale, hipStream_t stream) {
  switch (block) {
    case 8: return launch_g<8>(x, rows, k, ldx, set, codes, scales, fmt, tensor_scale, stream);
    case 16: return launch_g<16>(x, rows, k, ldx, set, codes, scales, fmt, tensor_scale, stream);
    case 32: return launch_g<32>(x, rows, k, ldx, set, codes, scales, fmt, tensor_scale, stream);
    case 64: return launch_g<64>(x, rows, k, ldx, set, codes, scales, fmt, tensor_scale, stream);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_dequantize_variant(const uint8_t* codes, const uint8_t* scales,
                                     const uint8_t* fmt, const float* tensor_scale, int64_t rows,
                                     int64_t k, int block, unsigned set, float* out,
                                     hipStream_t stream) {
  int ncand = 0, fmts = 0;
  for (int f = 0; f < 3; ++f)
    if (set & (1u << f)) fmts |= f << (4 * ncand++);
  const int64_t nblocks = rows * (k / block);
  const unsigned grid = grid_for(nblocks);
  switch (block) {
    case 8: dequantize_variant_kernel<8><<<grid, kVThreads, 0, stream>>>(codes, scales, fmt, tensor_scale, nblocks, ncand, fmts, out); break;
    case 16: dequantize_variant_kernel<16><<<grid, kVThreads, 0, stream>>>(codes, scales, fmt, tensor_scale, nblocks, ncand, fmts, out); break;
    case 32: dequantize_variant_kernel<32><<<grid, kVThreads, 0, stream>>>(codes, scales, fmt, tensor_scale, nblocks, ncand, fmts, out); break;
    case 64: dequantize_variant_kernel<64><<<grid, kVThreads, 0, stream>>>(codes, scales, fmt, tensor_scale, nblocks, ncand, fmts, out); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace mixfp4
