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

// Exact Err_E2M1 - Err_E1M2 of one block (fp64 sum form), used only when the
// fp32 estimate is too close to zero to decide.
__device__ __attribute__((noinline)) double exact_delta(uint4 v0, uint4 v1, double rs, uint2 pf,
                                                        uint2 pi, float sf, float si) {
  const uint32_t w[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
  double d = 0.0;
  for (int j = 0; j < 16; ++j) {
    const uint32_t word = w[j >> 1];
    const float X = (j & 1) ? bf16_hi(word) : bf16_lo(word);
    const double ax = (double)(float)((double)fabsf(X) * rs);
    const uint32_t cf = (((j < 8) ? pf.x : pf.y) >> (4 * (j & 7))) & 7u;
    const uint32_t ci = (((j < 8) ? pi.x : pi.y) >> (4 * (j & 7))) & 7u;
    const double df = (double)(e2m1_value(cf) * sf);
    const double di = (double)((float)ci * si);
    d += (di - df) * ((2.0 * ax - df) - di);
  }
  return d;
}

template <bool kContig>
__global__ __launch_bounds__(kThreads) void quantize_kernel(
    const uint16_t* __restrict__ x, int64_t nbk, int64_t ldx, int64_t nblocks,
    uint8_t* __restrict__ codes, uint8_t* __restrict__ scales,
    const float* __restrict__ tensor_scale) {
  // fl64(1 / E4M3(c)) for every 7-bit code (0 for the zero scale)
  __shared__ double rcp_tab[128];
  if (threadIdx.x < 128) {
    const float v = e4m3_value(threadIdx.x);
    rcp_tab[threadIdx.x] = (threadIdx.x > 0 && threadIdx.x < 127) ? 1.0 / (double)v : 0.0;
  }
  __syncthreads();
  const float s32 = *tensor_scale;
  const double rs = 1.0 / (double)s32;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  auto block_ptr = [&](int64_t g) -> const uint16_t* {
    if (kContig) return x + (g << 4);
    const int64_t r = g / nbk;
    return x + r * ldx + ((g - r * nbk) << 4);
  };
  int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  uint4 n0 = make_uint4(0, 0, 0, 0), n1 = n0;
  if (g < nblocks) {
    const uint16_t* src = block_ptr(g);
    n0 = *reinterpret_cast<const uint4*>(src);
    n1 = *reinterpret_cast<const uint4*>(src + 8);
  }
  for (; g < nblocks; g += stride) {
    const uint4 v0 = n0, v1 = n1;
    // prefetch the next block of this thread while this one is computed
    if (g + stride < nblocks) {
      const uint16_t* src = block_ptr(g + stride);
      n0 = *reinterpret_cast<const uint4*>(src);
      n1 = *reinterpret_cast<const uint4*>(src + 8);
    }
    const uint32_t w[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};

    // x = fl32(X / s32), signed, and its fp64 copy (Algorithm 1, FP8 domain)
    float xs[16];
    double xd[16];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      xs[2 * i] = (float)((double)bf16_lo(w[i]) * rs);
      xs[2 * i + 1] = (float)((double)bf16_hi(w[i]) * rs);
    }
    float bm = 0.0f;
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      bm = fmaxf(bm, fabsf(xs[j]));
      xd[j] = (double)xs[j];
    }
    // Candidate block scales E4M3(bm/6), E4M3(bm/7).  fl32(bm * fl64(1/d))
    // equals fl32(bm / d) for d = 6, 7: the exact quotients have periodic
    // binary expansions and never sit within 2^-50 of an fp32 midpoint.
    const double bmd = (double)bm;
    const uint32_t cf = e4m3_code((float)(bmd * (1.0 / 6.0)));
    const uint32_t ci = e4m3_code((float)(bmd * (1.0 / 7.0)));
    const float sf = e4m3_value(cf), si = e4m3_value(ci);
    const double rf = rcp_tab[cf], ri = rcp_tab[ci];
    // INT4 codes cannot exceed 7 when s_I is a normal E4M3 value below the
    // maximum (then max|x| / s_I < 7.47); other blocks clamp (rare path).
    const bool clamp_i = ci < 8u || ci >= 0x7Eu;

    uint32_t pf0 = 0, pf1 = 0, pi0 = 0, pi1 = 0;
    float accf = 0.0f, acci = 0.0f;
    // Elements J, J+1 (J even): E2M1 codes via the hardware converter into
    // byte (J%8)/2 of pf, decoded back for the error; INT4 codes by adding
    // 2^23 (integer in the low bits, round half to even), accumulated into pi
    // together with a constant 0x4B000000 per code that is removed below.
#define MIXFP4_PAIR(J, PF, PI)                                                       \
  {                                                                                  \
    const float yf0 = (float)(xd[J] * rf), yf1 = (float)(xd[J + 1] * rf);            \
    const float yi0 = fabsf((float)(xd[J] * ri)), yi1 = fabsf((float)(xd[J + 1] * ri)); \
    PF = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(PF, yf0, yf1, 1.0f, ((J) & 7) >> 1);  \
    const f32x2 qf = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(PF, 1.0f, ((J) & 7) >> 1); \
    const float rf0 = yf0 - qf.x, rf1 = yf1 - qf.y;                                  \
    accf = __builtin_fmaf(rf0, rf0, accf);                                           \
    accf = __builtin_fmaf(rf1, rf1, accf);                                           \
    const uint32_t b0 = __float_as_uint(yi0 + 0x1p23f);                              \
    const uint32_t b1 = __float_as_uint(yi1 + 0x1p23f);                              \
    const float ri0 = yi0 - (__uint_as_float(b0) - 0x1p23f);                         \
    const float ri1 = yi1 - (__uint_as_float(b1) - 0x1p23f);                         \
    acci = __builtin_fmaf(ri0, ri0, acci);                                           \
    acci = __builtin_fmaf(ri1, ri1, acci);                                           \
    PI += b0 << (4 * ((J) & 7));                                                     \
    PI += b1 << (4 * (((J) + 1) & 7));                                               \
  }
    MIXFP4_PAIR(0, pf0, pi0)
    MIXFP4_PAIR(2, pf0, pi0)
    MIXFP4_PAIR(4, pf0, pi0)
    MIXFP4_PAIR(6, pf0, pi0)
    MIXFP4_PAIR(8, pf1, pi1)
    MIXFP4_PAIR(10, pf1, pi1)
    MIXFP4_PAIR(12, pf1, pi1)
    MIXFP4_PAIR(14, pf1, pi1)
#undef MIXFP4_PAIR
    pi0 -= kMagicPack;
    pi1 -= kMagicPack;
    if (clamp_i) {
      // Subnormal or saturated s_I: codes above 7 are possible; redo the
      // INT4 branch with saturation.
      pi0 = pi1 = 0u;
      acci = 0.0f;
      for (int j = 0; j < 16; ++j) {
        const float yi = fabsf((float)(xd[j] * ri));
        const float q = fminf(rintf(yi), 7.0f);
        const float r = yi - q;
        acci = __builtin_fmaf(r, r, acci);
        if (j < 8) pi0 |= (uint32_t)q << (4 * j);
        else pi1 |= (uint32_t)q << (4 * (j - 8));
      }
    }

    // Err_E2M1 - Err_E1M2 ~= sf^2 * sum rf^2 - si^2 * sum ri^2.  Each r is off
    // by at most 7.5 * 2^-24 (y is a correctly rounded quotient), so each sum
    // is within 2^-15 of its exact value; tau covers that with margin.  Inside
    // tau the exact fp64 sum decides.
    const float sf2 = sf * sf, si2 = si * si;
    const float est = sf2 * accf - si2 * acci;
    const float tau = sf2 * (0x1p-13f + 0x1p-20f * accf) + si2 * (0x1p-13f + 0x1p-20f * acci);
    // A zero candidate scale makes that branch's error sum(x^2), which the
    // estimate does not model: such blocks (max below 7 * 2^-10 in the FP8
    // domain) take the exact path too.
    bool t1;
    if (cf != 0u && ci != 0u && fabsf(est) > tau) {
      t1 = !(est < 0.0f);
    } else {
      t1 = !(exact_delta(v0, v1, rs, make_uint2(pf0, pf1), make_uint2(pi0, pi1), sf, si) < 0.0);
    }
    // Sign of X into bit 3 of every nibble: the E2M1 codes already carry it.
    uint2 out;
    out.x = t1 ? (pi0 | (pf0 & 0x88888888u)) : pf0;
    out.y = t1 ? (pi1 | (pf1 & 0x88888888u)) : pf1;
    *reinterpret_cast<uint2*>(codes + (g << 3)) = out;
    scales[g] = (uint8_t)(t1 ? (0x80u | ci) : cf);
  }
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

hipError_t launch_quantize(const uint16_t* x, int64_t rows, int64_t k, int64_t ldx,
                           uint8_t* codes, uint8_t* scales, const float* tensor_scale,
                           hipStream_t stream) {
  const int64_t nbk = k / kBlock;
  const int64_t nblocks = rows * nbk;
  if (nblocks == 0) return hipSuccess;
  // Enough workgroups to keep ~8 per CU resident; beyond that each thread
  // walks several blocks (amortising its set-up, prefetching the next one).
  int64_t per_thread = nblocks / (2048LL * kThreads);
  per_thread = per_thread < 1 ? 1 : (per_thread > 8 ? 8 : per_thread);
  const int g = grid_for(nblocks, (int)per_thread);
  if (ldx == k)
    quantize_kernel<true><<<g, kThreads, 0, stream>>>(x, nbk, ldx, nblocks, codes, scales,
                                                       tensor_scale);
  else
    quantize_kernel<false><<<g, kThreads, 0, stream>>>(x, nbk, ldx, nblocks, codes, scales,
                                                        tensor_scale);
  return hipGetLastError();
}

}  // namespace mixfp4
