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
// byte.  All arithmetic that decides a code or the format bit is exact:
//   * x = fl32(X / s32) is computed as fl32(X * fl64(1/s32)); X has 8
//     significant bits, so the exact quotient is never within 2^-50 of an
//     fp32 rounding boundary while the fp64 product is within 2^-52.
//   * y = fl32(|x| / s8) likewise as fl32(|x| * fl64(1/s8)) (s8 has 4
//     significant bits); rounding y to a grid equals rounding the exact
//     quotient, because |x| sits more than half an fp32 ulp of y away from
//     every grid midpoint * s8 unless it is exactly on it.
//   * Grid rounding: E2M1 by adding and subtracting 2^22 / 2^23 / 2^24 (grid
//     spacing 0.5 / 1 / 2 below 2 / 4 / above), INT4 by rintf; both are
//     round-half-even, which is the even-code rule on these grids.
//   * The format choice compares the two squared errors through
//     sum_i (D_I - D_F) (2|x| - D_F - D_I) in fp64: every term is exact and
//     only elements whose two dequantized values differ contribute, which
//     keeps the running sum within 53 bits, so the sign is exact.
#include "formats.h"
#include "internal.h"

namespace mixfp4 {
namespace {

constexpr int kThreads = 256;

__global__ void clear_u32(uint32_t* p) { *p = 0u; }

// Max of |X| over a [rows, k] bf16 matrix (row pitch ldx), as fp32 bits.
__global__ __launch_bounds__(kThreads) void amax_kernel(const uint16_t* __restrict__ x,
                                                         int64_t rows, int64_t k, int64_t ldx,
                                                         uint32_t* __restrict__ out) {
  const int64_t vec_per_row = k >> 3;               // 8 bf16 per 16-byte vector
  const int64_t total = rows * vec_per_row;
  uint32_t m = 0u;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += stride) {
    int64_t off;
    if (ldx == k) {
      off = i << 3;
    } else {
      const int64_t r = i / vec_per_row;
      off = r * ldx + ((i - r * vec_per_row) << 3);
    }
    const uint4 v = *reinterpret_cast<const uint4*>(x + off);
    const uint32_t a = v.x & 0x7FFF7FFFu, b = v.y & 0x7FFF7FFFu;
    const uint32_t c = v.z & 0x7FFF7FFFu, d = v.w & 0x7FFF7FFFu;
    m = max(m, max(max(a & 0xFFFFu, a >> 16), max(b & 0xFFFFu, b >> 16)));
    m = max(m, max(max(c & 0xFFFFu, c >> 16), max(d & 0xFFFFu, d >> 16)));
  }
  for (int off = 32; off > 0; off >>= 1) m = max(m, (uint32_t)__shfl_xor((int)m, off));
  __shared__ uint32_t wave_max[kThreads / 64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) wave_max[wave] = m;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t r = wave_max[0];
    for (int w = 1; w < kThreads / 64; ++w) r = max(r, wave_max[w]);
    if (r) atomicMax(out, r << 16);                 // bf16 bits -> fp32 bits
  }
}

// In place: fp32 bits of max|X| -> s32 = fl32(amax / 2688), or 1.0 if zero.
__global__ void finalize_scale(uint32_t* p) {
  const float amax = __uint_as_float(*p);
  const float s = amax > 0.0f ? amax / 2688.0f : 1.0f;
  *reinterpret_cast<float*>(p) = s;
}

// E2M1 grid rounding of y >= 0: returns the 3-bit code, value in *q.
__device__ __forceinline__ uint32_t round_e2m1(float y, float* q) {
  const float c = y < 2.0f ? 0x1p22f : (y < 4.0f ? 0x1p23f : 0x1p24f);
  float r = (y + c) - c;
  r = fminf(r, 6.0f);
  *q = r;
  return r < 1.0f ? (uint32_t)(r + r) : (__float_as_uint(r) >> 22) - 252u;
}

template <bool kContig>
__global__ __launch_bounds__(kThreads) void quantize_kernel(
    const uint16_t* __restrict__ x, int64_t nbk, int64_t ldx, int64_t nblocks,
    uint8_t* __restrict__ codes, uint8_t* __restrict__ scales,
    const float* __restrict__ tensor_scale) {
  const float s32 = *tensor_scale;
  const double rs = 1.0 / (double)s32;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; g < nblocks; g += stride) {
    const uint16_t* src;
    if (kContig) {
      src = x + (g << 4);
    } else {
      const int64_t r = g / nbk;
      src = x + r * ldx + ((g - r * nbk) << 4);
    }
    const uint4 v0 = *reinterpret_cast<const uint4*>(src);
    const uint4 v1 = *reinterpret_cast<const uint4*>(src + 8);
    const uint32_t w[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};

    // |x| = fl32(|X| / s32) and the block maximum (Algorithm 1, FP8 domain).
    float ax[16];
    float bm = 0.0f;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      ax[2 * i] = (float)((double)fabsf(bf16_lo(w[i])) * rs);
      ax[2 * i + 1] = (float)((double)fabsf(bf16_hi(w[i])) * rs);
      bm = fmaxf(bm, fmaxf(ax[2 * i], ax[2 * i + 1]));
    }
    // Candidate E4M3 block scales: block-max / 6 (E2M1) and / 7 (E1M2).
    const uint32_t cf = e4m3_code(bm / 6.0f);
    const uint32_t ci = e4m3_code(bm / 7.0f);
    const float sf = e4m3_value(cf), si = e4m3_value(ci);
    const double rf = sf > 0.0f ? 1.0 / (double)sf : 0.0;
    const double ri = si > 0.0f ? 1.0 / (double)si : 0.0;

    uint32_t pf0 = 0, pf1 = 0, pi0 = 0, pi1 = 0;
    double delta = 0.0;   // Err_E2M1 - Err_E1M2 (sum form, exact)
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const double xd = (double)ax[j];
      const float yf = (float)(xd * rf);
      const float yi = (float)(xd * ri);
      float qf;
      const uint32_t codef = round_e2m1(yf, &qf);
      const float qi = fminf(rintf(yi), 7.0f);
      const float df = qf * sf, di = qi * si;          // exact in fp32
      const double t = (double)di - (double)df;
      const double u = (2.0 * xd - (double)df) - (double)di;
      delta += t * u;
      const uint32_t codei = (uint32_t)qi;
      if (j < 8) {
        pf0 |= codef << (4 * j);
        pi0 |= codei << (4 * j);
      } else {
        pf1 |= codef << (4 * (j - 8));
        pi1 |= codei << (4 * (j - 8));
      }
    }
    // Algorithm 1: keep E2M1 only if its error is strictly smaller.
    const bool t1 = !(delta < 0.0);
    // Sign bits of X into bit 3 of every nibble.
    uint32_t s0 = 0, s1 = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      s0 |= ((w[i] >> 15) & 1u) << (8 * i + 3);
      s0 |= (w[i] >> 31) << (8 * i + 7);
      s1 |= ((w[i + 4] >> 15) & 1u) << (8 * i + 3);
      s1 |= (w[i + 4] >> 31) << (8 * i + 7);
    }
    uint2 out;
    out.x = (t1 ? pi0 : pf0) | s0;
    out.y = (t1 ? pi1 : pf1) | s1;
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
                               float* tensor_scale, hipStream_t stream) {
  uint32_t* p = reinterpret_cast<uint32_t*>(tensor_scale);
  clear_u32<<<1, 1, 0, stream>>>(p);
  const int64_t total = rows * (k >> 3);
  if (total > 0) {
    int g = grid_for(total, 8);
    if (g > 2048) g = 2048;
    amax_kernel<<<g, kThreads, 0, stream>>>(x, rows, k, ldx, p);
  }
  finalize_scale<<<1, 1, 0, stream>>>(p);
  return hipGetLastError();
}

hipError_t launch_quantize(const uint16_t* x, int64_t rows, int64_t k, int64_t ldx,
                           uint8_t* codes, uint8_t* scales, const float* tensor_scale,
                           hipStream_t stream) {
  const int64_t nbk = k / kBlock;
  const int64_t nblocks = rows * nbk;
  if (nblocks == 0) return hipSuccess;
  const int g = grid_for(nblocks, 1);
  if (ldx == k)
    quantize_kernel<true><<<g, kThreads, 0, stream>>>(x, nbk, ldx, nblocks, codes, scales,
                                                       tensor_scale);
  else
    quantize_kernel<false><<<g, kThreads, 0, stream>>>(x, nbk, ldx, nblocks, codes, scales,
                                                        tensor_scale);
  return hipGetLastError();
}

}  // namespace mixfp4
