// MixFP4 block-scaled GEMM for gfx950: C[m, n] = s32_A s32_W sum_k a[m,k] w[n,k].
//
// Sec. 3.3 / App. B.5 decode both micro-formats into one value set (E2M2):
// E2M1 magnitudes gain a zero mantissa bit, E1M2 magnitudes go through a
// small table, T (scale bit 7) selects the path.  Here that unified value v
// is multiplied by the block's E4M3 scale s8 on the fly: s8 has at most 4
// significant bits and v at most 3, so a = s8 * v has at most 7 and lies in
// [2^-10, 3136] -- it is exact in bf16.  The bf16 operands feed
// v_mfma_f32_32x32x16_bf16 with fp32 accumulation (the accumulation format
// the paper keeps, Sec. 3.3); the per-tensor fp32 scales are applied once in
// the epilogue.  App. B.1's factored form (scale product per block) is not
// needed because the per-element decode is exact.
//
// Tiling: a 256-thread workgroup owns a 128 x 128 tile of C; its four waves
// each own 64 x 64 (2 x 2 MFMA tiles of 32 x 32).  The K loop steps over
// two 16-element scale blocks at a time: every thread decodes one block of A
// and one block of W into LDS (each element decoded once per workgroup),
// then the waves run their MFMAs from LDS.  Rows beyond m / n and blocks
// beyond k decode as zeros; stores are masked.
#include "formats.h"
#include "internal.h"

namespace mixfp4 {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kThreads = 256;
constexpr int kTileM = 128;
constexpr int kTileN = 128;
constexpr int kStepK = 32;                 // two scale blocks per K step
constexpr int kLdsPitch = kStepK + 8;      // bf16 elements per LDS row (80 bytes)

// Decode one 16-element block (8 code bytes + scale byte) to 16 bf16 values,
// packed two per dword (element 2j in the low half).
__device__ __forceinline__ void decode_block(uint2 c, uint32_t sb, uint32_t out[8]) {
  const bool t1 = (sb & 0x80u) != 0;
  const float s8 = e4m3_value(sb & 0x7Fu);
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const uint32_t byte = ((j < 4 ? c.x : c.y) >> (8 * (j & 3))) & 0xFFu;
    const uint32_t n0 = byte & 0xFu, n1 = byte >> 4;
    const float v0 = t1 ? (float)(n0 & 7u) : e2m1_value(n0 & 7u);
    const float v1 = t1 ? (float)(n1 & 7u) : e2m1_value(n1 & 7u);
    const uint32_t b0 = (__float_as_uint(s8 * v0) >> 16) | ((n0 & 8u) << 12);
    const uint32_t b1 = (__float_as_uint(s8 * v1) >> 16) | ((n1 & 8u) << 12);
    out[j] = b0 | (b1 << 16);
  }
}

__device__ __forceinline__ bf16x8 lds_frag(const uint16_t* p) {
  const uint4 v = *reinterpret_cast<const uint4*>(p);
  return __builtin_bit_cast(bf16x8, v);
}

__global__ __launch_bounds__(kThreads) void gemm_kernel(
    const uint8_t* __restrict__ a_codes, const uint8_t* __restrict__ a_scales,
    const float* __restrict__ a_ts, const uint8_t* __restrict__ w_codes,
    const uint8_t* __restrict__ w_scales, const float* __restrict__ w_ts, int64_t m,
    int64_t n, int64_t k, float* __restrict__ c) {
  __shared__ __attribute__((aligned(16))) uint16_t sa[kTileM * kLdsPitch];
  __shared__ __attribute__((aligned(16))) uint16_t sw[kTileN * kLdsPitch];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int64_t m0 = (int64_t)blockIdx.y * kTileM;
  const int64_t n0 = (int64_t)blockIdx.x * kTileN;
  const int wm = (wave >> 1) * 64, wn = (wave & 1) * 64;
  const int64_t kb_total = k / kBlock;
  const int64_t code_pitch = k / 2;

  // decode assignment: row tid/2 of the tile, block tid%2 of the K step
  const int drow = tid >> 1, dblk = tid & 1;
  const int64_t arow = m0 + drow, wrow = n0 + drow;

  f32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  for (int64_t kb = 0; kb < kb_total; kb += 2) {
    const int64_t blk = kb + dblk;
    uint32_t da[8], dw[8];
    if (arow < m && blk < kb_total) {
      const uint2 cc = *reinterpret_cast<const uint2*>(a_codes + arow * code_pitch + blk * 8);
      decode_block(cc, a_scales[arow * kb_total + blk], da);
    } else {
#pragma unroll
      for (int q = 0; q < 8; ++q) da[q] = 0u;
    }
    if (wrow < n && blk < kb_total) {
      const uint2 cc = *reinterpret_cast<const uint2*>(w_codes + wrow * code_pitch + blk * 8);
      decode_block(cc, w_scales[wrow * kb_total + blk], dw);
    } else {
#pragma unroll
      for (int q = 0; q < 8; ++q) dw[q] = 0u;
    }
    uint4* pa = reinterpret_cast<uint4*>(sa + drow * kLdsPitch + dblk * 16);
    uint4* pw = reinterpret_cast<uint4*>(sw + drow * kLdsPitch + dblk * 16);
    pa[0] = make_uint4(da[0], da[1], da[2], da[3]);
    pa[1] = make_uint4(da[4], da[5], da[6], da[7]);
    pw[0] = make_uint4(dw[0], dw[1], dw[2], dw[3]);
    pw[1] = make_uint4(dw[4], dw[5], dw[6], dw[7]);
    __syncthreads();

#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      const int koff = kk * 16 + (lane >> 5) * 8;
      bf16x8 fa[2], fw[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) fa[i] = lds_frag(sa + (wm + i * 32 + (lane & 31)) * kLdsPitch + koff);
#pragma unroll
      for (int j = 0; j < 2; ++j) fw[j] = lds_frag(sw + (wn + j * 32 + (lane & 31)) * kLdsPitch + koff);
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[i], fw[j], acc[i][j], 0, 0, 0);
    }
    __syncthreads();
  }

  const float s = (a_ts ? *a_ts : 1.0f) * (w_ts ? *w_ts : 1.0f);
  // 32 x 32 accumulator layout: lane holds column lane%32; register r holds
  // row 8*(r/4) + 4*(lane/32) + r%4.
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int64_t col = n0 + wn + j * 32 + (lane & 31);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t row = m0 + wm + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        if (row < m && col < n) c[row * n + col] = acc[i][j][r] * s;
      }
    }
}

__global__ void fill_zero(float* c, int64_t count) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < count; i += stride) c[i] = 0.0f;
}

}  // namespace

hipError_t launch_gemm(const uint8_t* a_codes, const uint8_t* a_scales, const float* a_ts,
                       const uint8_t* w_codes, const uint8_t* w_scales, const float* w_ts,
                       int64_t m, int64_t n, int64_t k, float* c, hipStream_t stream) {
  if (m == 0 || n == 0) return hipSuccess;
  if (k == 0) {
    int64_t g = (m * n + 255) / 256;
    if (g > 65536) g = 65536;
    fill_zero<<<(int)g, 256, 0, stream>>>(c, m * n);
    return hipGetLastError();
  }
  dim3 grid((unsigned)((n + kTileN - 1) / kTileN), (unsigned)((m + kTileM - 1) / kTileM));
  gemm_kernel<<<grid, kThreads, 0, stream>>>(a_codes, a_scales, a_ts, w_codes, w_scales, w_ts, m,
                                             n, k, c);
  return hipGetLastError();
}

}  // namespace mixfp4
