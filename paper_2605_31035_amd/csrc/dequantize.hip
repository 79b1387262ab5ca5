// MixFP4 -> fp32 decode (App. B.2-B.3): value = s32 * (E4M3(scale) * v) * sign,
// v from the E2M1 grid when scale bit 7 (T) is 0 and from the INT4 grid
// {0..7} (E1M2 x2) when it is 1.  E4M3 * v is exact in fp32, so every output
// is rounded once.  One lane decodes one 16-element block.
#include "formats.h"
#include "internal.h"

namespace mixfp4 {
namespace {

constexpr int kThreads = 256;

__global__ __launch_bounds__(kThreads) void dequantize_kernel(
    const uint8_t* __restrict__ codes, const uint8_t* __restrict__ scales,
    const float* __restrict__ tensor_scale, int64_t nblocks, float* __restrict__ out) {
  const float s32 = tensor_scale ? *tensor_scale : 1.0f;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; g < nblocks; g += stride) {
    const uint2 c = *reinterpret_cast<const uint2*>(codes + (g << 3));
    const uint32_t sb = scales[g];
    const bool t1 = (sb & 0x80u) != 0;
    const float s8 = e4m3_value(sb & 0x7Fu);
    float vals[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const uint32_t nib = ((j < 8 ? c.x : c.y) >> (4 * (j & 7))) & 0xFu;
      const uint32_t mag = nib & 7u;
      const float v = t1 ? (float)mag : e2m1_value(mag);
      const float a = s32 * (s8 * v);
      vals[j] = (nib & 8u) ? -a : a;
    }
    float4* dst = reinterpret_cast<float4*>(out + (g << 4));
#pragma unroll
    for (int q = 0; q < 4; ++q)
      dst[q] = make_float4(vals[4 * q], vals[4 * q + 1], vals[4 * q + 2], vals[4 * q + 3]);
  }
}

}  // namespace

hipError_t launch_dequantize(const uint8_t* codes, const uint8_t* scales,
                             const float* tensor_scale, int64_t rows, int64_t k, float* out,
                             hipStream_t stream) {
  const int64_t nblocks = rows * (k / kBlock);
  if (nblocks == 0) return hipSuccess;
  int64_t g = (nblocks + kThreads - 1) / kThreads;
  if (g > 65536) g = 65536;
  dequantize_kernel<<<(int)g, kThreads, 0, stream>>>(codes, scales, tensor_scale, nblocks, out);
  return hipGetLastError();
}

}  // namespace mixfp4
