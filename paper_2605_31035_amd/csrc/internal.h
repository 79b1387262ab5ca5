// Internal declarations shared by the MixFP4 HIP sources (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mixfp4 {

// Block size along the reduction dimension (App. B.1, V = 16).
constexpr int kBlock = 16;

// Launchers: shapes are validated by the ABI layer before these are called.
// Tensor scale s32 = max|X| / 2688 (1.0 for all-zero X) into *tensor_scale.
// `scratch` (may be NULL) is device memory of `scratch_bytes` that the call
// may overwrite before the quantize kernel writes it (the scale-byte output).
hipError_t launch_tensor_scale(const uint16_t* x, int64_t rows, int64_t k,
                               int64_t ldx, uint8_t* scratch, int64_t scratch_bytes,
                               float* tensor_scale, hipStream_t stream);
// `mode`: 0 MixFP4 selection, 1 E2M1 only (NVFP4), 2 E1M2 only (INT4).
hipError_t launch_quantize(const uint16_t* x, int64_t rows, int64_t k,
                           int64_t ldx, uint8_t* codes, uint8_t* scales,
                           const float* tensor_scale, int mode, hipStream_t stream);
// Tensor scale and quantization in one launch, for tensors with
// quantize_is_small(rows, k) (rows * k at most 2^18); rows, k > 0.
bool quantize_is_small(int64_t rows, int64_t k);
hipError_t launch_quantize_small(const uint16_t* x, int64_t rows, int64_t k,
                                 int64_t ldx, uint8_t* codes, uint8_t* scales,
                                 float* tensor_scale, int mode, hipStream_t stream);
hipError_t launch_dequantize(const uint8_t* codes, const uint8_t* scales,
                             const float* tensor_scale, int64_t rows,
                             int64_t k, float* out, hipStream_t stream);
hipError_t launch_gemm(const uint8_t* a_codes, const uint8_t* a_scales,
                       const float* a_ts, const uint8_t* w_codes,
                       const uint8_t* w_scales, const float* w_ts, int64_t m,
                       int64_t n, int64_t k, float* c, hipStream_t stream);

}  // namespace mixfp4
