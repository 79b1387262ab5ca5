// Internal declarations shared by the MixFP4 HIP sources (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>

namespace mixfp4 {

// Block size along the reduction dimension (App. B.1, V = 16).
constexpr int kBlock = 16;

// Stochastic rounding: Philox4x32-10 key (seed) and counter words 2-3
// (offset); words 0-1 of the counter are the block index.
struct SrParams {
  uint32_t seed_lo, seed_hi, off_lo, off_hi;
};

// Block-diagonal Hadamard rotation with blocks of b = 16 << lanes_log2.
struct HadamardParams {
  const int8_t* signs;   // b signs on the device (bit 7 set = -1), or NULL for all +1
  int lanes_log2;        // log2(b / 16), 0..4
  int odd;               // log2(b) odd: 1 / sqrt(b) is irrational
  double scale;          // 1 / sqrt(b) in fp64 (exact for even log2 b)
  double b;              // b as a double (for the midpoint decision)
};
HadamardParams hadamard_params(int b, const int8_t* signs);

// Options of one quantize call beyond the format mode.
struct QuantOptions {
  int mode = 0;              // 0 MixFP4 selection, 1 E2M1 only (NVFP4), 2 E1M2 only (INT4),
                             // 3 the 4/6 candidate set (E2M1 under max/6 or max/4)
  bool sr = false;           // stochastic rounding of the codes
  SrParams srp{};
  bool had = false;          // rotate first
  HadamardParams hp{};
};

// Workgroups of `threads` threads that the device keeps resident at once for
// `kernel` (occupancy per CU x CU count), at most max_per_cu per CU when that
// is positive.  `cache` holds one value per device (0 = not yet known);
// concurrent first calls may both query the runtime, and store the same value.
using ResidentCache = std::atomic<int64_t>[64];

template <typename Kernel>
int64_t resident_groups(Kernel kernel, ResidentCache& cache, int max_per_cu = 0,
                        int threads = 256) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 1024;
  const int64_t known = cache[dev].load(std::memory_order_relaxed);
  if (known) return known;
  int per_cu = 0, cus = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, threads, 0) != hipSuccess ||
      per_cu <= 0)
    per_cu = 4;
  if (max_per_cu > 0 && per_cu > max_per_cu) per_cu = max_per_cu;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      cus <= 0)
    cus = 256;
  const int64_t v = (int64_t)per_cu * cus;
  cache[dev].store(v, std::memory_order_relaxed);
  return v;
}

// Compute units of the current device (queried once per device; 256 if the
// query fails).
inline int64_t compute_units() {
  static std::atomic<int64_t> cache[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  const int64_t known = cache[dev].load(std::memory_order_relaxed);
  if (known) return known;
  int cus = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      cus <= 0)
    cus = 256;
  cache[dev].store(cus, std::memory_order_relaxed);
  return cus;
}

// Launchers: shapes are validated by the ABI layer before these are called.
// Tensor scale s32 = max|X| / 2688 (1.0 for all-zero X) into *tensor_scale.
// `scratch` (may be NULL) is device memory of `scratch_bytes` that the call
// may overwrite before the quantize kernel writes it (the scale-byte output).
hipError_t launch_tensor_scale(const uint16_t* x, int64_t rows, int64_t k,
                               int64_t ldx, uint8_t* scratch, int64_t scratch_bytes,
                               float* tensor_scale, hipStream_t stream);
// Tensor scale of the rotated tensor (the amax pass of a rotate-and-quantize
// call); same contract as launch_tensor_scale.
hipError_t launch_tensor_scale_rotated(const uint16_t* x, int64_t rows, int64_t k,
                                       int64_t ldx, const HadamardParams& hp,
                                       uint8_t* scratch, int64_t scratch_bytes,
                                       float* tensor_scale, hipStream_t stream);
hipError_t launch_quantize(const uint16_t* x, int64_t rows, int64_t k,
                           int64_t ldx, uint8_t* codes, uint8_t* scales,
                           const float* tensor_scale, const QuantOptions& opt,
                           hipStream_t stream);
// Tensor scale and quantization in one launch, for tensors with
// quantize_is_small(rows, k) (rows * k at most 2^18); rows, k > 0; no rotation.
bool quantize_is_small(int64_t rows, int64_t k);
hipError_t launch_quantize_small(const uint16_t* x, int64_t rows, int64_t k,
                                 int64_t ldx, uint8_t* codes, uint8_t* scales,
                                 float* tensor_scale, const QuantOptions& opt,
                                 hipStream_t stream);
// 2D (16 x 16 tile) quantization of W [n, k] (n, k multiples of 16) into
// the W layout and, when codes_t is not NULL, the W^T layout; mode as above.
hipError_t launch_quantize_2d(const uint16_t* w, int64_t n, int64_t k, int64_t ldw,
                              uint8_t* codes, uint8_t* scales, uint8_t* codes_t,
                              uint8_t* scales_t, const float* tensor_scale, int mode,
                              hipStream_t stream);
// Quantization of X^T for a row-major X [rows, k] (rows % 16 == 0): codes_t
// [k, rows/2], scales_t [k, rows/16]; rotation (opt.had) along the rows with
// b <= 64.
hipError_t launch_quantize_t(const uint16_t* x, int64_t rows, int64_t k, int64_t ldx,
                             uint8_t* codes_t, uint8_t* scales_t, const float* tensor_scale,
                             const QuantOptions& opt, hipStream_t stream);
// s32 of the rotated X^T (COMPUTE mode with opt.had and TRANSPOSE); scratch
// as for launch_tensor_scale.
hipError_t launch_tensor_scale_t_rotated(const uint16_t* x, int64_t rows, int64_t k, int64_t ldx,
                                         const HadamardParams& hp, uint8_t* scratch,
                                         int64_t scratch_bytes, float* tensor_scale,
                                         hipStream_t stream);
// Standalone rotation: y [rows, k] contiguous bf16.
hipError_t launch_hadamard(const uint16_t* x, int64_t rows, int64_t k, int64_t ldx,
                           const HadamardParams& hp, uint16_t* y, hipStream_t stream);
hipError_t launch_dequantize(const uint8_t* codes, const uint8_t* scales,
                             const float* tensor_scale, int64_t rows,
                             int64_t k, float* out, hipStream_t stream);
hipError_t launch_gemm(const uint8_t* a_codes, const uint8_t* a_scales,
                       const float* a_ts, const uint8_t* w_codes,
                       const uint8_t* w_scales, const float* w_ts, int64_t m,
                       int64_t n, int64_t k, float* c, hipStream_t stream);
// Two-pass GEMM (operands decoded once into a blocked fp16 layout in
// `workspace`, then an fp16 GEMM): applies for m > 16 and k % 32 == 0, and
// needs gemm_two_pass_workspace(m, n, k) bytes of 256-byte aligned workspace.
bool gemm_two_pass_applies(int64_t m, int64_t n, int64_t k);
int64_t gemm_two_pass_workspace(int64_t m, int64_t n, int64_t k);
hipError_t launch_gemm_two_pass(const uint8_t* a_codes, const uint8_t* a_scales, const float* a_ts,
                                const uint8_t* w_codes, const uint8_t* w_scales, const float* w_ts,
                                int64_t m, int64_t n, int64_t k, float* c, uint8_t* workspace,
                                hipStream_t stream);
// The two passes on their own: bytes of one decoded operand [rows, k]
// (rows padded to 256, k % 32 == 0), its decode, and the GEMM on two of them.
int64_t decoded_bytes(int64_t rows, int64_t k);
hipError_t launch_decode_blocked(const uint8_t* codes, const uint8_t* scales, int64_t rows,
                                 int64_t k, uint8_t* out, hipStream_t stream);
// Quantization of X [rows, k] (k % 32 == 0; s32 given on the device; `mode`
// a format mode of quant_block.h) fused with its decode into the blocked
// layout `out` (decoded_bytes(rows, k) bytes): codes and scales as
// launch_quantize writes them.
hipError_t launch_quantize_decode(const uint16_t* x, int64_t rows, int64_t k, int64_t ldx,
                                  uint8_t* codes, uint8_t* scales, const float* tensor_scale,
                                  int mode, uint8_t* out, hipStream_t stream);
hipError_t launch_gemm_decoded(const uint8_t* ablk, const float* a_ts, const uint8_t* wblk,
                               const float* w_ts, int64_t m, int64_t n, int64_t k, float* c,
                               hipStream_t stream);
// One-launch decode step (A[m, k] bf16 row-major, quantized in the launch,
// then C = A W^T): applies for 1 <= m <= 16 and k % 64 == 0 (the decode-
// shape GEMM's K split); `sync` is 4 zeroed uint32 on the device, returned
// to zero by the launch.
bool decode_step_applies(int64_t m, int64_t k);
hipError_t launch_decode_step(const uint16_t* x, int64_t m, int64_t k, const uint8_t* w_codes,
                              const uint8_t* w_scales, const float* w_ts, int64_t n,
                              uint8_t* a_codes, uint8_t* a_scales, float* a_ts, float* c,
                              uint32_t* sync, hipStream_t stream);
// Algorithm 1's selection over the candidate set `set` (bit 0 E2M1, bit 1
// E1M2 x2, bit 2 E3M0) with blocks of `block` (8, 16, 32, 64) elements along
// K; scales [rows, k/block] (T in bit 7 for two candidates), fmt [rows,
// k/block] the chosen index (may be NULL); s32 read from *tensor_scale.
hipError_t launch_quantize_variant(const uint16_t* x, int64_t rows, int64_t k, int64_t ldx,
                                   int block, unsigned set, uint8_t* codes, uint8_t* scales,
                                   uint8_t* fmt, const float* tensor_scale, hipStream_t stream);
hipError_t launch_dequantize_variant(const uint8_t* codes, const uint8_t* scales,
                                     const uint8_t* fmt, const float* tensor_scale, int64_t rows,
                                     int64_t k, int block, unsigned set, float* out,
                                     hipStream_t stream);
// The library's static workspace (mixfp4_gemm_noalloc): kStaticScratchBytes
// of device memory per GPU; *ptr receives its device address on the current
// device (looked up once per device).
constexpr int64_t kStaticScratchBytes = int64_t(64) << 20;
hipError_t static_scratch(void** ptr);

}  // namespace mixfp4
