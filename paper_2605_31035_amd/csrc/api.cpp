// C ABI of the MixFP4 library: argument checking and kernel launch order.
// Every check happens before anything is enqueued, so an error return leaves
// the caller's stream untouched.
#include "../../include/mixfp4.h"

#include <hip/hip_runtime.h>

#include "internal.h"

namespace {

thread_local const char* g_last_launch_error = "no error";

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

int launch_status(hipError_t e) {
  if (e == hipSuccess) return MIXFP4_OK;
  g_last_launch_error = hipGetErrorString(e);
  return MIXFP4_ERR_LAUNCH;
}

}  // namespace

extern "C" {

int mixfp4_abi_version(void) { return MIXFP4_ABI_VERSION; }

const char* mixfp4_status_string(int status) {
  switch (status) {
    case MIXFP4_OK: return "MIXFP4_OK";
    case MIXFP4_ERR_NULL: return "MIXFP4_ERR_NULL: a required pointer is NULL";
    case MIXFP4_ERR_SHAPE: return "MIXFP4_ERR_SHAPE: bad size (negative, K % 16 != 0, ldx < K or ldx % 8 != 0)";
    case MIXFP4_ERR_ALIGN: return "MIXFP4_ERR_ALIGN: pointer misaligned";
    case MIXFP4_ERR_FLAGS: return "MIXFP4_ERR_FLAGS: unknown flag bits or both FORCE flags";
    case MIXFP4_ERR_LAUNCH: return "MIXFP4_ERR_LAUNCH: kernel launch failed";
    default: return "unknown mixfp4 status";
  }
}

const char* mixfp4_last_launch_error(void) { return g_last_launch_error; }

int mixfp4_quantize(const uint16_t* x, int64_t rows, int64_t k, int64_t ldx, uint8_t* codes,
                    uint8_t* scales, float* tensor_scale, unsigned flags, void* stream) {
  if ((flags & ~(MIXFP4_SCALE_GIVEN | MIXFP4_FORCE_E2M1 | MIXFP4_FORCE_E1M2)) != 0u ||
      (flags & (MIXFP4_FORCE_E2M1 | MIXFP4_FORCE_E1M2)) == (MIXFP4_FORCE_E2M1 | MIXFP4_FORCE_E1M2))
    return MIXFP4_ERR_FLAGS;
  const bool given = (flags & MIXFP4_SCALE_GIVEN) != 0u;
  const int mode = (flags & MIXFP4_FORCE_E2M1) ? 1 : (flags & MIXFP4_FORCE_E1M2) ? 2 : 0;
  if (rows < 0 || k < 0 || (k % mixfp4::kBlock) != 0) return MIXFP4_ERR_SHAPE;
  if (rows > 0 && (ldx < k || (ldx % 8) != 0)) return MIXFP4_ERR_SHAPE;
  if (!tensor_scale) return MIXFP4_ERR_NULL;
  const bool empty = rows == 0 || k == 0;
  if (!empty && (!x || !codes || !scales)) return MIXFP4_ERR_NULL;
  if (!aligned(tensor_scale, 4)) return MIXFP4_ERR_ALIGN;
  if (!empty && (!aligned(x, 16) || !aligned(codes, 16))) return MIXFP4_ERR_ALIGN;
  hipStream_t s = static_cast<hipStream_t>(stream);
  (void)hipGetLastError();   // drop stale errors so a launch failure is ours
  if (!given && !empty && mixfp4::quantize_is_small(rows, k))
    return launch_status(mixfp4::launch_quantize_small(x, rows, k, ldx, codes, scales,
                                                       tensor_scale, mode, s));
  if (!given) {
    const int st = launch_status(mixfp4::launch_tensor_scale(
        x, empty ? 0 : rows, k, ldx, empty ? nullptr : scales,
        empty ? 0 : rows * (k / mixfp4::kBlock), tensor_scale, s));
    if (st != MIXFP4_OK) return st;
  }
  if (empty) return MIXFP4_OK;
  return launch_status(
      mixfp4::launch_quantize(x, rows, k, ldx, codes, scales, tensor_scale, mode, s));
}

int mixfp4_dequantize(const uint8_t* codes, const uint8_t* scales, const float* tensor_scale,
                      int64_t rows, int64_t k, float* out, void* stream) {
  if (rows < 0 || k < 0 || (k % mixfp4::kBlock) != 0) return MIXFP4_ERR_SHAPE;
  if (rows == 0 || k == 0) return MIXFP4_OK;
  if (!codes || !scales || !out) return MIXFP4_ERR_NULL;
  if (!aligned(codes, 16) || !aligned(out, 16)) return MIXFP4_ERR_ALIGN;
  if (tensor_scale && !aligned(tensor_scale, 4)) return MIXFP4_ERR_ALIGN;
  (void)hipGetLastError();
  return launch_status(mixfp4::launch_dequantize(codes, scales, tensor_scale, rows, k, out,
                                                 static_cast<hipStream_t>(stream)));
}

int mixfp4_gemm(const uint8_t* a_codes, const uint8_t* a_scales, const float* a_tensor_scale,
                const uint8_t* w_codes, const uint8_t* w_scales, const float* w_tensor_scale,
                int64_t m, int64_t n, int64_t k, float* c, void* stream) {
  if (m < 0 || n < 0 || k < 0 || (k % mixfp4::kBlock) != 0) return MIXFP4_ERR_SHAPE;
  if (m == 0 || n == 0) return MIXFP4_OK;
  if (!c) return MIXFP4_ERR_NULL;
  if (k > 0 && (!a_codes || !a_scales || !w_codes || !w_scales)) return MIXFP4_ERR_NULL;
  if (!aligned(c, 4)) return MIXFP4_ERR_ALIGN;
  if (k > 0 && (!aligned(a_codes, 16) || !aligned(w_codes, 16))) return MIXFP4_ERR_ALIGN;
  if ((a_tensor_scale && !aligned(a_tensor_scale, 4)) ||
      (w_tensor_scale && !aligned(w_tensor_scale, 4)))
    return MIXFP4_ERR_ALIGN;
  (void)hipGetLastError();
  return launch_status(mixfp4::launch_gemm(a_codes, a_scales, a_tensor_scale, w_codes, w_scales,
                                           w_tensor_scale, m, n, k, c,
                                           static_cast<hipStream_t>(stream)));
}

}  // extern "C"
