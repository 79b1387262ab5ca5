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

constexpr unsigned kModeFlags = MIXFP4_FORCE_E2M1 | MIXFP4_FORCE_E1M2 | MIXFP4_FOUR_SIX;

// Format mode of the flags: 0 MixFP4, 1 E2M1 only, 2 E1M2 only, 3 4/6; -1
// when more than one format flag is set.
int format_mode(unsigned flags) {
  const unsigned f = flags & kModeFlags;
  if (f == 0u) return 0;
  if (f == MIXFP4_FORCE_E2M1) return 1;
  if (f == MIXFP4_FORCE_E1M2) return 2;
  if (f == MIXFP4_FOUR_SIX) return 3;
  return -1;
}

bool valid_hadamard_block(int32_t b) {
  return b == 16 || b == 32 || b == 64 || b == 128 || b == 256;
}

int quantize_impl(const uint16_t* x, int64_t rows, int64_t k, int64_t ldx, uint8_t* codes,
                  uint8_t* scales, float* tensor_scale, unsigned flags, int32_t hadamard_block,
                  const int8_t* hadamard_signs, uint64_t seed, uint64_t offset, void* stream) {
  const unsigned known = MIXFP4_SCALE_GIVEN | kModeFlags | MIXFP4_STOCHASTIC | MIXFP4_TRANSPOSE;
  if ((flags & ~known) != 0u || format_mode(flags) < 0) return MIXFP4_ERR_FLAGS;
  const bool given = (flags & MIXFP4_SCALE_GIVEN) != 0u;
  mixfp4::QuantOptions opt;
  opt.mode = format_mode(flags);
  opt.sr = (flags & MIXFP4_STOCHASTIC) != 0u;
  opt.srp = {(uint32_t)seed, (uint32_t)(seed >> 32), (uint32_t)offset, (uint32_t)(offset >> 32)};
  const bool transpose = (flags & MIXFP4_TRANSPOSE) != 0u;
  if (rows < 0 || k < 0 || (k % mixfp4::kBlock) != 0) return MIXFP4_ERR_SHAPE;
  if (rows > 0 && (ldx < k || (ldx % 8) != 0)) return MIXFP4_ERR_SHAPE;
  if (transpose && (rows % mixfp4::kBlock) != 0) return MIXFP4_ERR_SHAPE;
  if (hadamard_block != 0) {
    // the rotation runs along the quantized dimension: k, or the rows of X
    // for a transposed quantization (there at most 64, one lane quad)
    const int64_t along = transpose ? rows : k;
    if (!valid_hadamard_block(hadamard_block) || (along % hadamard_block) != 0 ||
        (transpose && hadamard_block > 64))
      return MIXFP4_ERR_SHAPE;
    opt.had = true;
    opt.hp = mixfp4::hadamard_params(hadamard_block, hadamard_signs);
  }
  if (!tensor_scale) return MIXFP4_ERR_NULL;
  const bool empty = rows == 0 || k == 0;
  if (!empty && (!x || !codes || !scales)) return MIXFP4_ERR_NULL;
  if (!aligned(tensor_scale, 4)) return MIXFP4_ERR_ALIGN;
  if (!empty && (!aligned(x, 16) || !aligned(codes, 16))) return MIXFP4_ERR_ALIGN;
  hipStream_t s = static_cast<hipStream_t>(stream);
  (void)hipGetLastError();   // drop stale errors so a launch failure is ours
  if (transpose) {
    if (empty) {
      if (given) return MIXFP4_OK;
      return launch_status(mixfp4::launch_tensor_scale(x, 0, k, ldx, nullptr, 0, tensor_scale, s));
    }
    const int64_t nscr = rows * (k / mixfp4::kBlock);
    if (!given) {
      const hipError_t e =
          opt.had ? mixfp4::launch_tensor_scale_t_rotated(x, rows, k, ldx, opt.hp, scales, nscr,
                                                          tensor_scale, s)
                  : mixfp4::launch_tensor_scale(x, rows, k, ldx, scales, nscr, tensor_scale, s);
      const int st = launch_status(e);
      if (st != MIXFP4_OK) return st;
    }
    return launch_status(
        mixfp4::launch_quantize_t(x, rows, k, ldx, codes, scales, tensor_scale, opt, s));
  }
  if (!given && !empty && !opt.had && mixfp4::quantize_is_small(rows, k))
    return launch_status(mixfp4::launch_quantize_small(x, rows, k, ldx, codes, scales,
                                                       tensor_scale, opt, s));
  if (!given) {
    const int64_t nscr = empty ? 0 : rows * (k / mixfp4::kBlock);
    const hipError_t e =
        opt.had ? mixfp4::launch_tensor_scale_rotated(x, empty ? 0 : rows, k, ldx, opt.hp,
                                                      empty ? nullptr : scales, nscr,
                                                      tensor_scale, s)
                : mixfp4::launch_tensor_scale(x, empty ? 0 : rows, k, ldx,
                                              empty ? nullptr : scales, nscr, tensor_scale, s);
    const int st = launch_status(e);
    if (st != MIXFP4_OK) return st;
  }
  if (empty) return MIXFP4_OK;
  return launch_status(mixfp4::launch_quantize(x, rows, k, ldx, codes, scales, tensor_scale, opt, s));
}

}  // namespace

extern "C" {

int mixfp4_abi_version(void) { return MIXFP4_ABI_VERSION; }

const char* mixfp4_status_string(int status) {
  switch (status) {
    case MIXFP4_OK: return "MIXFP4_OK";
    case MIXFP4_ERR_NULL: return "MIXFP4_ERR_NULL: a required pointer is NULL";
    case MIXFP4_ERR_SHAPE: return "MIXFP4_ERR_SHAPE: bad size (negative, K % 16 != 0, ldx < K, ldx % 8 != 0, or a Hadamard block that is not 16..256 or does not divide K)";
    case MIXFP4_ERR_ALIGN: return "MIXFP4_ERR_ALIGN: pointer misaligned";
    case MIXFP4_ERR_FLAGS: return "MIXFP4_ERR_FLAGS: unknown flag bits, or more than one format mode";
    case MIXFP4_ERR_LAUNCH: return "MIXFP4_ERR_LAUNCH: kernel launch failed";
    case MIXFP4_ERR_SCRATCH: return "MIXFP4_ERR_SCRATCH: the shape needs more than the library's static workspace (mixfp4_gemm_noalloc), or its address could not be obtained";
    default: return "unknown mixfp4 status";
  }
}

const char* mixfp4_last_launch_error(void) { return g_last_launch_error; }

int mixfp4_quantize(const uint16_t* x, int64_t rows, int64_t k, int64_t ldx, uint8_t* codes,
                    uint8_t* scales, float* tensor_scale, unsigned flags, void* stream) {
  // stochastic rounding needs the seed of _ex; transposition is an _ex option
  if (flags & (MIXFP4_STOCHASTIC | MIXFP4_TRANSPOSE)) return MIXFP4_ERR_FLAGS;
  return quantize_impl(x, rows, k, ldx, codes, scales, tensor_scale, flags, 0, nullptr, 0, 0,
                       stream);
}

int mixfp4_quantize_ex(const uint16_t* x, int64_t rows, int64_t k, int64_t ldx, uint8_t* codes,
                       uint8_t* scales, float* tensor_scale, unsigned flags,
                       int32_t hadamard_block, const int8_t* hadamard_signs, uint64_t seed,
                       uint64_t offset, void* stream) {
  return quantize_impl(x, rows, k, ldx, codes, scales, tensor_scale, flags, hadamard_block,
                       hadamard_signs, seed, offset, stream);
}

int mixfp4_quantize_2d(const uint16_t* w, int64_t rows, int64_t k, int64_t ldw, uint8_t* codes,
                       uint8_t* scales, uint8_t* codes_t, uint8_t* scales_t, float* tensor_scale,
                       unsigned flags, void* stream) {
  if ((flags & ~(MIXFP4_SCALE_GIVEN | kModeFlags)) != 0u || format_mode(flags) < 0)
    return MIXFP4_ERR_FLAGS;
  const bool given = (flags & MIXFP4_SCALE_GIVEN) != 0u;
  const int mode = format_mode(flags);
  if (rows < 0 || k < 0 || (k % mixfp4::kBlock) != 0 || (rows % mixfp4::kBlock) != 0)
    return MIXFP4_ERR_SHAPE;
  if (rows > 0 && (ldw < k || (ldw % 8) != 0)) return MIXFP4_ERR_SHAPE;
  if (!tensor_scale) return MIXFP4_ERR_NULL;
  if ((codes_t == nullptr) != (scales_t == nullptr)) return MIXFP4_ERR_NULL;
  const bool empty = rows == 0 || k == 0;
  if (!empty && (!w || !codes || !scales)) return MIXFP4_ERR_NULL;
  if (!aligned(tensor_scale, 4)) return MIXFP4_ERR_ALIGN;
  if (!empty && (!aligned(w, 16) || !aligned(codes, 16) || (codes_t && !aligned(codes_t, 16))))
    return MIXFP4_ERR_ALIGN;
  hipStream_t s = static_cast<hipStream_t>(stream);
  (void)hipGetLastError();
  if (!given) {
    const int st = launch_status(mixfp4::launch_tensor_scale(
        w, empty ? 0 : rows, k, ldw, empty ? nullptr : scales,
        empty ? 0 : rows * (k / mixfp4::kBlock), tensor_scale, s));
    if (st != MIXFP4_OK) return st;
  }
  if (empty) return MIXFP4_OK;
  return launch_status(mixfp4::launch_quantize_2d(w, rows, k, ldw, codes, scales, codes_t,
                                                  scales_t, tensor_scale, mode, s));
}

int mixfp4_hadamard(const uint16_t* x, int64_t rows, int64_t k, int64_t ldx, int32_t block,
                    const int8_t* signs, uint16_t* y, void* stream) {
  if (!valid_hadamard_block(block)) return MIXFP4_ERR_SHAPE;
  if (rows < 0 || k < 0 || (k % block) != 0) return MIXFP4_ERR_SHAPE;
  if (rows > 0 && (ldx < k || (ldx % 8) != 0)) return MIXFP4_ERR_SHAPE;
  if (rows == 0 || k == 0) return MIXFP4_OK;
  if (!x || !y) return MIXFP4_ERR_NULL;
  if (!aligned(x, 16) || !aligned(y, 16)) return MIXFP4_ERR_ALIGN;
  (void)hipGetLastError();
  return launch_status(mixfp4::launch_hadamard(x, rows, k, ldx,
                                               mixfp4::hadamard_params(block, signs), y,
                                               static_cast<hipStream_t>(stream)));
}

namespace {
bool valid_variant(int32_t block, unsigned candidates) {
  return (block == 8 || block == 16 || block == 32 || block == 64) && candidates >= 1u &&
         candidates <= 7u;
}
}  // namespace

int mixfp4_quantize_variant(const uint16_t* x, int64_t rows, int64_t k, int64_t ldx, int32_t block,
                            unsigned candidates, uint8_t* codes, uint8_t* scales, uint8_t* fmt,
                            float* tensor_scale, unsigned flags, void* stream) {
  if ((flags & ~MIXFP4_SCALE_GIVEN) != 0u || candidates < 1u || candidates > 7u)
    return MIXFP4_ERR_FLAGS;
  if (!valid_variant(block, candidates)) return MIXFP4_ERR_SHAPE;
  if (rows < 0 || k < 0 || (k % block) != 0) return MIXFP4_ERR_SHAPE;
  if (rows > 0 && (ldx < k || (ldx % 8) != 0)) return MIXFP4_ERR_SHAPE;
  if (!tensor_scale) return MIXFP4_ERR_NULL;
  if (!aligned(tensor_scale, 4)) return MIXFP4_ERR_ALIGN;
  const bool empty = rows == 0 || k == 0;
  const bool three = candidates == 7u;
  if (!empty && (!x || !codes || !scales || (three && !fmt))) return MIXFP4_ERR_NULL;
  if (!empty && (!aligned(x, 16) || !aligned(codes, 16))) return MIXFP4_ERR_ALIGN;
  hipStream_t s = static_cast<hipStream_t>(stream);
  (void)hipGetLastError();
  if ((flags & MIXFP4_SCALE_GIVEN) == 0u) {
    const int st = launch_status(mixfp4::launch_tensor_scale(
        x, empty ? 0 : rows, k, ldx, empty ? nullptr : scales, empty ? 0 : rows * (k / block),
        tensor_scale, s));
    if (st != MIXFP4_OK) return st;
  }
  if (empty) return MIXFP4_OK;
  return launch_status(mixfp4::launch_quantize_variant(x, rows, k, ldx, block, candidates, codes,
                                                       scales, fmt, tensor_scale, s));
}

int mixfp4_dequantize_variant(const uint8_t* codes, const uint8_t* scales, const uint8_t* fmt,
                              const float* tensor_scale, int64_t rows, int64_t k, int32_t block,
                              unsigned candidates, float* out, void* stream) {
  if (candidates < 1u || candidates > 7u) return MIXFP4_ERR_FLAGS;
  if (!valid_variant(block, candidates)) return MIXFP4_ERR_SHAPE;
  if (rows < 0 || k < 0 || (k % block) != 0) return MIXFP4_ERR_SHAPE;
  if (rows == 0 || k == 0) return MIXFP4_OK;
  if (!codes || !scales || !out || (candidates == 7u && !fmt)) return MIXFP4_ERR_NULL;
  if (!aligned(codes, 16) || !aligned(out, 16)) return MIXFP4_ERR_ALIGN;
  if (tensor_scale && !aligned(tensor_scale, 4)) return MIXFP4_ERR_ALIGN;
  (void)hipGetLastError();
  return launch_status(mixfp4::launch_dequantize_variant(codes, scales, fmt, tensor_scale, rows, k,
                                                         block, candidates, out,
                                                         static_cast<hipStream_t>(stream)));
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

namespace {
// Argument checks shared by the GEMM entry points: MIXFP4_OK means "launch",
// kEmpty "nothing to compute" (m or n is 0), anything else is the error.
constexpr int kEmpty = -1;
int gemm_check(const uint8_t* a_codes, const uint8_t* a_scales, const float* a_tensor_scale,
               const uint8_t* w_codes, const uint8_t* w_scales, const float* w_tensor_scale,
               int64_t m, int64_t n, int64_t k, float* c) {
  if (m < 0 || n < 0 || k < 0 || (k % mixfp4::kBlock) != 0) return MIXFP4_ERR_SHAPE;
  if (m == 0 || n == 0) return kEmpty;
  if (!c) return MIXFP4_ERR_NULL;
  if (k > 0 && (!a_codes || !a_scales || !w_codes || !w_scales)) return MIXFP4_ERR_NULL;
  if (!aligned(c, 4)) return MIXFP4_ERR_ALIGN;
  if (k > 0 && (!aligned(a_codes, 16) || !aligned(w_codes, 16))) return MIXFP4_ERR_ALIGN;
  if ((a_tensor_scale && !aligned(a_tensor_scale, 4)) ||
      (w_tensor_scale && !aligned(w_tensor_scale, 4)))
    return MIXFP4_ERR_ALIGN;
  return MIXFP4_OK;
}
}  // namespace

int mixfp4_gemm(const uint8_t* a_codes, const uint8_t* a_scales, const float* a_tensor_scale,
                const uint8_t* w_codes, const uint8_t* w_scales, const float* w_tensor_scale,
                int64_t m, int64_t n, int64_t k, float* c, void* stream) {
  const int st = gemm_check(a_codes, a_scales, a_tensor_scale, w_codes, w_scales, w_tensor_scale,
                            m, n, k, c);
  if (st != MIXFP4_OK) return st == kEmpty ? MIXFP4_OK : st;
  (void)hipGetLastError();
  return launch_status(mixfp4::launch_gemm(a_codes, a_scales, a_tensor_scale, w_codes, w_scales,
                                           w_tensor_scale, m, n, k, c,
                                           static_cast<hipStream_t>(stream)));
}

int mixfp4_decode_step(const uint16_t* a, int64_t m, int64_t k, const uint8_t* w_codes,
                       const uint8_t* w_scales, const float* w_tensor_scale, int64_t n,
                       uint8_t* a_codes, uint8_t* a_scales, float* a_tensor_scale, float* c,
                       uint32_t* sync, void* stream) {
  if (!a || !w_codes || !w_scales || !a_codes || !a_scales || !a_tensor_scale || !c || !sync)
    return MIXFP4_ERR_NULL;
  if (n < 1 || !mixfp4::decode_step_applies(m, k)) return MIXFP4_ERR_SHAPE;
  if (!aligned(a, 16) || !aligned(a_codes, 16) || !aligned(a_scales, 4) || !aligned(w_scales, 4) ||
      !aligned(w_codes, 16) || !aligned(sync, 4) || !aligned(c, 4) || !aligned(a_tensor_scale, 4) ||
      (w_tensor_scale && !aligned(w_tensor_scale, 4)))
    return MIXFP4_ERR_ALIGN;
  (void)hipGetLastError();
  return launch_status(mixfp4::launch_decode_step(a, m, k, w_codes, w_scales, w_tensor_scale, n,
                                                  a_codes, a_scales, a_tensor_scale, c, sync,
                                                  static_cast<hipStream_t>(stream)));
}

int mixfp4_gemm_workspace_size(int64_t m, int64_t n, int64_t k, int64_t* bytes) {
  if (!bytes) return MIXFP4_ERR_NULL;
  if (m < 0 || n < 0 || k < 0 || (k % mixfp4::kBlock) != 0) return MIXFP4_ERR_SHAPE;
  *bytes = mixfp4::gemm_two_pass_workspace(m, n, k);
  return MIXFP4_OK;
}

int mixfp4_gemm_ws(const uint8_t* a_codes, const uint8_t* a_scales, const float* a_tensor_scale,
                   const uint8_t* w_codes, const uint8_t* w_scales, const float* w_tensor_scale,
                   int64_t m, int64_t n, int64_t k, float* c, void* workspace,
                   int64_t workspace_bytes, void* stream) {
  const int st = gemm_check(a_codes, a_scales, a_tensor_scale, w_codes, w_scales, w_tensor_scale,
                            m, n, k, c);
  if (st != MIXFP4_OK) return st == kEmpty ? MIXFP4_OK : st;
  if (workspace_bytes < 0) return MIXFP4_ERR_SHAPE;
  if (workspace && !aligned(workspace, 256)) return MIXFP4_ERR_ALIGN;
  (void)hipGetLastError();
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int64_t need = mixfp4::gemm_two_pass_workspace(m, n, k);
  if (need > 0 && workspace && workspace_bytes >= need)
    return launch_status(mixfp4::launch_gemm_two_pass(a_codes, a_scales, a_tensor_scale, w_codes,
                                                      w_scales, w_tensor_scale, m, n, k, c,
                                                      static_cast<uint8_t*>(workspace), s));
  return launch_status(mixfp4::launch_gemm(a_codes, a_scales, a_tensor_scale, w_codes, w_scales,
                                           w_tensor_scale, m, n, k, c, s));
}

int mixfp4_gemm_noalloc(const uint8_t* a_codes, const uint8_t* a_scales,
                        const float* a_tensor_scale, const uint8_t* w_codes,
                        const uint8_t* w_scales, const float* w_tensor_scale, int64_t m, int64_t n,
                        int64_t k, float* c, void* stream) {
  const int st = gemm_check(a_codes, a_scales, a_tensor_scale, w_codes, w_scales, w_tensor_scale,
                            m, n, k, c);
  if (st != MIXFP4_OK) return st == kEmpty ? MIXFP4_OK : st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int64_t need = mixfp4::gemm_two_pass_workspace(m, n, k);
  (void)hipGetLastError();
  if (need == 0)   // decode shapes and k % 32 != 0: the fused kernel, no workspace
    return launch_status(mixfp4::launch_gemm(a_codes, a_scales, a_tensor_scale, w_codes,
                                             w_scales, w_tensor_scale, m, n, k, c, s));
  if (need > mixfp4::kStaticScratchBytes) return MIXFP4_ERR_SCRATCH;
  void* ws = nullptr;
  if (mixfp4::static_scratch(&ws) != hipSuccess || !ws) return MIXFP4_ERR_SCRATCH;
  return launch_status(mixfp4::launch_gemm_two_pass(a_codes, a_scales, a_tensor_scale, w_codes,
                                                    w_scales, w_tensor_scale, m, n, k, c,
                                                    static_cast<uint8_t*>(ws), s));
}

int64_t mixfp4_gemm_noalloc_max_bytes(void) { return mixfp4::kStaticScratchBytes; }

int mixfp4_decode_operand(const uint8_t* codes, const uint8_t* scales, int64_t rows, int64_t k,
                          void* out, int64_t out_bytes, int64_t* bytes_needed, void* stream) {
  if (rows < 0 || k < 0 || (k % 32) != 0 || k > (int64_t(1) << 22)) return MIXFP4_ERR_SHAPE;
  const int64_t need = mixfp4::decoded_bytes(rows, k);
  if (bytes_needed) *bytes_needed = need;
  if (!out && out_bytes == 0) return MIXFP4_OK;        // size query
  if (rows == 0 || k == 0) return MIXFP4_OK;
  if (!codes || !scales || !out) return MIXFP4_ERR_NULL;
  if (out_bytes < need) return MIXFP4_ERR_SHAPE;
  if (!aligned(codes, 16) || !aligned(out, 256)) return MIXFP4_ERR_ALIGN;
  (void)hipGetLastError();
  return launch_status(mixfp4::launch_decode_blocked(codes, scales, rows, k,
                                                     static_cast<uint8_t*>(out),
                                                     static_cast<hipStream_t>(stream)));
}

int mixfp4_quantize_decode(const uint16_t* x, int64_t rows, int64_t k, int64_t ldx,
                           uint8_t* codes, uint8_t* scales, float* tensor_scale, void* out,
                           int64_t out_bytes, unsigned flags, void* stream) {
  if ((flags & ~(MIXFP4_SCALE_GIVEN | kModeFlags)) != 0u || format_mode(flags) < 0)
    return MIXFP4_ERR_FLAGS;
  if (rows < 0 || k < 0 || (k % 32) != 0 || k > (int64_t(1) << 22)) return MIXFP4_ERR_SHAPE;
  if (rows > 0 && (ldx < k || (ldx % 8) != 0)) return MIXFP4_ERR_SHAPE;
  if (!tensor_scale) return MIXFP4_ERR_NULL;
  if (!aligned(tensor_scale, 4)) return MIXFP4_ERR_ALIGN;
  const bool empty = rows == 0 || k == 0;
  if (!empty && (!x || !codes || !scales || !out)) return MIXFP4_ERR_NULL;
  if (!empty && out_bytes < mixfp4::decoded_bytes(rows, k)) return MIXFP4_ERR_SHAPE;
  if (!empty && (!aligned(x, 16) || !aligned(codes, 16) || !aligned(out, 256)))
    return MIXFP4_ERR_ALIGN;
  hipStream_t s = static_cast<hipStream_t>(stream);
  (void)hipGetLastError();
  if ((flags & MIXFP4_SCALE_GIVEN) == 0u) {
    const int st = launch_status(mixfp4::launch_tensor_scale(
        x, empty ? 0 : rows, k, ldx, empty ? nullptr : scales,
        empty ? 0 : rows * (k / mixfp4::kBlock), tensor_scale, s));
    if (st != MIXFP4_OK) return st;
  }
  if (empty) return MIXFP4_OK;
  return launch_status(mixfp4::launch_quantize_decode(x, rows, k, ldx, codes, scales, tensor_scale,
                                                      format_mode(flags),
                                                      static_cast<uint8_t*>(out), s));
}

int mixfp4_gemm_decoded(const void* a_decoded, const float* a_tensor_scale,
                        const void* w_decoded, const float* w_tensor_scale, int64_t m, int64_t n,
                        int64_t k, float* c, void* stream) {
  if (m < 0 || n < 0 || k < 0 || (k % 32) != 0 || k > (int64_t(1) << 22)) return MIXFP4_ERR_SHAPE;
  if (m == 0 || n == 0) return MIXFP4_OK;
  if (!c || (k > 0 && (!a_decoded || !w_decoded))) return MIXFP4_ERR_NULL;
  if (!aligned(c, 4) || (k > 0 && (!aligned(a_decoded, 256) || !aligned(w_decoded, 256))))
    return MIXFP4_ERR_ALIGN;
  if ((a_tensor_scale && !aligned(a_tensor_scale, 4)) ||
      (w_tensor_scale && !aligned(w_tensor_scale, 4)))
    return MIXFP4_ERR_ALIGN;
  (void)hipGetLastError();
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (k == 0)   // the fused path writes the zeros of an empty reduction
    return launch_status(mixfp4::launch_gemm(nullptr, nullptr, nullptr, nullptr, nullptr,
                                             nullptr, m, n, 0, c, s));
  return launch_status(mixfp4::launch_gemm_decoded(
      static_cast<const uint8_t*>(a_decoded), a_tensor_scale,
      static_cast<const uint8_t*>(w_decoded), w_tensor_scale, m, n, k, c, s));
}

}  // extern "C"
