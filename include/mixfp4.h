/*
 * mixfp4.h - C ABI of the MixFP4 quantizer, dequantizer and block-scaled GEMM
 * for AMD Instinct MI355X (gfx950).
 *
 * MixFP4 (Sec. 3.2 of the paper) stores a tensor as
 *   - 4-bit codes [s | p2 p1 p0] (App. B.2), two per byte, element 2j in the
 *     low nibble of byte j; one row of K elements takes K/2 bytes;
 *   - one scale byte per 16 consecutive elements along K (App. B.1, V = 16):
 *     bits 6:0 are an unsigned E4M3 (OCP E4M3FN) magnitude, bit 7 is the
 *     format type T (App. B.3): T = 0 -> the block's codes are E2M1
 *     (magnitudes {0,.5,1,1.5,2,3,4,6}), T = 1 -> E1M2 read through the x2
 *     INT4 remap (magnitudes {0,...,7}) (Sec. 3.1, App. B.2);
 *   - one fp32 per-tensor scale s32 (Sec. 2.1, Algorithm 1).
 * An element decodes to s32 * E4M3(scale & 0x7F) * v(code, T) * sign.
 *
 * General conventions for every entry point:
 *   - Every pointer argument is DEVICE memory owned by the caller.  The
 *     library never allocates, frees or synchronizes; it only enqueues
 *     kernels on `stream` (a hipStream_t; NULL means the default stream).
 *   - Arguments are checked on the host before anything is enqueued; on any
 *     error the function returns a nonzero mixfp4_status and the stream is
 *     left untouched.  A failed kernel launch returns MIXFP4_ERR_LAUNCH.
 *     Faults inside kernels surface at the caller's next synchronization.
 *   - Outputs must not alias inputs.  Calls are reentrant; calls that write
 *     the same outputs from different streams race.
 *   - Inputs must be finite (bf16 NaN / Inf are outside the contract).
 *   - Matrices are row-major.  Scale rows are K/16 bytes, code rows K/2
 *     bytes, both contiguous (no padding between rows).
 */
#ifndef MIXFP4_H
#define MIXFP4_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  MIXFP4_OK = 0,
  MIXFP4_ERR_NULL = 1,    /* a required pointer is NULL                      */
  MIXFP4_ERR_SHAPE = 2,   /* negative size, K % 16 != 0, ldx < K, ldx % 8,
                             or a bad Hadamard block size                 */
  MIXFP4_ERR_ALIGN = 3,   /* a pointer misses its required alignment         */
  MIXFP4_ERR_FLAGS = 4,   /* unknown flag bits                               */
  MIXFP4_ERR_LAUNCH = 5,  /* the HIP runtime rejected a kernel launch        */
  MIXFP4_ERR_SCRATCH = 6  /* mixfp4_gemm_noalloc: static workspace too small  */
} mixfp4_status;

/* Tensor-scale modes of mixfp4_quantize (flags argument). */
#define MIXFP4_SCALE_COMPUTE 0u /* compute s32 = max|X| / 2688 on the device  */
#define MIXFP4_SCALE_GIVEN 1u   /* read s32 from *tensor_scale                */
/* Format modes (OR-ed with one of the above; at most one of them).  Each
 * takes one branch of Algorithm 1 for every block, with the tensor scale,
 * rounding and packing unchanged, and sets T accordingly, so dequantize and
 * GEMM read the result like any MixFP4 tensor:                             */
#define MIXFP4_FORCE_E2M1 2u    /* E2M1 only (T = 0): NVFP4 (Sec. 2.1)        */
#define MIXFP4_FORCE_E1M2 4u    /* E1M2 x2 only (T = 1): INT4 codes           */
/* The 4/6 candidate set the paper compares against (Sec. 2.3, Sec. 4.2):
 * E2M1 under the block scale E4M3(max/6) or E4M3(max/4), whichever has the
 * smaller squared error (ties keep max/6); T = 0, i.e. plain NVFP4.        */
#define MIXFP4_FOUR_SIX 32u
/* Stochastic rounding of the codes (App. D); mixfp4_quantize_ex only.      */
#define MIXFP4_STOCHASTIC 8u
/* Quantize X^T (blocks of 16 consecutive rows of X); mixfp4_quantize_ex only.*/
#define MIXFP4_TRANSPOSE 16u

/*
 * mixfp4_quantize - Algorithm 1 ("MixFP4 data type quantization") on a bf16
 * matrix X [rows, k] with row pitch ldx elements.
 *
 * For each row and each block of 16 consecutive elements along k it computes
 * x = X / s32 in fp32 (the "FP8 domain"), the block maximum |x|, the two E4M3
 * candidate scales E4M3(max/6) and E4M3(max/7), quantizes the block to the
 * E2M1 grid and to the E1M2 (x2, INT4) grid, keeps E2M1 when its squared
 * error is strictly smaller and E1M2 otherwise (ties pick E1M2), stores T in
 * bit 7 of the scale byte and packs the codes (Sec. 3.2, App. B.3).  Rounding
 * is to nearest with ties to the even code, saturating; a code's sign bit is
 * the sign bit of X (also for a zero magnitude).  The result is bit-identical
 * to the CPU oracle and deterministic.
 *
 *   x            bf16 bit patterns, rows x ldx, 16-byte aligned; only the
 *                first k of each row are read.  ldx >= k, ldx % 8 == 0.
 *   rows, k      rows >= 0, k >= 0, k % 16 == 0.  rows * k == 0 writes no
 *                codes (and s32 = 1.0 in COMPUTE mode).
 *   codes        out, rows * k/2 bytes, 16-byte aligned.
 *   scales       out, rows * k/16 bytes, any alignment.
 *   tensor_scale 1 float, 4-byte aligned.  COMPUTE: written with
 *                fl32(max|X| / 2688), or 1.0f if X is all zero (Algorithm 1).
 *                GIVEN: read; must be finite and > 0.
 *   flags        MIXFP4_SCALE_COMPUTE or MIXFP4_SCALE_GIVEN, optionally OR-ed
 *                with one of MIXFP4_FORCE_E2M1 / MIXFP4_FORCE_E1M2 /
 *                MIXFP4_FOUR_SIX; any other bit (MIXFP4_STOCHASTIC and
 *                MIXFP4_TRANSPOSE included: they are mixfp4_quantize_ex
 *                options), or two format flags, returns MIXFP4_ERR_FLAGS.
 */
int mixfp4_quantize(const uint16_t *x, int64_t rows, int64_t k, int64_t ldx,
                    uint8_t *codes, uint8_t *scales, float *tensor_scale,
                    unsigned flags, void *stream);

/*
 * mixfp4_quantize_ex - mixfp4_quantize with the two steps the paper's FP4
 * training recipe puts around the quantizer (Sec. 3.2, Fig. 7; Sec. 4.3):
 * an optional random Hadamard rotation of X first, and optional stochastic
 * rounding of the codes (App. D).  With hadamard_block == 0 and without
 * MIXFP4_STOCHASTIC it is mixfp4_quantize.
 *
 *   x ... tensor_scale  as for mixfp4_quantize; with a rotation, COMPUTE
 *                mode takes s32 from the rotated tensor (two passes over X).
 *   flags        as for mixfp4_quantize, plus MIXFP4_STOCHASTIC and
 *                MIXFP4_TRANSPOSE.
 *   hadamard_block  0 (no rotation) or b in {16, 32, 64, 128, 256} with
 *                k % b == 0: X is first replaced by the bf16 result of
 *                mixfp4_hadamard(X, b, hadamard_signs), bit for bit, and
 *                that tensor is quantized.  Anything else: MIXFP4_ERR_SHAPE.
 *
 * MIXFP4_TRANSPOSE quantizes X^T (the operands of the weight-gradient GEMM
 * dW = dY^T X, which reduces over the token rows): the result is exactly
 * that of this call on the contiguous transpose of X [rows, k] (rotation,
 * rounding, stochastic draws and s32 included), without forming it.  Then
 * rows % 16 == 0, codes is [k, rows/2] and scales is [k, rows/16]; a rotation
 * runs along the rows and needs b <= 64 with rows % b == 0.
 *   hadamard_signs  device array of b bytes (bit 7 set = -1) or NULL.
 *   seed, offset Philox4x32-10 (Salmon et al., SC 2011) key and the high
 *                64 bits of its counter; block g = row * k/16 + column block
 *                takes counter (g, offset), and element j of the block the
 *                draw u = byte j % 4 of output word j / 4 (least significant
 *                first).  Ignored without MIXFP4_STOCHASTIC.
 *
 * Stochastic rounding replaces only the codes of the branch Algorithm 1
 * chose (scales, T and s32 are those of round-to-nearest, so the choice is
 * independent of the draws).  For the fp32 quotient y = |x| / s8 between
 * grid neighbours lo <= y < lo + d, the code is that of the nearer of lo and
 * lo + d to y + (eps - 1/2) d, ties to the even code, with
 * eps = (u + 1/2) / 256 for X >= 0 and (255 - u + 1/2) / 256 for X < 0 (App.
 * D's round(q + eps - 1/2) on the signed quotient); y at or above the
 * largest grid value gives that value.  Deterministic for a given seed and
 * offset, and bit-identical to the CPU oracle.
 */
int mixfp4_quantize_ex(const uint16_t *x, int64_t rows, int64_t k, int64_t ldx,
                       uint8_t *codes, uint8_t *scales, float *tensor_scale,
                       unsigned flags, int32_t hadamard_block,
                       const int8_t *hadamard_signs, uint64_t seed,
                       uint64_t offset, void *stream);

/*
 * mixfp4_quantize_2d - 2D block quantization of a weight W [rows, k], as the
 * FP4 training recipe the paper follows does for weights (Sec. 3.2, Fig. 7;
 * Sec. 4.3): Algorithm 1 with the block being a 16 x 16 tile of W (one
 * block maximum, one pair of candidate scales, one error comparison over the
 * 256 elements, one T); the tensor scale as in mixfp4_quantize.  The result
 * is written in the MixFP4 layout of W and, if codes_t is not NULL, of W^T:
 *   codes [rows, k/2], scales [rows, k/16]    (each tile's scale byte on
 *                                              each of its 16 rows)
 *   codes_t [k, rows/2], scales_t [k, rows/16]
 * so FPROP (A W^T: mixfp4_gemm(A, W)) and DGRAD (dY W: mixfp4_gemm(dY, W^T))
 * read the same quantized values.  rows % 16 == 0, k % 16 == 0, ldw as ldx
 * of mixfp4_quantize; codes and codes_t 16-byte aligned; codes_t and
 * scales_t both NULL or both given.  flags: MIXFP4_SCALE_COMPUTE/GIVEN and
 * at most one of FORCE_E2M1 / FORCE_E1M2 / FOUR_SIX.  Bit-identical to the CPU oracle.
 */
int mixfp4_quantize_2d(const uint16_t *w, int64_t rows, int64_t k, int64_t ldw,
                       uint8_t *codes, uint8_t *scales, uint8_t *codes_t,
                       uint8_t *scales_t, float *tensor_scale, unsigned flags,
                       void *stream);

/*
 * mixfp4_hadamard - block-diagonal (random) Hadamard transform along k, the
 * rotation applied before quantization in the paper's training recipe (RHT,
 * Sec. 3.2 / Fig. 7) and in its rotated PTQ runs (Sec. 4.2):
 *   y[r, c b + j] = sum_i s_i x[r, c b + i] H_b[i, j] / sqrt(b),
 * H_b the Sylvester Hadamard matrix (entry (-1)^popcount(i & j)), s_i = -1
 * where bit 7 of signs[i] is set, +1 otherwise (all +1 for signs == NULL).
 * Each output is the exact value rounded once to bf16 (nearest, ties to
 * even; Inf on overflow; an exactly zero result is +0), provided the nonzero
 * inputs of each b-block span at most a factor 2^(45 - log2 b) in magnitude
 * (2^37 at b = 256), which keeps every fp64 partial sum exact; beyond that
 * the sums are fp64 with their rounding.
 *
 *   x        bf16 [rows, k], row pitch ldx (>= k, % 8 == 0), 16-byte aligned.
 *   block    b in {16, 32, 64, 128, 256}, k % b == 0 (else MIXFP4_ERR_SHAPE).
 *   signs    device array of b bytes, or NULL.
 *   y        out, bf16 [rows, k] contiguous, 16-byte aligned, not aliasing x.
 */
int mixfp4_hadamard(const uint16_t *x, int64_t rows, int64_t k, int64_t ldx,
                    int32_t block, const int8_t *signs, uint16_t *y,
                    void *stream);

/*
 * mixfp4_dequantize - decode MixFP4 back to fp32 (App. B.2-B.3):
 *   out[r, i] = fl32(s32 * (E4M3(scale & 0x7F) * v(code, T))) * sign,
 * where the inner product is exact, so each output is rounded once.
 *
 *   codes, scales  as written by mixfp4_quantize for a [rows, k] matrix
 *                  (codes 16-byte aligned).
 *   tensor_scale   1 float (4-byte aligned), or NULL for 1.0 (the output is
 *                  then in Algorithm 1's FP8 domain).
 *   rows, k        rows >= 0, k >= 0, k % 16 == 0.
 *   out            out, rows * k floats, contiguous, 16-byte aligned.
 */
int mixfp4_dequantize(const uint8_t *codes, const uint8_t *scales,
                      const float *tensor_scale, int64_t rows, int64_t k,
                      float *out, void *stream);

/*
 * mixfp4_quantize_variant - the block-wise format selection of Algorithm 1
 * over another FP4 candidate set or block size, as the paper's ablations
 * study it (Sec. 2.3-2.4 and Fig. 3: the sets {E2M1}, {E2M1, E1M2},
 * {E2M1, E1M2, E3M0}; Table 5: block sizes 8, 16, 32, 64).  The tensor scale
 * and FP8 domain are Algorithm 1's (s32 = max|X| / 2688); each block of
 * `block` consecutive K elements takes, per candidate f, the E4M3 scale
 * FP8_E4M3(bm / Q_f) (Q = 6 for E2M1, 7 for E1M2 x2, 16 for E3M0), rounds
 * |x| / s_f to f's grid (nearest, ties to the even code, saturating), and
 * keeps the candidate with the smallest exact squared error, ties going to
 * the later candidate in the order E2M1, E1M2, E3M0 (so {E2M1, E1M2} at
 * block 16 is mixfp4_quantize's MixFP4, bit for bit).  E3M0 is the FP4
 * format with three exponent bits and bias 3: code p > 0 is 2^(p - 3), so
 * its grid is {0, 1/4, 1/2, 1, 2, 4, 8, 16}.
 *
 *   x, rows, k, ldx  as for mixfp4_quantize, with k % block == 0.
 *   block            8, 16, 32 or 64 (else MIXFP4_ERR_SHAPE).
 *   candidates       non-empty OR of MIXFP4_CAND_E2M1 / _E1M2 / _E3M0
 *                    (else MIXFP4_ERR_FLAGS).
 *   codes            out, [rows, k/2], nibble [sign | 3-bit code] as in
 *                    MixFP4, 16-byte aligned.
 *   scales           out, [rows, k/block]: the chosen candidate's E4M3 code in
 *                    bits 6:0; bit 7 is the chosen index for two candidates
 *                    (T, as in MixFP4) and 0 otherwise.
 *   fmt              out, [rows, k/block] chosen candidate index (0-based in
 *                    the order above), or NULL; required with all three
 *                    candidates (two bits do not fit the scale byte).
 *   tensor_scale, flags  as for mixfp4_quantize (MIXFP4_SCALE_COMPUTE or
 *                    MIXFP4_SCALE_GIVEN only).
 */
#define MIXFP4_CAND_E2M1 1u
#define MIXFP4_CAND_E1M2 2u
#define MIXFP4_CAND_E3M0 4u
int mixfp4_quantize_variant(const uint16_t *x, int64_t rows, int64_t k, int64_t ldx,
                            int32_t block, unsigned candidates, uint8_t *codes,
                            uint8_t *scales, uint8_t *fmt, float *tensor_scale,
                            unsigned flags, void *stream);

/*
 * mixfp4_dequantize_variant - decode mixfp4_quantize_variant's output:
 * out = fl32(s32 * (E4M3(scale & 0x7F) * v)) * sign with v from the block's
 * chosen candidate (fmt if given, else bit 7 of the scale byte for two
 * candidates, else the only one).  Arguments as for the quantizer; out is
 * rows * k floats, contiguous, 16-byte aligned; tensor_scale NULL means 1.0.
 */
int mixfp4_dequantize_variant(const uint8_t *codes, const uint8_t *scales,
                              const uint8_t *fmt, const float *tensor_scale,
                              int64_t rows, int64_t k, int32_t block,
                              unsigned candidates, float *out, void *stream);

/*
 * mixfp4_gemm - C[m, n] = sum_k A[m, k] * W[n, k] for two MixFP4 operands
 * (C = A W^T, both quantized along the reduction dimension K, App. B.1).
 * Each element is decoded through the unified E2M2 value set (Sec. 3.3,
 * App. B.5) to the 16-bit value E4M3 * v, the products accumulate in fp32 on
 * the matrix cores, and the epilogue multiplies by s32_A * s32_W.  The
 * decoded value has at most 7 significant bits (4 of the E4M3 scale, 3 of v)
 * and lies in [2^-10, 3136], so it is exact in fp16 and in bf16 alike; the
 * kernels feed fp16 operands to the fp16 matrix instructions.
 * Accuracy: |C - C_exact| <= 1e-5 * sum_k |A_hat * W_hat| + 1e-6, where
 * A_hat, W_hat are the exactly dequantized operands.
 *
 *   a_codes [m, k/2], a_scales [m, k/16], a_tensor_scale (NULL = 1.0)
 *   w_codes [n, k/2], w_scales [n, k/16], w_tensor_scale (NULL = 1.0)
 *   m, n, k        >= 0, k % 16 == 0; k == 0 writes zeros.
 *   c              out, m * n floats, row-major, 4-byte aligned.
 *   Code pointers 16-byte aligned; scale pointers any alignment.
 */
int mixfp4_gemm(const uint8_t *a_codes, const uint8_t *a_scales,
                const float *a_tensor_scale, const uint8_t *w_codes,
                const uint8_t *w_scales, const float *w_tensor_scale,
                int64_t m, int64_t n, int64_t k, float *c, void *stream);

/*
 * mixfp4_gemm_ws - mixfp4_gemm with caller-supplied device workspace, for the
 * compute-bound shapes.  The result satisfies the same accuracy bound as
 * mixfp4_gemm (every product is of the same exactly decoded operands, only
 * the fp32 summation order differs).
 *
 * With m > 16, k % 32 == 0, k <= 2^22 and workspace_bytes at least
 * mixfp4_gemm_workspace_size(m, n, k), the call runs two passes: each
 * operand's elements are decoded once (Sec. 3.3 / App. B.5: T selects the
 * E2M1 or E1M2 x2 value, times the E4M3 block scale, exactly) into 16-bit
 * values in the workspace, in a blocked layout private to the library; then
 * a GEMM on those values accumulates in fp32 on the matrix cores and applies
 * s32_A * s32_W in the epilogue (App. B.1).  Otherwise (decode-shape m,
 * k % 32 != 0, or too little workspace) it computes exactly what mixfp4_gemm
 * computes, without touching the workspace.
 *
 *   a_codes ... c      as for mixfp4_gemm.
 *   workspace          device memory, 256-byte aligned (MIXFP4_ERR_ALIGN
 *                      otherwise), or NULL; its contents on entry are
 *                      ignored and on return are unspecified.  Calls that
 *                      share a workspace must be ordered (same stream).
 *   workspace_bytes    its size; < 0 is MIXFP4_ERR_SHAPE.
 */
int mixfp4_gemm_ws(const uint8_t *a_codes, const uint8_t *a_scales,
                   const float *a_tensor_scale, const uint8_t *w_codes,
                   const uint8_t *w_scales, const float *w_tensor_scale,
                   int64_t m, int64_t n, int64_t k, float *c, void *workspace,
                   int64_t workspace_bytes, void *stream);

/*
 * mixfp4_gemm_noalloc - mixfp4_gemm_ws for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, hosts
 * that forbid allocation): the workspace is the library's own static device
 * array of mixfp4_gemm_noalloc_max_bytes() bytes (64 MiB), which each GPU the
 * library runs on holds until the process ends.  The call itself allocates
 * nothing.  Where mixfp4_gemm_ws would take the two-pass path the shape's
 * workspace (mixfp4_gemm_workspace_size) must fit in that array, else
 * MIXFP4_ERR_SCRATCH is returned and nothing is enqueued; decode shapes and
 * k % 32 != 0 run the fused kernel as mixfp4_gemm does.  The result equals
 * mixfp4_gemm_ws's bit for bit.  Every call on a GPU shares that GPU's
 * array, and calls whose work overlaps in time on one GPU (different
 * streams, or threads without ordering) race on it; calls ordered on one
 * stream do not.  `stream` must belong to the calling thread's current
 * device.
 */
int mixfp4_gemm_noalloc(const uint8_t *a_codes, const uint8_t *a_scales,
                        const float *a_tensor_scale, const uint8_t *w_codes,
                        const uint8_t *w_scales, const float *w_tensor_scale,
                        int64_t m, int64_t n, int64_t k, float *c, void *stream);
int64_t mixfp4_gemm_noalloc_max_bytes(void);

/*
 * mixfp4_gemm_workspace_size - bytes of workspace with which mixfp4_gemm_ws
 * takes the two-pass path for this shape: 2 * k * (m + n) rounded up to
 * whole 256-row tiles of A and of W, or 0 where that path does not apply.
 * Host-only; *bytes is written on MIXFP4_OK.  Negative sizes or k % 16 != 0:
 * MIXFP4_ERR_SHAPE; bytes == NULL: MIXFP4_ERR_NULL.
 */
int mixfp4_gemm_workspace_size(int64_t m, int64_t n, int64_t k, int64_t *bytes);

/*
 * The two passes of mixfp4_gemm_ws as separate calls, so that an operand
 * used by several GEMMs (activations against several weights) is decoded
 * once, and each pass can be timed on its own.
 *
 * mixfp4_decode_operand - decode a MixFP4 operand [rows, k] (codes, scales
 * as written by mixfp4_quantize) into the 16-bit values E4M3 * v(code, T)
 * (Sec. 3.3, App. B.5), exactly, in the library's blocked layout (rows
 * padded to a multiple of 256; the layout is private and only
 * mixfp4_gemm_decoded reads it; padding rows are left unwritten).  The
 * tensor scale is not applied.
 *   rows, k       rows >= 0, k % 32 == 0, k <= 2^22 (else MIXFP4_ERR_SHAPE).
 *   out           device memory of out_bytes, 256-byte aligned; bytes_needed
 *                 (may be NULL) receives the size the layout needs.  out ==
 *                 NULL with out_bytes == 0 only reports that size.  A
 *                 smaller out_bytes is MIXFP4_ERR_SHAPE.
 *
 * mixfp4_gemm_decoded - C[m, n] = s32_A s32_W sum_k a[m,k] w[n,k] from two
 * decoded operands (same k), fp32 accumulation on the matrix cores (App.
 * B.1), the tensor scales applied in the epilogue (NULL = 1.0).  Accuracy as
 * for mixfp4_gemm.  m, n >= 0; k as above; k == 0 writes zeros; C fp32
 * row-major [m, n], 4-byte aligned; decoded operands 256-byte aligned.
 */
int mixfp4_decode_operand(const uint8_t *codes, const uint8_t *scales,
                          int64_t rows, int64_t k, void *out, int64_t out_bytes,
                          int64_t *bytes_needed, void *stream);
int mixfp4_gemm_decoded(const void *a_decoded, const float *a_tensor_scale,
                        const void *w_decoded, const float *w_tensor_scale,
                        int64_t m, int64_t n, int64_t k, float *c, void *stream);

/*
 * mixfp4_quantize_decode - the activation's quantization fused with the first
 * pass of the two-pass GEMM (the activation quantized on the fly before the
 * block-scaled GEMM, Sec. 3.2 / Fig. 7): one pass over X writes its MixFP4
 * codes, scales and tensor scale exactly as mixfp4_quantize does (Algorithm
 * 1) and, in the same launch, the exact 16-bit decode of those codes in the
 * layout mixfp4_decode_operand writes (Sec. 3.3, App. B.5), ready for
 * mixfp4_gemm_decoded.  With MIXFP4_SCALE_COMPUTE the tensor scale takes one
 * read of X before that pass.
 *   x, rows, k, ldx, codes, scales, tensor_scale
 *                  as for mixfp4_quantize, with k % 32 == 0 and k <= 2^22.
 *   out, out_bytes the decoded operand: device memory of at least
 *                  mixfp4_decode_operand's size for [rows, k], 256-byte
 *                  aligned (padding rows beyond the next multiple of 32 are
 *                  left unwritten).
 *   flags          MIXFP4_SCALE_COMPUTE or MIXFP4_SCALE_GIVEN, optionally
 *                  one format mode (MIXFP4_FORCE_E2M1, MIXFP4_FORCE_E1M2,
 *                  MIXFP4_FOUR_SIX).
 */
int mixfp4_quantize_decode(const uint16_t *x, int64_t rows, int64_t k, int64_t ldx,
                           uint8_t *codes, uint8_t *scales, float *tensor_scale,
                           void *out, int64_t out_bytes, unsigned flags, void *stream);

/* Human-readable name of a mixfp4_status value (static storage). */
const char *mixfp4_status_string(int status);

/*
 * mixfp4_decode_step - one decode step in one kernel launch: the tensor
 * scale and MixFP4 quantization of the activation A (Algorithm 1, the
 * compute mode of mixfp4_quantize) and C = A W^T with W already in MixFP4
 * (App. B.1; the activation quantized on the fly before the block-scaled
 * GEMM, Sec. 3.2 and Fig. 7).  A's codes, scales and tensor scale are
 * written as outputs and equal mixfp4_quantize's bit for bit; C equals
 * mixfp4_gemm on them bit for bit.
 *   a          A, bf16 bit patterns, row-major [m, k] with row pitch k,
 *              16-byte aligned (device).
 *   m, k       1 <= m <= 16, k > 0, k % 64 == 0 (else MIXFP4_ERR_SHAPE).
 *   w_codes, w_scales, w_tensor_scale, n
 *              W [n, k] as for mixfp4_gemm (w_scales 4-byte aligned;
 *              w_tensor_scale NULL means 1.0); n >= 1.
 *   a_codes    out: A's codes [m, k/2], 16-byte aligned (device).
 *   a_scales   out: A's scale bytes [m, k/16], 4-byte aligned (device).
 *   a_tensor_scale  out: A's s32, one fp32 (device).
 *   c          out: C [m, n] fp32 row-major (device).
 *   sync       four uint32 on the device, zero before the first call; the
 *              launch returns them to zero.  Calls that share `sync` must
 *              not overlap in time (one stream orders them); a caller with
 *              concurrent streams gives each its own.
 * The first workgroups of the launch quantize A once and publish it to the
 * others through `sync` (release / acquire at device scope); every wait is
 * bounded, and a workgroup that gives up writes NaN into its columns of C.
 * Null pointers: MIXFP4_ERR_NULL; misaligned: MIXFP4_ERR_ALIGN.
 */
int mixfp4_decode_step(const uint16_t *a, int64_t m, int64_t k, const uint8_t *w_codes,
                       const uint8_t *w_scales, const float *w_tensor_scale, int64_t n,
                       uint8_t *a_codes, uint8_t *a_scales, float *a_tensor_scale, float *c,
                       uint32_t *sync, void *stream);

/* HIP error string of the last MIXFP4_ERR_LAUNCH on the calling thread. */
const char *mixfp4_last_launch_error(void);

/* ABI version of this header (major * 100 + minor). */
int mixfp4_abi_version(void);

#define MIXFP4_ABI_VERSION 109

#ifdef __cplusplus
}
#endif

#endif /* MIXFP4_H */
