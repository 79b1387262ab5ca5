// MixFP4 quantization for the training GEMMs (the paper's FP4 training
// recipe, Sec. 3.2 / Fig. 7 and Sec. 4.3):
//
//  * 2D block quantization of weights: Algorithm 1 with the block being a
//    16 x 16 tile (one block maximum, one candidate-scale pair, one error
//    comparison over 256 elements, one T).  The result is written in the 1D
//    MixFP4 layout for W (blocks along K; the tile's scale byte on each of
//    its 16 rows) and, optionally, for W^T (blocks along N), so FPROP
//    (A W^T) and DGRAD (dY W) both read an ordinary K-major operand.
//  * Transposed quantization: the MixFP4 layout of X^T for a row-major X,
//    i.e. blocks of 16 consecutive rows of X, as the WGRAD operands need
//    (dW = dY^T X reduces over the token rows).  Optional Hadamard rotation
//    along the rows (b <= 64) and stochastic rounding; the result equals
//    quantizing the explicit transpose, bit for bit.
//
// Both reuse the per-block arithmetic of quant_block.h.
#include <cmath>

#include "formats.h"
#include "hadamard.h"
#include "internal.h"
#include "philox.h"
#include "quant_block.h"

namespace mixfp4 {
namespace {

constexpr int kThreads2d = 256;

// x = fl32(X / s32) with the rescale of the 1D kernels folded in: X is
// multiplied by xmul (1, or 2^+-64 when s32 is outside [2^-90, 2^120]).
struct ScaleArgs {
  float xmul, sx, rx;
};

__device__ __forceinline__ ScaleArgs scale_args(float s32) {
  ScaleArgs a;
  a.xmul = (s32 >= 0x1p-90f && s32 <= 0x1p120f) ? 1.0f : (s32 < 1.0f ? 0x1p64f : 0x1p-64f);
  a.sx = s32 * a.xmul;
  a.rx = __fdiv_rn(1.0f, a.sx);
  return a;
}

// 2D: each wave takes 4 tiles (16 lanes each, lane i = tile row i); a
// workgroup of 4 waves takes 16 consecutive tiles (row-major over the tile
// grid) per iteration.  Trip counts are uniform over the workgroup; lanes of
// a tile past the end compute on the last tile and store nothing.  With
// kT, the tile's codes are transposed through a per-wave LDS byte matrix
// (column i written by lane i, row j read by lane j).
template <int kMode, bool kT>
__global__ __launch_bounds__(kThreads2d) void quantize_2d_kernel(
    const uint16_t* __restrict__ w, int64_t n, int64_t k, int64_t ldw,
    uint8_t* __restrict__ codes, uint8_t* __restrict__ scales, uint8_t* __restrict__ codes_t,
    uint8_t* __restrict__ scales_t, const float* __restrict__ tensor_scale) {
  __shared__ ScaleRecip tab[128];
  __shared__ uint8_t tr[kThreads2d / 64][4][16][16];
  fill_scale_table(tab);
  __syncthreads();
  const ScaleArgs sa = scale_args(*tensor_scale);
  const int64_t tk = k >> 4, ntiles = (n >> 4) * tk;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int i = lane & 15, tw = lane >> 4;
  for (int64_t base = (int64_t)blockIdx.x * 16; base < ntiles; base += (int64_t)gridDim.x * 16) {
    const int64_t tt = base + wave * 4 + tw;
    const bool valid = tt < ntiles;
    const int64_t tc = valid ? tt : ntiles - 1;
    const int64_t a = tc / tk, b = tc - a * tk;
    const uint16_t* src = w + (16 * a + i) * ldw + 16 * b;
    const uint4 v0 = *reinterpret_cast<const uint4*>(src);
    const uint4 v1 = *reinterpret_cast<const uint4*>(src + 8);
    float xs[16];
    to_fp8_domain<true>(v0, v1, sa.xmul, sa.sx, sa.rx, xs);
    uint2 out;
    uint32_t sb;
    quantize_xs<kMode, false, true>(xs, tab, out, sb, make_uint4(0, 0, 0, 0));
    if (valid) {
      *reinterpret_cast<uint2*>(codes + (16 * a + i) * (k >> 1) + 8 * b) = out;
      scales[(16 * a + i) * tk + b] = (uint8_t)sb;
    }
    if constexpr (kT) {
      const uint32_t wd[2] = {out.x, out.y};
#pragma unroll
      for (int j = 0; j < 16; ++j) tr[wave][tw][j][i] = (uint8_t)((wd[j >> 3] >> (4 * (j & 7))) & 0xFu);
      __syncthreads();
      const uint4 row = *reinterpret_cast<const uint4*>(&tr[wave][tw][i][0]);   // nibbles of column i
      const uint32_t r[4] = {row.x, row.y, row.z, row.w};
      uint32_t o[2];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        // bytes b0..b7 (one nibble each) -> 8 nibbles, element 2m in the low half of byte m
        const uint32_t p = r[2 * h], q = r[2 * h + 1];
        const uint32_t lo = (p & 0xFu) | ((p >> 4) & 0xF0u) | ((p >> 8) & 0xF00u) | ((p >> 12) & 0xF000u);
        const uint32_t hi = (q & 0xFu) | ((q >> 4) & 0xF0u) | ((q >> 8) & 0xF00u) | ((q >> 12) & 0xF000u);
        o[h] = lo | (hi << 16);
      }
      if (valid) {
        const int64_t nn = n >> 4;
        *reinterpret_cast<uint2*>(codes_t + (16 * b + i) * (n >> 1) + 8 * a) = make_uint2(o[0], o[1]);
        scales_t[(16 * b + i) * nn + a] = (uint8_t)sb;
      }
      __syncthreads();
    }
  }
}

// Transposed quantization.  A workgroup stages a 64 x 64 tile of X in LDS
// transposed (column-major), then thread t owns column c = t / 4 and row
// block t % 4 of the tile: its 16 values are the X^T block (c, row block),
// read as two 16-byte vectors, exactly the input of the 1D block code.  A
// Hadamard block of b = 16 L rows spans the L lanes of a quad.  Blocks of
// X^T are numbered g = column * rows/16 + row block (the stochastic-rounding
// counter), as in the 1D layout of X^T.  kAmax: only max|rotated X| per
// workgroup (COMPUTE mode with a rotation).
constexpr int kTileR = 64, kTileC = 64, kPitch = kTileR + 8;   // LDS row pitch (elements)

template <int kMode, bool kSR, bool kHad, bool kAmax>
__global__ __launch_bounds__(kThreads2d) void quantize_t_kernel(
    const uint16_t* __restrict__ x, int64_t rows, int64_t k, int64_t ldx,
    uint8_t* __restrict__ codes_t, uint8_t* __restrict__ scales_t,
    const float* __restrict__ tensor_scale, SrParams sr, HadamardParams hp,
    uint32_t* __restrict__ partials) {
  __shared__ ScaleRecip tab[128];
  __shared__ uint16_t xt[kTileC][kPitch];
  __shared__ uint32_t wave_max[kThreads2d / 64];
  if constexpr (!kAmax) fill_scale_table(tab);
  ScaleArgs sa{1.0f, 1.0f, 1.0f};
  if constexpr (!kAmax) sa = scale_args(*tensor_scale);
  SignMasks sm;
  if constexpr (kHad) sm = load_sign_masks(hp, (int)(threadIdx.x & ((1u << hp.lanes_log2) - 1u)));
  const int64_t trs = (rows + kTileR - 1) / kTileR, tcs = (k + kTileC - 1) / kTileC;
  const int64_t ntiles = trs * tcs, rb_total = rows >> 4;
  const int c = threadIdx.x >> 2, rbl = threadIdx.x & 3;
  uint32_t m = 0u;
  for (int64_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
    const int64_t tr0 = tile / tcs, tc0 = tile - tr0 * tcs;
    const int64_t r0 = tr0 * kTileR, c0 = tc0 * kTileC;
    __syncthreads();                         // previous tile's reads are done (and the table is built)
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int q = threadIdx.x + kThreads2d * h;
      const int row = q >> 3, ch = q & 7;
      uint4 v = make_uint4(0, 0, 0, 0);
      if (r0 + row < rows && c0 + 8 * ch < k)
        v = *reinterpret_cast<const uint4*>(x + (r0 + row) * ldx + c0 + 8 * ch);
      const uint32_t e[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        xt[8 * ch + 2 * j][row] = (uint16_t)e[j];
        xt[8 * ch + 2 * j + 1][row] = (uint16_t)(e[j] >> 16);
      }
    }
    __syncthreads();
    uint4 v0 = *reinterpret_cast<const uint4*>(&xt[c][16 * rbl]);
    uint4 v1 = *reinterpret_cast<const uint4*>(&xt[c][16 * rbl + 8]);
    const bool valid = c0 + c < k && (r0 >> 4) + rbl < rb_total;
    if constexpr (kHad) hadamard_rotate(v0, v1, sm, hp);
    if constexpr (kAmax) {
      if (valid) m = max(m, max(absmax8(v0), absmax8(v1)));
    } else {
      float xs[16];
      to_fp8_domain<true>(v0, v1, sa.xmul, sa.sx, sa.rx, xs);
      const int64_t col = c0 + c, rb = (r0 >> 4) + rbl;
      const int64_t g = col * rb_total + rb;
      uint2 out;
      uint32_t sb;
      quantize_xs<kMode, kSR>(xs, tab, out, sb, kSR ? block_draws(g, sr) : make_uint4(0, 0, 0, 0));
      if (valid) {
        *reinterpret_cast<uint2*>(codes_t + (g << 3)) = out;
        scales_t[g] = (uint8_t)sb;
      }
    }
  }
  if constexpr (kAmax) {
    for (int off = 32; off > 0; off >>= 1) m = max(m, (uint32_t)__shfl_xor((int)m, off));
    if ((threadIdx.x & 63) == 0) wave_max[threadIdx.x >> 6] = m;
    __syncthreads();
    if (threadIdx.x == 0) {
      uint32_t r = wave_max[0];
      for (int wv = 1; wv < kThreads2d / 64; ++wv) r = max(r, wave_max[wv]);
      partials[blockIdx.x] = r;
    }
  }
}

// One workgroup: fold per-workgroup maxima (bf16 magnitude bits) into s32.
__global__ __launch_bounds__(kThreads2d) void reduce_scale_t(const uint32_t* __restrict__ partials,
                                                             int count, float* __restrict__ out) {
  uint32_t m = 0u;
  for (int i = threadIdx.x; i < count; i += kThreads2d) m = max(m, partials[i]);
  for (int off = 32; off > 0; off >>= 1) m = max(m, (uint32_t)__shfl_xor((int)m, off));
  __shared__ uint32_t wave_max[kThreads2d / 64];
  if ((threadIdx.x & 63) == 0) wave_max[threadIdx.x >> 6] = m;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t r = wave_max[0];
    for (int wv = 1; wv < kThreads2d / 64; ++wv) r = max(r, wave_max[wv]);
    *out = tensor_scale_of(r);
  }
}

int grid_2d(int64_t work_items, int64_t per_group) {
  int64_t g = (work_items + per_group - 1) / per_group;
  if (g < 1) g = 1;
  if (g > 4096) g = 4096;
  return (int)g;
}

template <int kMode>
hipError_t launch_2d_mode(const uint16_t* w, int64_t n, int64_t k, int64_t ldw, uint8_t* codes,
                          uint8_t* scales, uint8_t* codes_t, uint8_t* scales_t,
                          const float* tensor_scale, hipStream_t stream) {
  const int g = grid_2d((n >> 4) * (k >> 4), 16);
  if (codes_t)
    quantize_2d_kernel<kMode, true><<<g, kThreads2d, 0, stream>>>(w, n, k, ldw, codes, scales,
                                                                  codes_t, scales_t, tensor_scale);
  else
    quantize_2d_kernel<kMode, false><<<g, kThreads2d, 0, stream>>>(w, n, k, ldw, codes, scales,
                                                                   nullptr, nullptr, tensor_scale);
  return hipGetLastError();
}

template <int kMode, bool kSR, bool kHad>
hipError_t launch_t_mode(const uint16_t* x, int64_t rows, int64_t k, int64_t ldx,
                         uint8_t* codes_t, uint8_t* scales_t, const float* tensor_scale,
                         const QuantOptions& opt, hipStream_t stream) {
  const int64_t tiles = ((rows + kTileR - 1) / kTileR) * ((k + kTileC - 1) / kTileC);
  const int g = grid_2d(tiles, 1);
  quantize_t_kernel<kMode, kSR, kHad, false><<<g, kThreads2d, 0, stream>>>(
      x, rows, k, ldx, codes_t, scales_t, tensor_scale, opt.srp, opt.hp, nullptr);
  return hipGetLastError();
}

template <int kMode>
hipError_t launch_t_opts(const uint16_t* x, int64_t rows, int64_t k, int64_t ldx,
                         uint8_t* codes_t, uint8_t* scales_t, const float* tensor_scale,
                         const QuantOptions& opt, hipStream_t stream) {
  if (opt.sr)
    return opt.had ? launch_t_mode<kMode, true, true>(x, rows, k, ldx, codes_t, scales_t,
                                                      tensor_scale, opt, stream)
                   : launch_t_mode<kMode, true, false>(x, rows, k, ldx, codes_t, scales_t,
                                                       tensor_scale, opt, stream);
  return opt.had ? launch_t_mode<kMode, false, true>(x, rows, k, ldx, codes_t, scales_t,
                                                     tensor_scale, opt, stream)
                 : launch_t_mode<kMode, false, false>(x, rows, k, ldx, codes_t, scales_t,
                                                      tensor_scale, opt, stream);
}

}  // namespace

hipError_t launch_quantize_2d(const uint16_t* w, int64_t n, int64_t k, int64_t ldw,
                              uint8_t* codes, uint8_t* scales, uint8_t* codes_t,
                              uint8_t* scales_t, const float* tensor_scale, int mode,
                              hipStream_t stream) {
  if (n == 0 || k == 0) return hipSuccess;
  if (mode == 3)
    return launch_2d_mode<3>(w, n, k, ldw, codes, scales, codes_t, scales_t, tensor_scale, stream);
  if (mode == 1)
    return launch_2d_mode<1>(w, n, k, ldw, codes, scales, codes_t, scales_t, tensor_scale, stream);
  if (mode == 2)
    return launch_2d_mode<2>(w, n, k, ldw, codes, scales, codes_t, scales_t, tensor_scale, stream);
  return launch_2d_mode<0>(w, n, k, ldw, codes, scales, codes_t, scales_t, tensor_scale, stream);
}

hipError_t launch_quantize_t(const uint16_t* x, int64_t rows, int64_t k, int64_t ldx,
                             uint8_t* codes_t, uint8_t* scales_t, const float* tensor_scale,
                             const QuantOptions& opt, hipStream_t stream) {
  if (rows == 0 || k == 0) return hipSuccess;
  if (opt.mode == 3)
    return launch_t_opts<3>(x, rows, k, ldx, codes_t, scales_t, tensor_scale, opt, stream);
  if (opt.mode == 1)
    return launch_t_opts<1>(x, rows, k, ldx, codes_t, scales_t, tensor_scale, opt, stream);
  if (opt.mode == 2)
    return launch_t_opts<2>(x, rows, k, ldx, codes_t, scales_t, tensor_scale, opt, stream);
  return launch_t_opts<0>(x, rows, k, ldx, codes_t, scales_t, tensor_scale, opt, stream);
}

hipError_t launch_tensor_scale_t_rotated(const uint16_t* x, int64_t rows, int64_t k, int64_t ldx,
                                         const HadamardParams& hp, uint8_t* scratch,
                                         int64_t scratch_bytes, float* tensor_scale,
                                         hipStream_t stream) {
  // per-workgroup maxima in the caller's scale-byte output (>= 1 slot per
  // workgroup: rows * k / 16 bytes hold at least one 4-byte slot per 64 x 64 tile)
  const int64_t tiles = ((rows + kTileR - 1) / kTileR) * ((k + kTileC - 1) / kTileC);
  const uintptr_t base = reinterpret_cast<uintptr_t>(scratch);
  const uintptr_t aligned = (base + 3u) & ~uintptr_t(3);
  const int64_t slots = (scratch_bytes - (int64_t)(aligned - base)) / 4;
  int g = grid_2d(tiles, 1);
  if (g > slots) g = (int)slots;
  if (g < 1) return hipErrorInvalidValue;
  uint32_t* partials = reinterpret_cast<uint32_t*>(aligned);
  quantize_t_kernel<0, false, true, true><<<g, kThreads2d, 0, stream>>>(
      x, rows, k, ldx, nullptr, nullptr, nullptr, SrParams{}, hp, partials);
  reduce_scale_t<<<1, kThreads2d, 0, stream>>>(partials, g, tensor_scale);
  return hipGetLastError();
}

}  // namespace mixfp4
