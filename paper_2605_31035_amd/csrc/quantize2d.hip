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

// 2D, W's layout only: each wave takes 4 tiles (16 lanes each, lane i =
// tile row i); a workgroup of 4 waves takes 16 consecutive tiles (row-major
// over the tile grid) per iteration.  Trip counts are uniform over the
// workgroup; lanes of a tile past the end compute on the last tile and store
// nothing.
template <int kMode>
__global__ __launch_bounds__(kThreads2d) void quantize_2d_kernel(
    const uint16_t* __restrict__ w, int64_t n, int64_t k, int64_t ldw,
    uint8_t* __restrict__ codes, uint8_t* __restrict__ scales,
    const float* __restrict__ tensor_scale) {
  __shared__ ScaleRecip tab[128];
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
  }
}

// 2D, both layouts.  A workgroup takes super-blocks of kSR tile rows x kSC
// tile columns of W.  Each iteration quantizes 16 tiles (16 / kSC tile rows
// of kSC tiles; wave w takes tiles 4w..4w+3, lane i of a tile its row i) and
// stores them in W's layout directly.  The tile's codes are then transposed
// in registers across its 16 lanes (one DPP row), so lane i holds row i of
// the W^T tile.  A W^T row of the super-block collects one 8-byte code chunk
// and one scale byte from each of its kSR tile rows, so those rows are
// staged in LDS (the chunk slot XOR-swizzled by the row, so that the 16
// lanes of a tile, one row each, write kSR different slots rather than the
// same one) and written out after the last
// iteration as runs of 8 kSR code bytes and kSR scale bytes.  Stored one
// chunk per lane, the W^T rows cost a separate memory transaction for every
// 8 bytes of codes and every scale byte.
template <int kMode, int kSR, int kSC>
__global__ __launch_bounds__(kThreads2d) void quantize_2d_both_kernel(
    const uint16_t* __restrict__ w, int64_t n, int64_t k, int64_t ldw,
    uint8_t* __restrict__ codes, uint8_t* __restrict__ scales, uint8_t* __restrict__ codes_t,
    uint8_t* __restrict__ scales_t, const float* __restrict__ tensor_scale) {
  constexpr int kRowsT = 16 * kSC;               // W^T rows of a super-block
  constexpr int kTileRowsIt = 16 / kSC;          // tile rows per iteration
  constexpr int kPairs = kSR / 2;                // 16-byte code pairs per staged row
  static_assert((kSR == 8 || kSR == 16) && kTileRowsIt * kSC == 16 && kRowsT <= kThreads2d,
                "super-block shape");
  __shared__ ScaleRecip tab[128];
  __shared__ uint4 st_codes[kRowsT * kPairs];    // row r: kSR chunks of 8 bytes
  __shared__ uint2 st_scales[kRowsT * kSR / 8];  // row r: kSR scale bytes
  fill_scale_table(tab);
  __syncthreads();
  const ScaleArgs sa = scale_args(*tensor_scale);
  const int64_t ta = n >> 4, tb = k >> 4;        // tile rows and columns of W
  const int64_t nsa = (ta + kSR - 1) / kSR, nsb = (tb + kSC - 1) / kSC;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int i = lane & 15, q = wave * 4 + (lane >> 4);   // tile slot of an iteration
  const int dr = q / kSC, db = q % kSC;
  const int rt = db * 16 + i;                     // this lane's W^T row in the super-block
  const Transpose16 tsel = transpose16_setup(i);
  const int64_t pitch_t = n >> 1;                 // W^T code row, bytes
  const bool codes_al16 = (n & 31) == 0;
  const bool scales_al = (ta % kSR) == 0 && (reinterpret_cast<uintptr_t>(scales_t) % kSR) == 0;
  uint2* const st_chunk = reinterpret_cast<uint2*>(st_codes);
  uint8_t* const st_byte = reinterpret_cast<uint8_t*>(st_scales);
  for (int64_t sbi = blockIdx.x; sbi < nsa * nsb; sbi += gridDim.x) {
    const int64_t a0 = (sbi / nsb) * kSR, b0 = (sbi % nsb) * kSC;
    const int ra = (int)(ta - a0 < kSR ? ta - a0 : kSR);
    const int rb = (int)(tb - b0 < kSC ? tb - b0 : kSC);
    const bool b_ok = db < rb;
    const int64_t b = b_ok ? b0 + db : tb - 1;
    const int iters = (ra + kTileRowsIt - 1) / kTileRowsIt;
    for (int it = 0; it < iters; ++it) {
      const int sl = it * kTileRowsIt + dr;      // tile row a0 + sl
      const bool a_ok = sl < ra;
      const int64_t a = a0 + (a_ok ? sl : ra - 1);
      const uint16_t* src = w + (16 * a + i) * ldw + 16 * b;
      const uint4 v0 = *reinterpret_cast<const uint4*>(src);
      const uint4 v1 = *reinterpret_cast<const uint4*>(src + 8);
      float xs[16];
      to_fp8_domain<true>(v0, v1, sa.xmul, sa.sx, sa.rx, xs);
      uint2 out;
      uint32_t sb;
      quantize_xs<kMode, false, true>(xs, tab, out, sb, make_uint4(0, 0, 0, 0));
      if (a_ok && b_ok) {
        *reinterpret_cast<uint2*>(codes + (16 * a + i) * (k >> 1) + 8 * b) = out;
        scales[(16 * a + i) * tb + b] = (uint8_t)sb;
      }
      uint32_t o0 = out.x, o1 = out.y;
      transpose16_nibbles(tsel, o0, o1);
      if (a_ok) {
        st_chunk[rt * kSR + (sl ^ (rt & (kSR - 1)))] = make_uint2(o0, o1);
        st_byte[rt * kSR + sl] = (uint8_t)sb;
      }
    }
    __syncthreads();
    // W^T row 16 b0 + r: chunks 2c, 2c+1 sit in the pair c ^ (x >> 1), x =
    // r mod kSR, swapped when x is odd
    for (int idx = threadIdx.x; idx < kRowsT * kPairs; idx += kThreads2d) {
      const int r = idx / kPairs, c = idx % kPairs;
      if (r >= 16 * rb || 2 * c >= ra) continue;
      const int x = r & (kSR - 1);
      const uint4 v = st_codes[r * kPairs + (c ^ (x >> 1))];
      const bool odd = (x & 1) != 0;
      const uint2 lo = odd ? make_uint2(v.z, v.w) : make_uint2(v.x, v.y);
      const uint2 hi = odd ? make_uint2(v.x, v.y) : make_uint2(v.z, v.w);
      uint8_t* dst = codes_t + (16 * b0 + r) * pitch_t + 8 * a0 + 16 * c;
      if (2 * c + 1 < ra && codes_al16) {
        *reinterpret_cast<uint4*>(dst) = make_uint4(lo.x, lo.y, hi.x, hi.y);
      } else {
        *reinterpret_cast<uint2*>(dst) = lo;
        if (2 * c + 1 < ra) *reinterpret_cast<uint2*>(dst + 8) = hi;
      }
    }
    if (threadIdx.x < 16 * rb) {
      const int r = threadIdx.x;
      uint8_t* dst = scales_t + (16 * b0 + r) * ta + a0;
      if (ra == kSR && scales_al) {
        if constexpr (kSR == 16) {
          *reinterpret_cast<uint4*>(dst) =
              make_uint4(st_scales[2 * r].x, st_scales[2 * r].y, st_scales[2 * r + 1].x,
                         st_scales[2 * r + 1].y);
        } else {
          *reinterpret_cast<uint2*>(dst) = st_scales[r];
        }
      } else {
        for (int j = 0; j < ra; ++j) dst[j] = st_byte[r * kSR + j];
      }
    }
    __syncthreads();   // the next super-block overwrites the staging rows
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
  if (codes_t) {
    // super-blocks of 8 x 8 tiles: 64-byte runs of codes in both layouts.
    // Measured on 11008 x 4096: 33-35 us, against 37-41 us for 16 x 16, 16 x 8
    // or 8 x 16 tiles (fewer, longer workgroups balance worse over the CUs).
    constexpr int kSR = 8, kSC = 8;
    const int64_t supers = (((n >> 4) + kSR - 1) / kSR) * (((k >> 4) + kSC - 1) / kSC);
    quantize_2d_both_kernel<kMode, kSR, kSC><<<grid_2d(supers, 1), kThreads2d, 0, stream>>>(
        w, n, k, ldw, codes, scales, codes_t, scales_t, tensor_scale);
  } else {
    quantize_2d_kernel<kMode><<<grid_2d((n >> 4) * (k >> 4), 16), kThreads2d, 0, stream>>>(
        w, n, k, ldw, codes, scales, tensor_scale);
  }
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
