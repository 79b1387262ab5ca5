// MixFP4 tensor scale and block quantizer (Algorithm 1) for gfx950: the 1D
// kernels (one lane per 16-element block along K), the rotation kernels and
// the launchers.  The per-block arithmetic lives in quant_block.h.
//
// Tensor scale (Algorithm 1, first step): s32 = max|X| / 2688, where
// 2688 = 6 * 448 = 7 * 384 makes the block holding the tensor maximum land on
// the largest E4M3 scales.  Per-workgroup maxima of |X| (integer max on the
// bf16 magnitude bits) are folded by one small workgroup, or, without a
// scratch buffer, by one atomic max of the fp32 bit pattern (order free, so
// deterministic).
//
// Quantizer: one lane owns one 16-element block (App. B.1, V = 16): two
// 16-byte loads, no cross-lane traffic, one 8-byte code store and one scale
// byte.  Codes, scales and the format bit are exactly those of Algorithm 1:
//   * x = fl32(X / s32), the candidate-scale quotients and the grid
//     quotients y = fl32(|x| / s8) are correctly rounded fp32 divisions:
//     X / s32 with Markstein's division step from a correctly rounded
//     reciprocal (div_rn), the quotients by 6, 7 and the E4M3 block scales
//     (at most 4 significant bits) with one fma on a two-term reciprocal
//     (div_scale); both proved exhaustively for the operand classes used.
//     Rounding y to a grid equals rounding the exact quotient, because a
//     grid midpoint times s8 is exact in fp32.
//   * E2M1 rounding uses the gfx950 FP4 converter with scale 1 (round to
//     nearest even onto the E2M1 grid, ties to the even code, saturating,
//     sign kept); INT4 rounding is rint (round half to even).
//   * The format choice: an fp32 estimate s_F^2 sum q_F^2 - s_I^2 sum q_I^2
//     + 2 (s_I sum |x| q_I - s_F sum x q_F) decides when it is farther from
//     zero than its proven error bound; otherwise the exact fp64 sum
//     sum_i (D_I - D_F)(2|x| - D_F - D_I) decides (every term exact, only
//     elements whose two dequantized values differ contribute, so the sum
//     is exact in any order).
#include <cmath>

#include "formats.h"
#include "hadamard.h"
#include "internal.h"
#include "philox.h"
#include "quant_block.h"

typedef int mixfp4_i32x4q __attribute__((ext_vector_type(4)));

namespace mixfp4 {
namespace {

constexpr int kThreads = 256;

__global__ void clear_u32(uint32_t* p) { *p = 0u; }

// Per-workgroup max of |X| over a [rows, k] bf16 matrix (row pitch ldx) as
// bf16 magnitude bits.  Each thread keeps four 16-byte loads in flight.
// With `partials` the result of workgroup b goes to partials[b]; otherwise it
// is folded into *out with an atomic max of the fp32 bit pattern.
__global__ __launch_bounds__(kThreads) void amax_kernel(const uint16_t* __restrict__ x,
                                                         int64_t rows, int64_t k, int64_t ldx,
                                                         uint32_t* __restrict__ partials,
                                                         uint32_t* __restrict__ out) {
  const int64_t vec_per_row = k >> 3;               // 8 bf16 per 16-byte vector
  const int64_t total = rows * vec_per_row;
  auto vec_ptr = [&](int64_t i) -> const uint4* {
    if (ldx == k) return reinterpret_cast<const uint4*>(x) + i;
    const int64_t r = i / vec_per_row;
    return reinterpret_cast<const uint4*>(x + r * ldx) + (i - r * vec_per_row);
  };
  uint32_t m = 0u;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  for (; i + 3 * stride < total; i += 4 * stride) {
    const uint4 a = *vec_ptr(i), b = *vec_ptr(i + stride);
    const uint4 c = *vec_ptr(i + 2 * stride), d = *vec_ptr(i + 3 * stride);
    m = max(m, max(max(absmax8(a), absmax8(b)), max(absmax8(c), absmax8(d))));
  }
  for (; i < total; i += stride) m = max(m, absmax8(*vec_ptr(i)));
  for (int off = 32; off > 0; off >>= 1) m = max(m, (uint32_t)__shfl_xor((int)m, off));
  __shared__ uint32_t wave_max[kThreads / 64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) wave_max[wave] = m;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t r = wave_max[0];
    for (int w = 1; w < kThreads / 64; ++w) r = max(r, wave_max[w]);
    if (partials) partials[blockIdx.x] = r;
    else if (r) atomicMax(out, r << 16);            // bf16 bits -> fp32 bits
  }
}

// The same maximum over a contiguous X: each wave reads windows of 4 KB
// (256 16-byte vectors), four loads per lane that each cover 1 KB of
// contiguous memory, with the non-temporal hint (X is read once here), the
// next window's loads in flight while this one is reduced.  Windows past the
// end read zeros (buffer range check), which leave the maximum unchanged.
constexpr int kAmaxWindow = 256;      // vectors of 8 bf16 per wave per iteration

__global__ __launch_bounds__(kThreads) void amax_stream_kernel(const uint16_t* __restrict__ x,
                                                                int64_t nvec,
                                                                uint32_t* __restrict__ partials,
                                                                uint32_t* __restrict__ out) {
  typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
  const int lane = (int)(threadIdx.x & 63);
  const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const int64_t windows = (nvec + kAmaxWindow - 1) / kAmaxWindow;
  const int64_t waves = (int64_t)gridDim.x * (kThreads / 64);
  const int64_t iters = (windows + waves - 1) / waves;
  auto load = [&](int64_t i, u32x4 (&v)[4]) {
    const int64_t base = ((i * gridDim.x + blockIdx.x) * (kThreads / 64) + wave) * kAmaxWindow;
    int64_t rem = nvec - base;
    rem = rem < 0 ? 0 : (rem < kAmaxWindow ? rem : kAmaxWindow);
    const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(x + base * 8), 0, (int)(rem * 16), 0x00020000);
#pragma unroll
    for (int j = 0; j < 4; ++j)
      v[j] = __builtin_amdgcn_raw_buffer_load_b128(r, lane * 16 + j * 1024, 0, 2);
  };
  u32x4 cur[4], nxt[4];
  load(0, cur);
  uint32_t m = 0u;
  for (int64_t i = 0; i < iters; ++i) {
    load(i + 1, nxt);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      m = max(m, absmax8(make_uint4(cur[j].x, cur[j].y, cur[j].z, cur[j].w)));
      cur[j] = nxt[j];
    }
  }
  for (int off = 32; off > 0; off >>= 1) m = max(m, (uint32_t)__shfl_xor((int)m, off));
  __shared__ uint32_t wave_max[kThreads / 64];
  if (lane == 0) wave_max[wave] = m;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t r = wave_max[0];
    for (int w = 1; w < kThreads / 64; ++w) r = max(r, wave_max[w]);
    if (partials) partials[blockIdx.x] = r;
    else if (r) atomicMax(out, r << 16);            // bf16 bits -> fp32 bits
  }
}

// One workgroup: fold the per-workgroup maxima and write s32.
__global__ __launch_bounds__(kThreads) void reduce_scale(const uint32_t* __restrict__ partials,
                                                          int count, float* __restrict__ out) {
  uint32_t m = 0u;
  for (int i = threadIdx.x; i < count; i += kThreads) m = max(m, partials[i]);
  for (int off = 32; off > 0; off >>= 1) m = max(m, (uint32_t)__shfl_xor((int)m, off));
  __shared__ uint32_t wave_max[kThreads / 64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) wave_max[wave] = m;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t r = wave_max[0];
    for (int w = 1; w < kThreads / 64; ++w) r = max(r, wave_max[w]);
    *out = tensor_scale_of(r);
  }
}

// In place: fp32 bits of max|X| -> s32 = fl32(amax / 2688), or 1.0 if zero.
__global__ void finalize_scale(uint32_t* p) {
  *reinterpret_cast<float*>(p) = tensor_scale_of(*p >> 16);
}

// The FP8 domain x = fl32(X / s32): kTwoTerm from the two-term reciprocal
// {rh, rl} of s32 (tensor scales that passed the check below), otherwise
// X * xmul (exact) divided by sx = s32 * xmul with Markstein's step on
// rx = fl32(1 / sx).
struct XDomain {
  float xmul, sx, rx, rh, rl;
};

// How x = fl32(X / s32) is computed: the two-term reciprocal of s32
// (kTwoTerm), Markstein's step on X (kMarkstein), or Markstein's step on
// X * xmul for tensor scales outside [2^-90, 2^120] (kScaledX).
constexpr int kTwoTerm = 0, kMarkstein = 1, kScaledX = 2;

template <int kDiv>
__device__ __forceinline__ void to_x(uint4 r0, uint4 r1, const XDomain& xd, float (&xs)[16]) {
  if constexpr (kDiv == kTwoTerm)
    to_fp8_domain_two_term(r0, r1, xd.rh, xd.rl, xs);
  else
    to_fp8_domain<kDiv == kScaledX>(r0, r1, xd.xmul, xd.sx, xd.rx, xs);
}

// Grid-stride walk over the blocks of X in registers (row-strided X, and
// the rotating quantizer, whose fp64 butterflies need the registers more
// than the stream loop's bytes in flight help it: measured 400 against 446
// us for 128-blocks on the 2^28 tensor).  The next block of this thread is
// loaded as soon as the current one has been turned into x, so its load
// overlaps this block's arithmetic.
//
// kSR: stochastic rounding with Philox draws per block (its global index).
// kHad: each block is first rotated (block-diagonal Hadamard across the
// L = b / 16 lanes holding one Hadamard block; the grid stride is a multiple
// of 256, so a thread keeps its position in its Hadamard block and every
// Hadamard block is processed by lanes of one wave in one iteration).
template <int kDiv, bool kContig, int kMode, bool kSR, bool kHad>
__device__ __forceinline__ void quantize_loop(const uint16_t* __restrict__ x, int64_t nbk,
                                              int64_t ldx, int64_t nblocks,
                                              uint8_t* __restrict__ codes,
                                              uint8_t* __restrict__ scales, const XDomain& xd,
                                              const ScaleRecip* tab, const SrParams& sr,
                                              const HadamardParams& hp) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  // Loads are unconditional (a block index past the end reads the last
  // block, whose data is then never used), so they need no branch and no
  // register copies.
  auto load = [&](int64_t gi, uint4& p, uint4& q) {
    gi = gi < nblocks ? gi : nblocks - 1;
    const uint16_t* src;
    if constexpr (kContig) {
      src = x + (gi << 4);
    } else {
      const int64_t r = gi / nbk;
      src = x + r * ldx + ((gi - r * nbk) << 4);
    }
    p = *reinterpret_cast<const uint4*>(src);
    q = *reinterpret_cast<const uint4*>(src + 8);
  };
  int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  SignMasks sm;
  if constexpr (kHad) sm = load_sign_masks(hp, (int)(threadIdx.x & ((1u << hp.lanes_log2) - 1u)));
  uint4 a0, a1;
  load(g, a0, a1);
  for (; g < nblocks; g += stride) {
    float xs[16];
    uint4 r0 = a0, r1 = a1;
    if constexpr (kHad) hadamard_rotate(r0, r1, sm, hp);
    to_x<kDiv>(r0, r1, xd, xs);
    load(g + stride, a0, a1);
    uint2 out;
    uint32_t sb;
    quantize_xs<kMode, kSR>(xs, tab, out, sb, kSR ? block_draws(g, sr) : make_uint4(0, 0, 0, 0));
    *reinterpret_cast<uint2*>(codes + (g << 3)) = out;
    scales[g] = (uint8_t)sb;
  }
}

// Contiguous X: each wave streams windows of 64 blocks (2 KB of X) through a
// ring of two 2 KB LDS slots with 16-byte buffer loads that write straight
// into LDS, one window ahead; lane l then reads block l of the window (32 B)
// from LDS.  Every load instruction covers 1 KB of contiguous memory and
// carries the non-temporal hint (X is read once), and the bytes in flight
// hold no registers.  Measured on MI355X with this traffic (2 B read, 0.5625
// B written per element) and no arithmetic: 6.36 TB/s, against 5.45 TB/s for
// two 16-byte loads per lane straight into registers, which is what the
// quantizer did before.  Windows are dealt round-robin over the waves of the
// grid; every wave runs the same number of iterations, and windows past the
// end read zeros and store nothing (buffer range checks), so the loop has no
// divergent exit.  Codes and scales leave through buffer stores on the same
// window bases.
constexpr int kWindow = 64;          // blocks per wave per iteration
constexpr int kWindowBytes = kWindow * 32;
constexpr int kRingAux = 2;          // non-temporal loads

typedef mixfp4_i32x4q i32x4q;
__device__ __forceinline__ i32x4q raw_rsrc(const void* base, uint32_t bytes) {
  const uint64_t b = reinterpret_cast<uint64_t>(base);
  i32x4q r;
  r[0] = (int)(uint32_t)b;
  r[1] = (int)(uint32_t)(b >> 32);
  r[2] = (int)bytes;
  r[3] = 0x00020000;
  return r;
}
__device__ __forceinline__ __amdgpu_buffer_rsrc_t store_rsrc(void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(base, 0, (int)bytes, 0x00020000);
}

}  // namespace
}  // namespace mixfp4

// The 16-byte buffer load that writes straight into LDS (destination M0 +
// offset + 16 * lane).
__device__ void mixfp4_q_buffer_load_lds(mixfp4_i32x4q rsrc,
                                         __attribute__((address_space(3))) uint32_t* lds,
                                         int size, int voffset, int soffset, int offset,
                                         int aux) __asm("llvm.amdgcn.raw.buffer.load.lds");

namespace mixfp4 {
namespace {

template <int kDiv, int kMode, bool kSR, bool kHad>
__device__ __forceinline__ void stream_loop(const uint16_t* __restrict__ x, int64_t nblocks,
                                            uint8_t* __restrict__ codes,
                                            uint8_t* __restrict__ scales, const XDomain& xd,
                                            const ScaleRecip* tab, const SrParams& sr,
                                            const HadamardParams& hp, uint8_t* ring) {
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const int64_t windows = (nblocks + kWindow - 1) / kWindow;
  const int64_t waves = (int64_t)gridDim.x * (kThreads / 64);
  const int64_t iters = (windows + waves - 1) / waves;
  uint8_t* slots = ring + wave * 2 * kWindowBytes;
  auto first_block = [&](int64_t i) {
    return ((i * gridDim.x + blockIdx.x) * (kThreads / 64) + wave) * kWindow;
  };
  auto blocks_in = [&](int64_t base) {
    const int64_t rem = nblocks - base;
    return rem < 0 ? 0 : (rem < kWindow ? rem : kWindow);
  };
  auto issue = [&](int64_t i) {
    const int64_t base = first_block(i);
    const i32x4q r = raw_rsrc(x + base * 16, (uint32_t)(blocks_in(base) * 32));
    __attribute__((address_space(3))) uint32_t* l =
        (__attribute__((address_space(3))) uint32_t*)(uintptr_t)(
            reinterpret_cast<uintptr_t>(slots + (i & 1) * kWindowBytes));
    mixfp4_q_buffer_load_lds(r, l, 16, lane * 16, 0, 0, kRingAux);
    mixfp4_q_buffer_load_lds(r, l, 16, lane * 16, 0, 1024, kRingAux);
  };
  SignMasks sm;
  if constexpr (kHad) sm = load_sign_masks(hp, lane & ((1 << hp.lanes_log2) - 1));
  issue(0);
  for (int64_t i = 0; i < iters; ++i) {
    // Vector memory operations complete in issue order, and vmcnt counts
    // stores as well as loads: after window i's two loads this wave issued
    // only the previous window's two stores, which may stay in flight.
    if (i == 0)
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    else
      asm volatile("s_waitcnt vmcnt(2)" ::: "memory");
    const uint4* src = reinterpret_cast<const uint4*>(slots + (i & 1) * kWindowBytes + lane * 32);
    uint4 r0 = src[0], r1 = src[1];
    // The other slot held window i - 1, whose reads finished last iteration.
    issue(i + 1);
    const int64_t base = first_block(i);
    if constexpr (kHad) hadamard_rotate(r0, r1, sm, hp);
    float xs[16];
    to_x<kDiv>(r0, r1, xd, xs);
    uint2 out;
    uint32_t sb;
    quantize_xs<kMode, kSR>(xs, tab, out, sb,
                            kSR ? block_draws(base + lane, sr) : make_uint4(0, 0, 0, 0));
    const int64_t n = blocks_in(base);
    typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
    __builtin_amdgcn_raw_buffer_store_b64(u32x2{out.x, out.y},
                                          store_rsrc(codes + base * 8, (uint32_t)(n * 8)), lane * 8,
                                          0, 0);
    __builtin_amdgcn_raw_buffer_store_b8((uint8_t)sb, store_rsrc(scales + base, (uint32_t)n),
                                         lane, 0, 0);
  }
}

// Quantize the blocks of X with tensor scale s32.  The division steps stay
// in the normal range for every element that can get a nonzero code when
// 2^-90 <= s32 <= 2^120; beyond that both X and s32 are rescaled by 2^64 or
// 2^-64 first.  Within that range, the two-term division is used when it
// reproduces the exact quotient on all 128 bf16 mantissas (checked by the
// first 128 threads of every workgroup, so every workgroup takes the same,
// deterministic decision); the kernel's barrier publishes the check and the
// scale table together.
template <bool kContig, int kMode, bool kSR, bool kHad>
__global__ __launch_bounds__(kThreads) void quantize_kernel(
    const uint16_t* __restrict__ x, int64_t nbk, int64_t ldx, int64_t nblocks,
    uint8_t* __restrict__ codes, uint8_t* __restrict__ scales,
    const float* __restrict__ tensor_scale, SrParams sr, HadamardParams hp) {
  __shared__ ScaleRecip tab[128];
  fill_scale_table(tab);
  const float s32 = *tensor_scale;
  const bool direct = s32 >= 0x1p-90f && s32 <= 0x1p120f;
  XDomain xd;
  xd.xmul = direct ? 1.0f : (s32 < 1.0f ? 0x1p64f : 0x1p-64f);
  xd.sx = s32 * xd.xmul;
  xd.rx = __fdiv_rn(1.0f, xd.sx);
  const ScaleRecip r32 = scale_recip(s32);
  xd.rh = r32.rh;
  xd.rl = r32.rl;
  int ok = 1;
  if (direct && threadIdx.x < 128) {
    // mantissa t at the exponent of s32, so that the quotient is near 1
    const float xt = __uint_as_float((__float_as_uint(s32) & 0x7F800000u) | (threadIdx.x << 16));
    ok = __float_as_uint(div_rn(xt, xd.sx, xd.rx)) == __float_as_uint(div_scale(xt, xd.rh, xd.rl));
  }
  const bool two_term = __syncthreads_and(ok) && direct;
  if constexpr (kContig && !kHad) {
    __shared__ __attribute__((aligned(1024))) uint8_t ring[(kThreads / 64) * 2 * kWindowBytes];
    if (two_term)
      stream_loop<kTwoTerm, kMode, kSR, kHad>(x, nblocks, codes, scales, xd, tab, sr, hp, ring);
    else if (direct)
      stream_loop<kMarkstein, kMode, kSR, kHad>(x, nblocks, codes, scales, xd, tab, sr, hp, ring);
    else
      stream_loop<kScaledX, kMode, kSR, kHad>(x, nblocks, codes, scales, xd, tab, sr, hp, ring);
  } else {
    if (two_term)
      quantize_loop<kTwoTerm, kContig, kMode, kSR, kHad>(x, nbk, ldx, nblocks, codes, scales, xd, tab, sr,
                                                hp);
    else if (direct)
      quantize_loop<kMarkstein, kContig, kMode, kSR, kHad>(x, nbk, ldx, nblocks, codes, scales, xd, tab,
                                                  sr, hp);
    else
      quantize_loop<kScaledX, kContig, kMode, kSR, kHad>(x, nbk, ldx, nblocks, codes, scales, xd, tab, sr,
                                                hp);
  }
}

// Small tensors with the tensor scale computed (at most kSmallElems
// elements): one launch, at most one block per thread.  Every workgroup reads
// the whole tensor for max|X| (a few hundred KB, from L2 after the first), so
// all of them hold the same s32 without talking to each other; workgroup 0
// stores it.  The read walks blocks in the order of the quantize assignment
// (block w * kSmallThreads + t of workgroup w goes to its thread t), so each
// thread keeps its own block from that pass and quantizes it without a
// second read.  The maximum is order-independent: the result is the
// two-pass one, bit for bit.
constexpr int kSmallThreads = 1024;
constexpr int64_t kSmallElems = int64_t(1) << 18;

template <bool kContig, int kMode, bool kSR>
__global__ __launch_bounds__(kSmallThreads) void quantize_small_kernel(
    const uint16_t* __restrict__ x, int64_t nbk, int64_t ldx, int64_t nblocks,
    uint8_t* __restrict__ codes, uint8_t* __restrict__ scales, float* __restrict__ tensor_scale,
    SrParams sr) {
  __shared__ ScaleRecip tab[128];
  __shared__ uint32_t wave_max[kSmallThreads / 64];
  fill_scale_table(tab);
  auto block_ptr = [&](int64_t g) -> const uint16_t* {
    if (kContig) return x + (g << 4);
    const int64_t r = g / nbk;
    return x + r * ldx + ((g - r * nbk) << 4);
  };
  // max|X| as bf16 magnitude bits; eight blocks in flight per thread
  constexpr int kInFlight = 8;
  const int64_t rounds = (nblocks + kSmallThreads - 1) / kSmallThreads;
  const int64_t mine = blockIdx.x;                  // round holding this thread's block
  uint32_t mx = 0u;
  uint4 k0 = make_uint4(0, 0, 0, 0), k1 = k0;
  for (int64_t r0 = 0; r0 < rounds; r0 += kInFlight) {
    uint4 v0[kInFlight], v1[kInFlight];
#pragma unroll
    for (int j = 0; j < kInFlight; ++j) {
      int64_t g = (r0 + j) * kSmallThreads + threadIdx.x;
      g = g < nblocks ? g : nblocks - 1;           // past the end: re-read the last block
      const uint16_t* src = block_ptr(g);
      v0[j] = *reinterpret_cast<const uint4*>(src);
      v1[j] = *reinterpret_cast<const uint4*>(src + 8);
    }
#pragma unroll
    for (int j = 0; j < kInFlight; ++j) {
      mx = max(mx, max(absmax8(v0[j]), absmax8(v1[j])));
      if (r0 + j == mine) {
        k0 = v0[j];
        k1 = v1[j];
      }
    }
  }
  for (int off = 32; off > 0; off >>= 1) mx = max(mx, (uint32_t)__shfl_xor((int)mx, off));
  if ((threadIdx.x & 63) == 0) wave_max[threadIdx.x >> 6] = mx;
  __syncthreads();                                  // also publishes the scale table
  uint32_t r = wave_max[0];
#pragma unroll
  for (int w = 1; w < kSmallThreads / 64; ++w) r = max(r, wave_max[w]);
  const float s32 = tensor_scale_of(r);
  if (blockIdx.x == 0 && threadIdx.x == 0) *tensor_scale = s32;

  const int64_t g = mine * kSmallThreads + threadIdx.x;
  if (g >= nblocks) return;
  const bool direct = s32 >= 0x1p-90f && s32 <= 0x1p120f;
  float xs[16];
  if (direct) {
    to_fp8_domain<false>(k0, k1, 1.0f, s32, __fdiv_rn(1.0f, s32), xs);
  } else {
    const float xmul = s32 < 1.0f ? 0x1p64f : 0x1p-64f;
    const float sx = s32 * xmul;
    to_fp8_domain<true>(k0, k1, xmul, sx, __fdiv_rn(1.0f, sx), xs);
  }
  uint2 out;
  uint32_t sb;
  quantize_xs<kMode, kSR>(xs, tab, out, sb, kSR ? block_draws(g, sr) : make_uint4(0, 0, 0, 0));
  *reinterpret_cast<uint2*>(codes + (g << 3)) = out;
  scales[g] = (uint8_t)sb;
}

// Per-workgroup max|Y| of the rotated tensor (bf16 magnitude bits of the
// rounded results), same lane-per-block walk as the quantizer so that every
// Hadamard block sits in consecutive lanes of one wave.  Results go to
// partials[blockIdx.x] or, without partials, into *out by atomic max.
template <bool kContig>
__global__ __launch_bounds__(kThreads) void amax_rotated_kernel(
    const uint16_t* __restrict__ x, int64_t nbk, int64_t ldx, int64_t nblocks, HadamardParams hp,
    uint32_t* __restrict__ partials, uint32_t* __restrict__ out) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const SignMasks sm = load_sign_masks(hp, (int)(threadIdx.x & ((1u << hp.lanes_log2) - 1u)));
  uint32_t m = 0u;
  for (int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; g < nblocks; g += stride) {
    const uint16_t* src;
    if (kContig) {
      src = x + (g << 4);
    } else {
      const int64_t r = g / nbk;
      src = x + r * ldx + ((g - r * nbk) << 4);
    }
    uint4 v0 = *reinterpret_cast<const uint4*>(src);
    uint4 v1 = *reinterpret_cast<const uint4*>(src + 8);
    hadamard_rotate(v0, v1, sm, hp);
    m = max(m, max(absmax8(v0), absmax8(v1)));
  }
  for (int off = 32; off > 0; off >>= 1) m = max(m, (uint32_t)__shfl_xor((int)m, off));
  __shared__ uint32_t wave_max[kThreads / 64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) wave_max[wave] = m;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t r = wave_max[0];
    for (int w = 1; w < kThreads / 64; ++w) r = max(r, wave_max[w]);
    if (partials) partials[blockIdx.x] = r;
    else if (r) atomicMax(out, r << 16);
  }
}

// Standalone rotation: y[g] = rotated block g (y contiguous [rows, k]).
template <bool kContig>
__global__ __launch_bounds__(kThreads) void hadamard_kernel(const uint16_t* __restrict__ x,
                                                            int64_t nbk, int64_t ldx,
                                                            int64_t nblocks, HadamardParams hp,
                                                            uint16_t* __restrict__ y) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const SignMasks sm = load_sign_masks(hp, (int)(threadIdx.x & ((1u << hp.lanes_log2) - 1u)));
  for (int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; g < nblocks; g += stride) {
    const uint16_t* src;
    if (kContig) {
      src = x + (g << 4);
    } else {
      const int64_t r = g / nbk;
      src = x + r * ldx + ((g - r * nbk) << 4);
    }
    uint4 v0 = *reinterpret_cast<const uint4*>(src);
    uint4 v1 = *reinterpret_cast<const uint4*>(src + 8);
    hadamard_rotate(v0, v1, sm, hp);
    uint4* dst = reinterpret_cast<uint4*>(y + (g << 4));
    dst[0] = v0;
    dst[1] = v1;
  }
}

int grid_for(int64_t work, int per_thread) {
  int64_t g = (work + (int64_t)kThreads * per_thread - 1) / ((int64_t)kThreads * per_thread);
  if (g < 1) g = 1;
  if (g > 65536) g = 65536;
  return (int)g;
}

// Per-workgroup maxima: to the caller's scratch (the scale-byte output, which
// the quantize kernel overwrites afterwards) when it holds at least 16 slots,
// else an atomic on *tensor_scale.  `run(grid, partials, out)` launches the
// maximum kernel; `grid` is capped by the slots.
template <typename Run>
hipError_t tensor_scale_with(int64_t work, int grid, uint8_t* scratch, int64_t scratch_bytes,
                             float* tensor_scale, hipStream_t stream, Run run) {
  const uintptr_t base = reinterpret_cast<uintptr_t>(scratch);
  const uintptr_t aligned = (base + 3u) & ~uintptr_t(3);
  const int64_t slots = scratch ? (scratch_bytes - (int64_t)(aligned - base)) / 4 : 0;
  if (work > 0 && slots >= 16) {
    if (grid > slots) grid = (int)slots;
    uint32_t* partials = reinterpret_cast<uint32_t*>(aligned);
    run(grid, partials, (uint32_t*)nullptr);
    reduce_scale<<<1, kThreads, 0, stream>>>(partials, grid, tensor_scale);
    return hipGetLastError();
  }
  uint32_t* p = reinterpret_cast<uint32_t*>(tensor_scale);
  clear_u32<<<1, 1, 0, stream>>>(p);
  if (work > 0) run(grid, (uint32_t*)nullptr, p);
  finalize_scale<<<1, 1, 0, stream>>>(p);
  return hipGetLastError();
}

}  // namespace

HadamardParams hadamard_params(int b, const int8_t* signs) {
  HadamardParams hp{};
  int level = 0;
  while ((1 << level) < b) ++level;
  hp.signs = signs;
  hp.lanes_log2 = level - 4;
  hp.odd = level & 1;
  // 1 / sqrt(b) = 2^-(level / 2) (times the fp64 sqrt(1/2) for odd levels)
  hp.scale = std::ldexp(hp.odd ? 0.70710678118654752440 : 1.0, -(level / 2));
  hp.b = (double)b;
  return hp;
}

hipError_t launch_tensor_scale(const uint16_t* x, int64_t rows, int64_t k, int64_t ldx,
                               uint8_t* scratch, int64_t scratch_bytes, float* tensor_scale,
                               hipStream_t stream) {
  const int64_t total = rows * (k >> 3);
  if (ldx == k) {
    // one window of 4 KB per wave, four waves per workgroup, at most 4
    // workgroups per CU (a persistent grid for large tensors)
    static ResidentCache cache;
    const int64_t wanted = (total + 4 * kAmaxWindow - 1) / (4 * kAmaxWindow);
    const int64_t resident = resident_groups(amax_stream_kernel, cache, 4);
    const int g = (int)(wanted < resident ? (wanted > 0 ? wanted : 1) : resident);
    return tensor_scale_with(total, g, scratch, scratch_bytes, tensor_scale, stream,
                             [&](int grid, uint32_t* partials, uint32_t* out) {
                               amax_stream_kernel<<<grid, kThreads, 0, stream>>>(x, total,
                                                                                  partials, out);
                             });
  }
  // up to 1024 workgroups x 256 threads x 4 loads of 16 B keeps ~16 MB in flight
  int g = grid_for(total, 4);
  if (g > 1024) g = 1024;
  return tensor_scale_with(total, g, scratch, scratch_bytes, tensor_scale, stream,
                           [&](int grid, uint32_t* partials, uint32_t* out) {
                             amax_kernel<<<grid, kThreads, 0, stream>>>(x, rows, k, ldx, partials,
                                                                         out);
                           });
}

hipError_t launch_tensor_scale_rotated(const uint16_t* x, int64_t rows, int64_t k, int64_t ldx,
                                       const HadamardParams& hp, uint8_t* scratch,
                                       int64_t scratch_bytes, float* tensor_scale,
                                       hipStream_t stream) {
  const int64_t nbk = k / kBlock, nblocks = rows * nbk;
  static ResidentCache cache_c, cache_s;
  const int64_t resident = ldx == k ? resident_groups(amax_rotated_kernel<true>, cache_c)
                                    : resident_groups(amax_rotated_kernel<false>, cache_s);
  const int64_t wanted = (nblocks + kThreads - 1) / kThreads;
  int g = (int)(wanted < resident ? wanted : resident);
  if (g < 1) g = 1;
  return tensor_scale_with(nblocks, g, scratch, scratch_bytes, tensor_scale, stream,
                           [&](int grid, uint32_t* partials, uint32_t* out) {
                             if (ldx == k)
                               amax_rotated_kernel<true><<<grid, kThreads, 0, stream>>>(
                                   x, nbk, ldx, nblocks, hp, partials, out);
                             else
                               amax_rotated_kernel<false><<<grid, kThreads, 0, stream>>>(
                                   x, nbk, ldx, nblocks, hp, partials, out);
                           });
}

namespace {

template <int kMode, bool kSR>
hipError_t launch_small_mode(const uint16_t* x, int64_t rows, int64_t k, int64_t ldx,
                             uint8_t* codes, uint8_t* scales, float* tensor_scale,
                             const SrParams& sr, hipStream_t stream) {
  const int64_t nbk = k / kBlock, nblocks = rows * nbk;
  const int64_t g = (nblocks + kSmallThreads - 1) / kSmallThreads;   // one block per thread
  if (ldx == k)
    quantize_small_kernel<true, kMode, kSR><<<(unsigned)g, kSmallThreads, 0, stream>>>(
        x, nbk, ldx, nblocks, codes, scales, tensor_scale, sr);
  else
    quantize_small_kernel<false, kMode, kSR><<<(unsigned)g, kSmallThreads, 0, stream>>>(
        x, nbk, ldx, nblocks, codes, scales, tensor_scale, sr);
  return hipGetLastError();
}

template <int kMode, bool kSR, bool kHad>
hipError_t launch_mode(const uint16_t* x, int64_t rows, int64_t k, int64_t ldx, uint8_t* codes,
                       uint8_t* scales, const float* tensor_scale, const QuantOptions& opt,
                       hipStream_t stream) {
  const int64_t nbk = k / kBlock;
  const int64_t nblocks = rows * nbk;
  static ResidentCache cache_c, cache_s, capped_c, capped_s;
  if (ldx == k && !kHad) {
    // Contiguous X (stream_loop): one window of 64 blocks per wave, four
    // per workgroup; a tensor with more windows is walked by a persistent
    // grid of at most 3 workgroups per CU (measured on the 2^28 tensor: 3,
    // 4 and 6 per CU within 3% for every mode, 3 the fastest or tied).
    constexpr int kStreamPerCU = 3;
    const int64_t wanted = (nblocks + kThreads - 1) / kThreads;
    const int64_t capped =
        resident_groups(quantize_kernel<true, kMode, kSR, kHad>, capped_c, kStreamPerCU);
    const int g = (int)(wanted <= capped ? wanted : capped);
    quantize_kernel<true, kMode, kSR, kHad><<<g, kThreads, 0, stream>>>(
        x, nbk, ldx, nblocks, codes, scales, tensor_scale, opt.srp, opt.hp);
    return hipGetLastError();
  }
  // Row-strided X: a tensor that one round of resident workgroups covers
  // gets one block per thread.  Larger ones are walked by a persistent grid,
  // one wave of resident workgroups, so no partial second wave is left at
  // the end, with at most kMaxPerCU workgroups per CU.  The single-format
  // encodings do little arithmetic per byte and stream HBM better with fewer
  // resident waves than their registers allow (E2M1-only at 3 workgroups per
  // CU against 8: 118 us against 137 us on a contiguous 2^28 tensor;
  // E1M2-only is best at 4).  For the other modes 4 to 8 measure the same.
  constexpr int kMaxPerCU = kMode == kForceE2M1 ? 3 : (kMode == kForceE1M2 ? 4 : 6);
  const int64_t wanted = (nblocks + kThreads - 1) / kThreads;
  const bool contig = ldx == k;
  const int64_t resident =
      contig ? resident_groups(quantize_kernel<true, kMode, kSR, kHad>, cache_c)
             : resident_groups(quantize_kernel<false, kMode, kSR, kHad>, cache_s);
  const int64_t capped =
      contig ? resident_groups(quantize_kernel<true, kMode, kSR, kHad>, capped_c, kMaxPerCU)
             : resident_groups(quantize_kernel<false, kMode, kSR, kHad>, capped_s, kMaxPerCU);
  const int g = (int)(wanted <= resident ? wanted : capped);
  if (contig)
    quantize_kernel<true, kMode, kSR, kHad><<<g, kThreads, 0, stream>>>(
        x, nbk, ldx, nblocks, codes, scales, tensor_scale, opt.srp, opt.hp);
  else
    quantize_kernel<false, kMode, kSR, kHad><<<g, kThreads, 0, stream>>>(
        x, nbk, ldx, nblocks, codes, scales, tensor_scale, opt.srp, opt.hp);
  return hipGetLastError();
}

template <int kMode>
hipError_t launch_mode_opts(const uint16_t* x, int64_t rows, int64_t k, int64_t ldx,
                            uint8_t* codes, uint8_t* scales, const float* tensor_scale,
                            const QuantOptions& opt, hipStream_t stream) {
  if (opt.sr)
    return opt.had ? launch_mode<kMode, true, true>(x, rows, k, ldx, codes, scales, tensor_scale,
                                                    opt, stream)
                   : launch_mode<kMode, true, false>(x, rows, k, ldx, codes, scales,
                                                     tensor_scale, opt, stream);
  return opt.had ? launch_mode<kMode, false, true>(x, rows, k, ldx, codes, scales, tensor_scale,
                                                   opt, stream)
                 : launch_mode<kMode, false, false>(x, rows, k, ldx, codes, scales, tensor_scale,
                                                    opt, stream);
}

template <int kMode>
hipError_t launch_small_opts(const uint16_t* x, int64_t rows, int64_t k, int64_t ldx,
                             uint8_t* codes, uint8_t* scales, float* tensor_scale,
                             const QuantOptions& opt, hipStream_t stream) {
  return opt.sr ? launch_small_mode<kMode, true>(x, rows, k, ldx, codes, scales, tensor_scale,
                                                 opt.srp, stream)
                : launch_small_mode<kMode, false>(x, rows, k, ldx, codes, scales, tensor_scale,
                                                  opt.srp, stream);
}

}  // namespace

hipError_t launch_quantize_small(const uint16_t* x, int64_t rows, int64_t k, int64_t ldx,
                                 uint8_t* codes, uint8_t* scales, float* tensor_scale,
                                 const QuantOptions& opt, hipStream_t stream) {
  if (opt.mode == kFourSix)
    return launch_small_opts<kFourSix>(x, rows, k, ldx, codes, scales, tensor_scale, opt, stream);
  if (opt.mode == kForceE2M1)
    return launch_small_opts<kForceE2M1>(x, rows, k, ldx, codes, scales, tensor_scale, opt, stream);
  if (opt.mode == kForceE1M2)
    return launch_small_opts<kForceE1M2>(x, rows, k, ldx, codes, scales, tensor_scale, opt, stream);
  return launch_small_opts<kSelect>(x, rows, k, ldx, codes, scales, tensor_scale, opt, stream);
}

bool quantize_is_small(int64_t rows, int64_t k) { return rows * k <= kSmallElems; }

hipError_t launch_quantize(const uint16_t* x, int64_t rows, int64_t k, int64_t ldx,
                           uint8_t* codes, uint8_t* scales, const float* tensor_scale,
                           const QuantOptions& opt, hipStream_t stream) {
  if (rows * (k / kBlock) == 0) return hipSuccess;
  if (opt.mode == kFourSix)
    return launch_mode_opts<kFourSix>(x, rows, k, ldx, codes, scales, tensor_scale, opt, stream);
  if (opt.mode == kForceE2M1)
    return launch_mode_opts<kForceE2M1>(x, rows, k, ldx, codes, scales, tensor_scale, opt, stream);
  if (opt.mode == kForceE1M2)
    return launch_mode_opts<kForceE1M2>(x, rows, k, ldx, codes, scales, tensor_scale, opt, stream);
  return launch_mode_opts<kSelect>(x, rows, k, ldx, codes, scales, tensor_scale, opt, stream);
}

hipError_t launch_hadamard(const uint16_t* x, int64_t rows, int64_t k, int64_t ldx,
                           const HadamardParams& hp, uint16_t* y, hipStream_t stream) {
  const int64_t nbk = k / kBlock, nblocks = rows * nbk;
  if (nblocks == 0) return hipSuccess;
  static ResidentCache cache_c, cache_s;
  const int64_t resident = ldx == k ? resident_groups(hadamard_kernel<true>, cache_c)
                                    : resident_groups(hadamard_kernel<false>, cache_s);
  const int64_t wanted = (nblocks + kThreads - 1) / kThreads;
  const int g = (int)(wanted < resident ? wanted : resident);
  if (ldx == k)
    hadamard_kernel<true><<<g, kThreads, 0, stream>>>(x, nbk, ldx, nblocks, hp, y);
  else
    hadamard_kernel<false><<<g, kThreads, 0, stream>>>(x, nbk, ldx, nblocks, hp, y);
  return hipGetLastError();
}

}  // namespace mixfp4
