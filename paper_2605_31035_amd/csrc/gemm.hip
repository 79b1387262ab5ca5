// MixFP4 block-scaled GEMM for gfx950: C[m, n] = s32_A s32_W sum_k a[m,k] w[n,k].
//
// Numerics.  Sec. 3.3 / App. B.5 decode both micro-formats into one value
// set (E2M2): E2M1 magnitudes gain a zero mantissa bit, E1M2 magnitudes go
// through a small table, T (scale bit 7) selects the path.  Here the unified
// value v is multiplied by the block's E4M3 scale s8 during decode: s8 has at
// most 4 significant bits and v at most 3, so a = s8 * v has at most 7 and lies
// in [2^-10, 3136] -- exact in fp16 (normal range, 11-bit significand).  The
// fp16 operands feed v_mfma_f32_32x32x16_f16 (the bf16 rate) with fp32
// accumulation (the paper keeps FP16/FP32 accumulation unchanged, Sec. 3.3);
// the two fp32 tensor scales are applied once in the epilogue.  App. B.1's
// factored per-block scale is not needed because the per-element decode is
// exact.
//
// Decode.  Every unscaled unified value (E2M1 {0,.5,1,1.5,2,3,4,6}, E1M2 x2 =
// INT4 {0..7}) has a zero low byte in fp16, so the 8 magnitudes of a codebook
// are one 8-byte constant of high bytes.  A code dword (8 nibbles) decodes
// with v_perm_b32 byte lookups into that constant (picked by T), the nibble
// sign bit is OR-ed in, two more perms place the bytes as fp16 pairs, and
// v_pk_mul_f16 multiplies by s8 (E4M3 -> fp32 by the hardware converter,
// then to an fp16 pair).  No lookup depends on the scale byte, so decoding
// reads nothing from LDS.  The decoded 8 values are kept in the order
// [e0 e2 e4 e6 e1 e3 e5 e7]; A and W use the same order, and a dot product
// does not depend on the order of k.
//
// Tiling.  A workgroup of 64 * WM * WN threads owns a BM x BN tile of C; each
// wave owns (BM/WM) x (BN/WN) as 32 x 32 MFMA tiles.  The K loop steps 64
// (four 16-element scale blocks).  Per step every thread loads the packed
// codes + scale bytes of (BM+BN)/threads rows two steps ahead into
// registers, decodes the next step's rows into the idle half of a
// double-buffered LDS tile while the waves run MFMAs from the other half, so
// every element is decoded once per workgroup and one barrier separates the
// steps.  LDS layout per buffer: [slice s (16 K)][half h (8 K)][row of A|W]
// [16 B]; the 64 lanes of a fragment read and the threads of a decode write
// both hit consecutive 16-byte words.  Rows beyond m / n and blocks beyond k
// decode as zeros; stores are masked.
#include <type_traits>

#include "decode.h"
#include "formats.h"
#include "internal.h"
#include "quant_block.h"
#include "tile_order.h"

namespace mixfp4 {
namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kStepBlocks = 4;               // scale blocks per K step (64 elements)

template <int BM, int BN, int WM, int WN>
struct Tile {
  static constexpr int kThreads = 64 * WM * WN;
  static constexpr int kRowsAll = BM + BN;                 // A rows then W rows
  static constexpr int kRowsPerThread = (kRowsAll + kThreads - 1) / kThreads;
  static constexpr bool kEven = kRowsAll % kThreads == 0;  // every thread decodes R rows
  static constexpr int kWaveM = BM / WM, kWaveN = BN / WN;
  static constexpr int kTM = kWaveM / 32, kTN = kWaveN / 32;
  // uint4 words per (slice, half) plane and per buffer
  static constexpr int kPlane = kRowsAll;
  static constexpr int kBuf = kStepBlocks * 2 * kPlane;
  static_assert(kTM >= 1 && kTN >= 1, "wave tile must hold whole 32x32 MFMA tiles");
};

// Packed inputs of one row for one K step: 4 code qwords (4 blocks) + 4 scale bytes.
struct RowPack {
  uint2 c[kStepBlocks];
  uint32_t s;   // scale bytes, block b in byte b
};

// Fast path (k % 64 == 0, word-aligned scales): rows are clamped into range
// and the step index into [0, steps), so loads never branch and never leave
// the operands; data of clamped rows only reaches masked-out outputs, data of
// clamped steps is never decoded into a buffer that is read.
__device__ __forceinline__ void load_row_fast(RowPack& p, const uint8_t* __restrict__ crow,
                                              const uint8_t* __restrict__ srow, int64_t kb0) {
  const uint4 lo = *reinterpret_cast<const uint4*>(crow + kb0 * 8);
  const uint4 hi = *reinterpret_cast<const uint4*>(crow + kb0 * 8 + 16);
  p.c[0] = make_uint2(lo.x, lo.y);
  p.c[1] = make_uint2(lo.z, lo.w);
  p.c[2] = make_uint2(hi.x, hi.y);
  p.c[3] = make_uint2(hi.z, hi.w);
  p.s = *reinterpret_cast<const uint32_t*>(srow + kb0);
}

// General path: blocks beyond k and rows beyond m / n load as zeros.
__device__ __forceinline__ void load_row_masked(RowPack& p, const uint8_t* __restrict__ crow,
                                                const uint8_t* __restrict__ srow, bool row_ok,
                                                int64_t kb0, int64_t kb_total) {
  p.s = 0u;
#pragma unroll
  for (int b = 0; b < kStepBlocks; ++b) {
    const bool ok = row_ok && (kb0 + b) < kb_total;
    p.c[b] = ok ? *reinterpret_cast<const uint2*>(crow + (kb0 + b) * 8) : make_uint2(0u, 0u);
    p.s |= (ok ? (uint32_t)srow[kb0 + b] : 0u) << (8 * b);
  }
}

// Scheduling hints for one K slice: N_READ LDS loads, then N_MFMA times
// (one MFMA, four VALU), then N_WRITE LDS stores.
template <int N>
__device__ __forceinline__ void sched_mfma_valu() {
  if constexpr (N > 0) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x002, 4, 0);
    sched_mfma_valu<N - 1>();
  }
}
template <int N_READ, int N_MFMA, int N_WRITE>
__device__ __forceinline__ void sched_slice() {
  __builtin_amdgcn_sched_group_barrier(0x100, N_READ, 0);
  sched_mfma_valu<N_MFMA>();
  __builtin_amdgcn_sched_group_barrier(0x200, N_WRITE, 0);
}

template <int BM, int BN, int WM, int WN, bool kFast, bool kSchedule>
__global__ __launch_bounds__(64 * WM * WN, 1) void gemm_kernel(
    const uint8_t* __restrict__ a_codes, const uint8_t* __restrict__ a_scales,
    const float* __restrict__ a_ts, const uint8_t* __restrict__ w_codes,
    const uint8_t* __restrict__ w_scales, const float* __restrict__ w_ts, int64_t m,
    int64_t n, int64_t k, float* __restrict__ c, int64_t ldc) {
  using T = Tile<BM, BN, WM, WN>;
  constexpr int R = T::kRowsPerThread;
  // Two separate buffers (not one indexed array) so the compiler can see that
  // the decode stores of one step never alias the fragment loads of the other
  // and may interleave them with the MFMAs.
  __shared__ uint4 lds0[T::kBuf];
  __shared__ uint4 lds1[T::kBuf];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int64_t kb_total = k / kBlock;
  const int64_t code_pitch = k / 2;
  const int64_t steps = (kb_total + kStepBlocks - 1) / kStepBlocks;
  const int64_t ntm = (m + BM - 1) / BM, ntn = (n + BN - 1) / BN;
  const int64_t tile = grouped_tile(xcd_item(blockIdx.x, gridDim.x), ntm, ntn);
  const int64_t s_begin = 0, s_end = steps;
  const int64_t m0 = (tile / ntn) * BM;
  const int64_t n0 = (tile % ntn) * BN;
  const int wm = (wave / WN) * T::kWaveM, wn = (wave % WN) * T::kWaveN;

  // rows this thread decodes: g = tid + threads * r over [A rows | W rows]
  const uint8_t* rc[R];
  const uint8_t* rs[R];
  bool rok[R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    // threads past the last row of an uneven split load row 0 of A (never
    // decoded) so that their loads stay in bounds
    const int g0 = tid + T::kThreads * r;
    const bool in_tile = T::kEven || g0 < T::kRowsAll;
    const int g = in_tile ? g0 : 0;
    const bool is_a = g < BM;
    int64_t row = is_a ? m0 + g : n0 + (g - BM);
    const int64_t lim = is_a ? m : n;
    rok[r] = in_tile && row < lim;
    if (kFast && row >= lim) row = lim - 1;
    rc[r] = (is_a ? a_codes : w_codes) + row * code_pitch;
    rs[r] = (is_a ? a_scales : w_scales) + row * kb_total;
  }

  auto load_step = [&](RowPack (&p)[R], int64_t step) {
#pragma unroll
    for (int r = 0; r < R; ++r) {
      if (kFast) {
        const int64_t st = step < s_end ? step : s_end - 1;
        load_row_fast(p[r], rc[r], rs[r], st * kStepBlocks);
      } else {
        load_row_masked(p[r], rc[r], rs[r], rok[r], step * kStepBlocks, kb_total);
      }
    }
  };
  auto decode_block = [&](const RowPack (&p)[R], uint4* wr, int b) {
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int g = tid + T::kThreads * r;
      if (!T::kEven && g >= T::kRowsAll) continue;
      const BlockDec d = block_dec((p[r].s >> (8 * b)) & 0xFFu);
      uint4* dst = wr + (b * 2) * T::kPlane + g;
      dst[0] = decode8(p[r].c[b].x, d);
      dst[T::kPlane] = decode8(p[r].c[b].y, d);
    }
  };

  f32x16 acc[T::kTM][T::kTN];
#pragma unroll
  for (int i = 0; i < T::kTM; ++i)
#pragma unroll
    for (int j = 0; j < T::kTN; ++j)
#pragma unroll
      for (int q = 0; q < 16; ++q) acc[i][j][q] = 0.0f;

  const int half = lane >> 5, lrow = lane & 31;
  // One K step: MFMAs over `rd`, interleaved with decoding `p` (the next
  // step) into `wr`; `pn` receives the step after that.
  auto body = [&](const uint4* rd, uint4* wr, const RowPack (&p)[R], RowPack (&pn)[R],
                  int64_t s, bool decode) {
    if (decode) load_step(pn, s + 2);
    // keep the prefetch at the top of the step so its latency hides under the MFMAs
    __builtin_amdgcn_sched_barrier(0);
    f16x8 fa[2][T::kTM], fw[2][T::kTN];
    auto load_frags = [&](int buf, int sl) {
      const uint4* plane = rd + (sl * 2 + half) * T::kPlane;
#pragma unroll
      for (int i = 0; i < T::kTM; ++i)
        fa[buf][i] = __builtin_bit_cast(f16x8, plane[wm + i * 32 + lrow]);
#pragma unroll
      for (int j = 0; j < T::kTN; ++j)
        fw[buf][j] = __builtin_bit_cast(f16x8, plane[BM + wn + j * 32 + lrow]);
    };
    load_frags(0, 0);
#pragma unroll
    for (int sl = 0; sl < kStepBlocks; ++sl) {
      const int cb = sl & 1;
      if (sl + 1 < kStepBlocks) load_frags(cb ^ 1, sl + 1);   // next slice's fragments
#pragma unroll
      for (int i = 0; i < T::kTM; ++i)
#pragma unroll
        for (int j = 0; j < T::kTN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(fa[cb][i], fw[cb][j], acc[i][j], 0, 0, 0);
      if (decode) decode_block(p, wr, sl);
    }
    if constexpr (kSchedule) {
      // Per slice: the next slice's fragment loads, then every MFMA followed
      // by a few decode VALU ops, then the decoded stores.
      sched_slice<T::kTM + T::kTN + R, T::kTM * T::kTN, 2 * R>();
      sched_slice<T::kTM + T::kTN + R, T::kTM * T::kTN, 2 * R>();
      sched_slice<T::kTM + T::kTN + R, T::kTM * T::kTN, 2 * R>();
      sched_slice<R, T::kTM * T::kTN, 2 * R>();
    }
  };

  RowPack pa[R], pb[R];
  load_step(pa, s_begin);
#pragma unroll
  for (int b = 0; b < kStepBlocks; ++b) decode_block(pa, lds0, b);
  load_step(pa, s_begin + 1);

  // Step s reads buffer (s-s_begin)%2 and decodes step s+1 into the other
  // one; one barrier per step orders "decoded" before "read" and "read"
  // before "overwritten".  On the fast path the last step decodes clamped
  // data into a buffer that is never read again.  Steps run in branch-free
  // pairs (an odd last step is peeled) so that each pair is one basic block:
  // the prefetch issued at the top of a step then stays there instead of
  // being sunk into the next step's block right before its use.
  int64_t s = s_begin;
  for (; s + 1 < s_end; s += 2) {
    __syncthreads();
    body(lds0, lds1, pa, pb, s, kFast || s + 1 < s_end);
    __syncthreads();
    body(lds1, lds0, pb, pa, s + 1, kFast || s + 2 < s_end);
  }
  if (s < s_end) {
    __syncthreads();
    body(lds0, lds1, pa, pb, s, kFast);
  }

  const float scale = (a_ts ? *a_ts : 1.0f) * (w_ts ? *w_ts : 1.0f);
  // 32 x 32 accumulator layout: lane holds column lane%32; register q holds
  // row 8*(q/4) + 4*(lane/32) + q%4.
#pragma unroll
  for (int i = 0; i < T::kTM; ++i)
#pragma unroll
    for (int j = 0; j < T::kTN; ++j) {
      const int64_t col = n0 + wn + j * 32 + lrow;
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const int64_t row = m0 + wm + i * 32 + 8 * (q >> 2) + 4 * half + (q & 3);
        if (row < m && col < n) c[row * ldc + col] = acc[i][j][q] * scale;
      }
    }
}

// ---------------------------------------------------------------------------
// Decode-shape GEMM (m <= 16): HBM-bound, W is read once.
//
// A workgroup owns 16 G columns of C (G = 1 to 8 MFMA column groups, so that
// one workgroup per CU covers W): one range of G groups for G <= 6, or for
// G = 7, 8 two ranges of 4 and G - 4 groups worked on at the same time by two
// sets of kW waves (two waves per SIMD).  A set splits K (k % 64 == 0) over
// its kW waves in whole 256-wide steps, the last wave also taking the rest of
// K % 256 as a tail step (skinny_waves: 2 equal shares when
// floor(k / 256) is 2 mod 4, else 4 shares that differ by at most one step); each
// wave walks its K range in steps of 256 with no barrier and no LDS until the
// end.  Lane (nn, g) = (lane % 16, lane / 16) owns W rows
// nn + 16 c (c < kCG, one per 16-column group) and the quarter
// [64 g, 64 g + 64) of every step: per row 32 code bytes and 4 scale bytes,
// loaded one step ahead.  It decodes them straight into the B operands of
// v_mfma_f32_16x16x32_f16, and decodes its own A operand -- A row nn, the
// same 64 elements -- once per step for all its column groups.  MFMA i of a
// 32-element group takes elements 8 i + j in K slot (g, j); A and W use the
// same order.  The waves' partial sums are added through LDS in a fixed
// order at the end, so every column's sum is formed in the same order
// whatever kCG is.
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kSkinnyRows = 16;
constexpr int kSkinnyStep = 256;                   // K per wave step
constexpr int kSkinnyK = 64;                       // K multiple the kernel takes (a lane's share of a step)
constexpr int kSkinnyVec = kSkinnyStep / 128;      // 16-byte code loads per row per lane per step
constexpr int kSkinnySw = kSkinnyStep / 256;       // scale dwords per row per lane per step

template <int kCG>
struct WPack {
  uint4 c[kCG][kSkinnyVec];     // kCG rows x 64 codes
  uint32_t s[kCG][kSkinnySw];   // their scale bytes
};
struct APack {
  uint4 c[kSkinnyVec];
  uint32_t s[kSkinnySw];
};

// The body of the decode-shape GEMM for columns [col0, col0 + 16 ng), run by
// one set of kW waves (`wave` = 0 .. kW - 1 within the set) with its own
// reduction buffer `red`.  With kMasked, only the first ng <= kCG groups are
// active (uniform: a set of the shorter range skips the last group's loads
// and work); otherwise all kCG are.  `before_a` runs
// once, after this lane's first W loads are issued and before any A load; it
// returns false to poison these outputs (NaN) when A never became available.
template <int kW, int kCG, bool kMasked, typename BeforeA>
__device__ __forceinline__ void skinny_body(
    int wave, f32x4 (*red)[kCG][64], int ng, int64_t col0, const uint8_t* __restrict__ a_codes,
    const uint8_t* __restrict__ a_scales, const float* __restrict__ a_ts,
    const uint8_t* __restrict__ w_codes, const uint8_t* __restrict__ w_scales,
    const float* __restrict__ w_ts, int64_t m, int64_t n, int64_t k, float* __restrict__ c,
    BeforeA before_a) {
  const int lane = threadIdx.x & 63;
  const int nn = lane & 15, g = lane >> 4;
  auto active = [&](int cg) { return !kMasked || cg < ng; };
  const int64_t code_pitch = k / 2, scale_pitch = k / kBlock;
  // this wave's K range: steps [S w / kW, S (w + 1) / kW) of the S = k / 256
  // (an equal share when kW divides S; a wave may have none when S < kW)
  const int64_t total_steps = k / kSkinnyStep;
  const int64_t s_first = total_steps * wave / kW;
  const int64_t steps = total_steps * (wave + 1) / kW - s_first;
  const int64_t kbase = s_first * kSkinnyStep;
  // K % 256 = 64, 128 or 192: the set's last wave takes one more step after
  // its range, the tail, in which the lanes past it (64 g >= tail) get zeros
  const int tail = (int)(k % kSkinnyStep);
  const bool has_tail = tail != 0 && wave == kW - 1;
  const uint8_t* wc[kCG];
  const uint8_t* ws[kCG];
#pragma unroll
  for (int cg = 0; cg < kCG; ++cg) {
    int64_t r = col0 + 16 * cg + nn;
    r = r < n ? r : n - 1;                          // clamped rows feed masked-out columns
    wc[cg] = w_codes + r * code_pitch + kbase / 2 + (kSkinnyStep / 8) * g;
    ws[cg] = w_scales + r * scale_pitch + kbase / 16 + (kSkinnyStep / 64) * g;
  }
  const int64_t arow = nn < m ? nn : m - 1;
  const uint8_t* ac = a_codes + arow * code_pitch + kbase / 2 + (kSkinnyStep / 8) * g;
  const uint8_t* as = a_scales + arow * scale_pitch + kbase / 16 + (kSkinnyStep / 64) * g;
  auto load_w = [&](WPack<kCG>& p, int64_t st) {
    st = st < steps ? st : steps - 1;
#pragma unroll
    for (int cg = 0; cg < kCG; ++cg)
      if (active(cg)) {
#pragma unroll
        for (int v = 0; v < kSkinnyVec; ++v)
          p.c[cg][v] = *reinterpret_cast<const uint4*>(wc[cg] + (kSkinnyStep / 2) * st + 16 * v);
      }
#pragma unroll
    for (int cg = 0; cg < kCG; ++cg)
      if (active(cg)) {
#pragma unroll
        for (int v = 0; v < kSkinnySw; ++v)
          p.s[cg][v] = *reinterpret_cast<const uint32_t*>(ws[cg] + (kSkinnyStep / 16) * st + 4 * v);
      }
  };
  auto load_a = [&](APack& p, int64_t st) {
    st = st < steps ? st : steps - 1;
#pragma unroll
    for (int v = 0; v < kSkinnyVec; ++v)
      p.c[v] = *reinterpret_cast<const uint4*>(ac + (kSkinnyStep / 2) * st + 16 * v);
#pragma unroll
    for (int v = 0; v < kSkinnySw; ++v)
      p.s[v] = *reinterpret_cast<const uint32_t*>(as + (kSkinnyStep / 16) * st + 4 * v);
  };
  f32x4 acc[kCG];
#pragma unroll
  for (int cg = 0; cg < kCG; ++cg) acc[cg] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
  auto compute = [&](const APack& pa, const WPack<kCG>& pw) {
    BlockDec dA[4];
    block_dec4(pa.s[0], dA);
    BlockDec dW[kCG][4];
#pragma unroll
    for (int cg = 0; cg < kCG; ++cg)
      if (active(cg)) block_dec4(pw.s[cg][0], dW[cg]);
#pragma unroll
    for (int v = 0; v < kSkinnyVec; ++v) {
      // 16-byte word v holds 32 elements = blocks 2v, 2v + 1 (scale bytes 2v, 2v + 1)
      const BlockDec da0 = dA[2 * v], da1 = dA[2 * v + 1];
      const uint32_t ca[4] = {pa.c[v].x, pa.c[v].y, pa.c[v].z, pa.c[v].w};
      f16x8 fa[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) fa[i] = __builtin_bit_cast(f16x8, decode8(ca[i], i < 2 ? da0 : da1));
#pragma unroll
      for (int cg = 0; cg < kCG; ++cg) {
        if (!active(cg)) continue;
        const BlockDec d0 = dW[cg][2 * v], d1 = dW[cg][2 * v + 1];
        const uint32_t cw[4] = {pw.c[cg][v].x, pw.c[cg][v].y, pw.c[cg][v].z, pw.c[cg][v].w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const f16x8 fb = __builtin_bit_cast(f16x8, decode8(cw[i], i < 2 ? d0 : d1));
          acc[cg] = __builtin_amdgcn_mfma_f32_16x16x32_f16(fa[i], fb, acc[cg], 0, 0, 0);
        }
      }
    }
  };
  // Two packs alternate: step s computes pack s % 2 after issuing the loads of
  // step s + 1 into the other one (free since step s - 1).  The pair-unrolled
  // loop keeps the pack indices static, so no pack is copied while its loads
  // are in flight.
  WPack<kCG> wp[2];
  APack ap[2];
  if (steps > 0) load_w(wp[0], 0);
  const bool a_ok = before_a();                     // every wave: it may synchronize
  if (steps > 0) load_a(ap[0], 0);
  auto step = [&](auto I_, int64_t s) {
    constexpr int I = decltype(I_)::value;
    __builtin_amdgcn_sched_barrier(0);
    load_a(ap[I ^ 1], s + 1);
    load_w(wp[I ^ 1], s + 1);
    __builtin_amdgcn_sched_barrier(0);
    compute(ap[I], wp[I]);
  };
  using I0 = std::integral_constant<int, 0>;
  using I1 = std::integral_constant<int, 1>;
  int64_t s = 0;
  for (; s + 1 < steps; s += 2) {
    step(I0{}, s);
    step(I1{}, s + 1);
  }
  if (s < steps) step(I0{}, s);
  if (has_tail) {
    // the tail follows this wave's range (step `steps`); a lane past it
    // loads its row's first tail piece instead and zeroes it
    const bool in_tail = kSkinnyVec * 32 * g < tail;
    const int64_t back = in_tail ? 0 : (kSkinnyStep / 8) * g;     // code bytes back to piece 0
    const int64_t sback = in_tail ? 0 : (kSkinnyStep / 64) * g;   // scale bytes back
    const uint4 z4 = make_uint4(0u, 0u, 0u, 0u);
    WPack<kCG> tw;
    APack ta;
#pragma unroll
    for (int cg = 0; cg < kCG; ++cg)
      if (active(cg)) {
#pragma unroll
        for (int v = 0; v < kSkinnyVec; ++v) {
          const uint4 x = *reinterpret_cast<const uint4*>(wc[cg] - back + (kSkinnyStep / 2) * steps + 16 * v);
          tw.c[cg][v] = in_tail ? x : z4;
        }
#pragma unroll
        for (int v = 0; v < kSkinnySw; ++v) {
          const uint32_t x = *reinterpret_cast<const uint32_t*>(ws[cg] - sback + (kSkinnyStep / 16) * steps + 4 * v);
          tw.s[cg][v] = in_tail ? x : 0u;
        }
      }
#pragma unroll
    for (int v = 0; v < kSkinnyVec; ++v) {
      const uint4 x = *reinterpret_cast<const uint4*>(ac - back + (kSkinnyStep / 2) * steps + 16 * v);
      ta.c[v] = in_tail ? x : z4;
    }
#pragma unroll
    for (int v = 0; v < kSkinnySw; ++v) {
      const uint32_t x = *reinterpret_cast<const uint32_t*>(as - sback + (kSkinnyStep / 16) * steps + 4 * v);
      ta.s[v] = in_tail ? x : 0u;
    }
    compute(ta, tw);
  }

  if (wave > 0) {
#pragma unroll
    for (int cg = 0; cg < kCG; ++cg) red[wave - 1][cg][lane] = acc[cg];
  }
  __syncthreads();
  if (wave == 0) {
    const float scale = a_ok ? (a_ts ? *a_ts : 1.0f) * (w_ts ? *w_ts : 1.0f) : __builtin_nanf("");
#pragma unroll
    for (int cg = 0; cg < kCG; ++cg) {
      if (!active(cg)) continue;
      f32x4 t = acc[cg];
#pragma unroll
      for (int w = 0; w < kW - 1; ++w) t += red[w][cg][lane];
      const int64_t col = col0 + 16 * cg + nn;
      // 16 x 16 accumulator layout: lane holds column lane%16, register r holds row 4*(lane/16) + r
      if (col < n) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int row = 4 * g + r;
          if (row < m) c[row * n + col] = t[r] * scale;
        }
      }
    }
  }
}

// Columns [16 (kA + kB) b, 16 (kA + kB) (b + 1)) of workgroup b: kA groups
// (kB = 0: one range, kW waves), or waves 0 .. kW - 1 on kA = 4 groups and
// waves kW .. 2 kW - 1 on the kB <= 4 groups after them, both with the same
// body.  Each column's sum is formed in the same order whatever the split, so
// C does not depend on it.
template <int kA, int kB>
constexpr int skinny_sets() { return kB > 0 ? 2 : 1; }

template <int kW, int kA, int kB, typename BeforeA>
__device__ __forceinline__ void skinny_columns(
    const uint8_t* __restrict__ a_codes, const uint8_t* __restrict__ a_scales,
    const float* __restrict__ a_ts, const uint8_t* __restrict__ w_codes,
    const uint8_t* __restrict__ w_scales, const float* __restrict__ w_ts, int64_t m,
    int64_t n, int64_t k, float* __restrict__ c, BeforeA before_a) {
  static_assert(kB == 0 || (kA == 4 && kB <= 4), "two ranges are 4 + (1 .. 4) groups");
  __shared__ f32x4 red[skinny_sets<kA, kB>()][kW - 1][kA][64];
  const int64_t col0 = (int64_t)blockIdx.x * 16 * (kA + kB);
  const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const int set = wave / kW;
  skinny_body<kW, kA, (kB > 0)>(wave - set * kW, red[set], set ? kB : kA, col0 + set * 16 * kA,
                                a_codes, a_scales, a_ts, w_codes, w_scales, w_ts, m, n, k, c,
                                before_a);
}

template <int kW, int kA, int kB>
__global__ __launch_bounds__(64 * kW * (kB > 0 ? 2 : 1)) void gemm_skinny_kernel(
    const uint8_t* __restrict__ a_codes, const uint8_t* __restrict__ a_scales,
    const float* __restrict__ a_ts, const uint8_t* __restrict__ w_codes,
    const uint8_t* __restrict__ w_scales, const float* __restrict__ w_ts, int64_t m,
    int64_t n, int64_t k, float* __restrict__ c) {
  skinny_columns<kW, kA, kB>(a_codes, a_scales, a_ts, w_codes, w_scales, w_ts, m, n, k, c,
                             []() { return true; });
}

// ---------------------------------------------------------------------------
// One-launch decode step: tensor scale and MixFP4 quantization of the
// activation A[m <= 16, k] (Algorithm 1), then C = A W^T by the decode-shape
// GEMM above (the activation quantized on the fly and fed to the block-scaled
// GEMM, Sec. 3.2 / Fig. 7, App. B.1).
//
// Quantizing A in every workgroup would multiply its VALU work by the number
// of workgroups, so it is done once, by the first P <= 32 workgroups of the
// grid ("producers"; workgroups are dispatched in index order, so the
// producers are resident before any other workgroup of the launch).  Each
// producer reads all of A for max|A| (256 KB at most, from L2 after the
// first reader on an XCD) and forms s32 = max|A| / 2688 itself, so the
// producers never wait for each other: an exchange of partial maxima costs a
// chain of device-scope atomics, each a round trip of ~1.5 us across the
// XCDs, and measured 4.7 us against ~2.5 us for the redundant read.  A
// producer then quantizes its 1/P of the blocks with the quantizer's own
// per-block code (quantize_xs), writing A's codes and scales (producer 0
// also s32), and counts itself in sync[0] with release semantics at device
// scope.
// Every workgroup (producers included, after their part) then runs the GEMM
// body: it issues its first W loads, waits for sync[0] == P (acquire), and
// reads A's codes, scales and s32 from the outputs.  The last workgroup to
// finish (sync[1]) returns the counters to zero for the next call.  All
// waits are bounded (kSpinLimit polls with a sleep between them, far beyond
// any real wait); a workgroup that gives up writes NaN to its columns of C.
// Codes, scales and s32 are bit-identical to mixfp4_quantize in the compute
// mode, and C to mixfp4_gemm on them (same GEMM body, same order).
//
// Measured on 16 x 28672 x 8192 (one workgroup per CU): the producers have
// s32 after ~6 us and A quantized after ~8.5 us, and the consumers see the
// count at ~11.8 us; the GEMM bodies then take ~31 us.  A separate quantize
// launch before the GEMM costs less (~7 us, kernel boundaries being the
// cheapest grid-wide synchronization here), so the one-launch step serves
// callers that want a single dispatch, not speed.
constexpr int kStepProducers = 32;
constexpr uint32_t kSpinLimit = 1u << 22;
constexpr int kSyncDone = 0, kSyncExit = 1;

// Polls are relaxed device-scope loads (no cache maintenance per poll); one
// acquire fence follows the poll that sees the count, so the waiting
// workgroup's later loads see everything the counting workgroups released.
// (An acquire on every poll would invalidate the XCD's caches at each of
// them, under every other workgroup's loads.)
__device__ __forceinline__ bool wait_at_least(uint32_t* p, uint32_t target) {
  for (uint32_t i = 0; i < kSpinLimit; ++i) {
    if (__hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >= target) {
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
      return true;
    }
    __builtin_amdgcn_s_sleep(1);
  }
  return false;
}

// Producer blockIdx.x < producers: s32 from all of A, then the blocks
// [b0, b1) of its share of the m * k / 16 blocks of A (row-major, k per row).
__device__ __forceinline__ void produce_a(const uint16_t* __restrict__ x, int64_t m, int64_t k,
                                          uint8_t* __restrict__ a_codes,
                                          uint8_t* __restrict__ a_scales, float* __restrict__ a_ts,
                                          uint32_t* sync, int producers) {
  __shared__ ScaleRecip tab[128];
  __shared__ uint32_t wave_max[16];
  fill_scale_table(tab);
  const int tid = (int)threadIdx.x, nt = (int)blockDim.x;
  // max |A| over all of A: 16-byte words, eight loads in flight per thread
  const int64_t nvec = m * k / 8;
  const uint4* xv = reinterpret_cast<const uint4*>(x);
  uint32_t mx = 0u;
  int64_t i = tid;
  for (; i + 7 * nt < nvec; i += 8 * nt) {
    uint4 v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = xv[i + j * nt];
#pragma unroll
    for (int j = 0; j < 8; ++j) mx = max(mx, absmax8(v[j]));
  }
  for (; i < nvec; i += nt) mx = max(mx, absmax8(xv[i]));
  for (int off = 32; off > 0; off >>= 1) mx = max(mx, (uint32_t)__shfl_xor((int)mx, off));
  if ((tid & 63) == 0) wave_max[tid >> 6] = mx;
  __syncthreads();                                  // also publishes the scale table
  uint32_t r = wave_max[0];
  for (int w = 1; w < nt / 64; ++w) r = max(r, wave_max[w]);
  const float s32 = tensor_scale_of(r);
  if (blockIdx.x == 0 && tid == 0) *a_ts = s32;
  const int64_t nb = m * (k / kBlock);
  const int64_t per = (nb + producers - 1) / producers;
  const int64_t b0 = (int64_t)blockIdx.x * per;
  const int64_t b1 = b0 + per < nb ? b0 + per : nb;
  const bool direct = s32 >= 0x1p-90f && s32 <= 0x1p120f;
  const float xmul = direct ? 1.0f : (s32 < 1.0f ? 0x1p64f : 0x1p-64f);
  const float sx = s32 * xmul, rx = __fdiv_rn(1.0f, sx);
  for (int64_t g = b0 + tid; g < b1; g += nt) {
    const uint4* src = reinterpret_cast<const uint4*>(x + (g << 4));
    const uint4 v0 = src[0], v1 = src[1];
    float xs[16];
    if (direct)
      to_fp8_domain<false>(v0, v1, 1.0f, sx, rx, xs);
    else
      to_fp8_domain<true>(v0, v1, xmul, sx, rx, xs);
    uint2 out;
    uint32_t sb;
    quantize_xs<kSelect, false>(xs, tab, out, sb, make_uint4(0, 0, 0, 0));
    *reinterpret_cast<uint2*>(a_codes + (g << 3)) = out;
    a_scales[g] = (uint8_t)sb;
  }
  __syncthreads();                                  // every thread's stores are complete
  if (tid == 0)
    __hip_atomic_fetch_add(sync + kSyncDone, 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
}

template <int kW, int kA, int kB>
__global__ __launch_bounds__(64 * kW * (kB > 0 ? 2 : 1)) void decode_step_kernel(
    const uint16_t* __restrict__ x, uint8_t* __restrict__ a_codes, uint8_t* __restrict__ a_scales,
    float* __restrict__ a_ts, const uint8_t* __restrict__ w_codes,
    const uint8_t* __restrict__ w_scales, const float* __restrict__ w_ts, int64_t m, int64_t n,
    int64_t k, float* __restrict__ c, uint32_t* sync, int producers) {
  __shared__ int ok_sh;
  if ((int)blockIdx.x < producers) produce_a(x, m, k, a_codes, a_scales, a_ts, sync, producers);
  skinny_columns<kW, kA, kB>(a_codes, a_scales, a_ts, w_codes, w_scales, w_ts, m, n, k, c, [&]() {
    if (threadIdx.x == 0) ok_sh = wait_at_least(sync + kSyncDone, (uint32_t)producers);
    __syncthreads();
    return ok_sh != 0;
  });
  __syncthreads();
  if (threadIdx.x == 0) {
    // (relaxed: the count only needs atomicity; no data rides on it)
    const uint32_t done = __hip_atomic_fetch_add(sync + kSyncExit, 1u, __ATOMIC_RELAXED,
                                                 __HIP_MEMORY_SCOPE_AGENT);
    if (done + 1 == gridDim.x) {
      // every workgroup has passed its waits: ready the counters for the next call
#pragma unroll
      for (int i = 0; i < 4; ++i)
        __hip_atomic_store(sync + i, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

__global__ void fill_zero(float* c, int64_t count) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < count; i += stride) c[i] = 0.0f;
}

template <int BM, int BN, int WM, int WN>
hipError_t launch_tile(const uint8_t* a_codes, const uint8_t* a_scales, const float* a_ts,
                       const uint8_t* w_codes, const uint8_t* w_scales, const float* w_ts,
                       int64_t m, int64_t n, int64_t k, float* c, int64_t ldc,
                       hipStream_t stream) {
  const unsigned tiles = (unsigned)(((m + BM - 1) / BM) * ((n + BN - 1) / BN));
  constexpr int threads = 64 * WM * WN;
  const bool fast = k % 64 == 0 && ((reinterpret_cast<uintptr_t>(a_scales) |
                                     reinterpret_cast<uintptr_t>(w_scales)) & 3u) == 0;
  if (fast)
    gemm_kernel<BM, BN, WM, WN, true, false><<<tiles, threads, 0, stream>>>(
        a_codes, a_scales, a_ts, w_codes, w_scales, w_ts, m, n, k, c, ldc);
  else
    gemm_kernel<BM, BN, WM, WN, false, false><<<tiles, threads, 0, stream>>>(
        a_codes, a_scales, a_ts, w_codes, w_scales, w_ts, m, n, k, c, ldc);
  return hipGetLastError();
}

// Waves splitting K in the decode-shape kernel, by the S = floor(k / 256)
// whole steps: 2 when S is even but not a multiple of 4 (equal shares, as
// measured best), else 4 (equal shares when S % 4 == 0, otherwise shares
// differing by one step); a K tail goes to the last wave either way.
inline int skinny_waves(int64_t k) {
  const int64_t s = k / kSkinnyStep;
  return (s % 4 != 0 && s % 2 == 0) ? 2 : 4;
}

template <int kA, int kB>
hipError_t launch_skinny(const uint8_t* a_codes, const uint8_t* a_scales, const float* a_ts,
                         const uint8_t* w_codes, const uint8_t* w_scales, const float* w_ts,
                         int64_t m, int64_t n, int64_t k, float* c, hipStream_t stream) {
  const unsigned groups = (unsigned)((n + 16 * (kA + kB) - 1) / (16 * (kA + kB)));
  constexpr int sets = skinny_sets<kA, kB>();
  if (skinny_waves(k) == 4)
    gemm_skinny_kernel<4, kA, kB><<<groups, 256 * sets, 0, stream>>>(
        a_codes, a_scales, a_ts, w_codes, w_scales, w_ts, m, n, k, c);
  else
    gemm_skinny_kernel<2, kA, kB><<<groups, 128 * sets, 0, stream>>>(
        a_codes, a_scales, a_ts, w_codes, w_scales, w_ts, m, n, k, c);
  return hipGetLastError();
}

template <int kA, int kB>
hipError_t launch_step(const uint16_t* x, uint8_t* a_codes, uint8_t* a_scales, float* a_ts,
                       const uint8_t* w_codes, const uint8_t* w_scales, const float* w_ts,
                       int64_t m, int64_t n, int64_t k, float* c, uint32_t* sync,
                       hipStream_t stream) {
  const int64_t groups = (n + 16 * (kA + kB) - 1) / (16 * (kA + kB));
  const int producers = (int)(groups < kStepProducers ? groups : kStepProducers);
  constexpr int sets = skinny_sets<kA, kB>();
  if (skinny_waves(k) == 4)
    decode_step_kernel<4, kA, kB><<<(unsigned)groups, 256 * sets, 0, stream>>>(
        x, a_codes, a_scales, a_ts, w_codes, w_scales, w_ts, m, n, k, c, sync, producers);
  else
    decode_step_kernel<2, kA, kB><<<(unsigned)groups, 128 * sets, 0, stream>>>(
        x, a_codes, a_scales, a_ts, w_codes, w_scales, w_ts, m, n, k, c, sync, producers);
  return hipGetLastError();
}

// Column groups per workgroup of the decode-shape GEMM: the fewest 16-column
// groups G that cover W with at most one workgroup per CU, run as one range
// (G <= 6) or as 4 + (G - 4) on two sets of waves (G = 7, 8); beyond 8
// groups, 4 per workgroup and several workgroups per CU.  Narrow W then still
// spreads over every CU, and no CU gets two workgroups while others get one.
// Measured, m = 16: k = 4096, n = 4096: 5.3 us with G = 1 against 11.7 with
// 4; n = 8192 7.5 against 11.8; n = 11008 9.7 against 11.6; 16 x 28672 x 8192:
// 33.3 us with 4 + 3 groups on 256 workgroups against 35.4 with 4 groups on
// 448 (192 CUs with two of them).  Against 4 + (G - 4) run one after the
// other by the same 4 waves: one range of 5 (6) groups 23.0 (17.5) us
// against 26.2 (19.0) on 16 x 20480 x 8192 (16 x 24576 x 4096); concurrent
// sets 22.0 against 24.3 us on 16 x 32768 x 4096, 31.0 against 33.1 on
// 1 x 28672 x 8192, 19.5 against 20.9 on 8 x 28672 x 4096, 15.2 against 17.4
// on 16 x 28672 x 2816, 33.5 against 33.8 on 16 x 28672 x 8192.
template <typename Launch>
hipError_t by_column_split(int64_t n, Launch launch) {
  const int64_t cus = compute_units();
  const int64_t g = (n + 16 * cus - 1) / (16 * cus);
  switch (g) {
    case 1: return launch(std::integral_constant<int, 1>{}, std::integral_constant<int, 0>{});
    case 2: return launch(std::integral_constant<int, 2>{}, std::integral_constant<int, 0>{});
    case 3: return launch(std::integral_constant<int, 3>{}, std::integral_constant<int, 0>{});
    case 4: return launch(std::integral_constant<int, 4>{}, std::integral_constant<int, 0>{});
    case 5: return launch(std::integral_constant<int, 5>{}, std::integral_constant<int, 0>{});
    case 6: return launch(std::integral_constant<int, 6>{}, std::integral_constant<int, 0>{});
    case 7: return launch(std::integral_constant<int, 4>{}, std::integral_constant<int, 3>{});
    case 8: return launch(std::integral_constant<int, 4>{}, std::integral_constant<int, 4>{});
    default: return launch(std::integral_constant<int, 4>{}, std::integral_constant<int, 0>{});
  }
}

}  // namespace

bool decode_step_applies(int64_t m, int64_t k) {
  return m >= 1 && m <= kSkinnyRows && k > 0 && k % kSkinnyK == 0;
}

hipError_t launch_decode_step(const uint16_t* x, int64_t m, int64_t k, const uint8_t* w_codes,
                              const uint8_t* w_scales, const float* w_ts, int64_t n,
                              uint8_t* a_codes, uint8_t* a_scales, float* a_ts, float* c,
                              uint32_t* sync, hipStream_t stream) {
  // the column split of the decode-shape GEMM (launch_gemm)
  return by_column_split(n, [&](auto A, auto B) {
    return launch_step<decltype(A)::value, decltype(B)::value>(
        x, a_codes, a_scales, a_ts, w_codes, w_scales, w_ts, m, n, k, c, sync, stream);
  });
}

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
  // decode shape: the waves split K in 256-wide steps and a tail of 64, 128
  // or 192 (skinny_waves);
  // scale loads are 4-byte words
  const bool skinny_aligned = ((reinterpret_cast<uintptr_t>(w_scales) |
                                reinterpret_cast<uintptr_t>(a_scales)) & 3u) == 0;
  if (m <= kSkinnyRows && skinny_aligned && k % kSkinnyK == 0) {
    return by_column_split(n, [&](auto A, auto B) {
      return launch_skinny<decltype(A)::value, decltype(B)::value>(
          a_codes, a_scales, a_ts, w_codes, w_scales, w_ts, m, n, k, c, stream);
    });
  }
  // Tile choice (measured on MI355X): 256 x 256 with 8 waves is the most
  // efficient tile per compute unit (least LDS traffic and decode work per
  // MFMA), so it is used whenever it fills at least three quarters of a round
  // of the 256 compute units (2048 x 6144 x 4096: 127 us on 192 such tiles,
  // 177 us on 384 tiles of 128 x 256).  A short last round goes to 128 x 256
  // tiles in a second launch (2048 x 11008 x 4096: 207 us against 216 us).
  // Below that, 128 x 256 (same wave tiles, half the rows) if it fills most
  // of a round, else 128 x 128.
  const int64_t tm = (m + 255) / 256, tn = (n + 255) / 256;
  const int64_t tiles256 = tm * tn;
  const int64_t tiles128x256 = ((m + 127) / 128) * tn;
  const int64_t cus = compute_units();
  if (4 * tiles256 >= 3 * cus) {
    // A short last round of 256 x 256 tiles keeps only a few CUs busy for a
    // whole tile time.  Its columns go to a second launch of 128 x 256 tiles
    // (half the work per CU) when those fit in one round: every output still
    // sums its K range in the same order, so C is bit-identical.
    const int64_t nt1 = (tiles256 / cus) * cus / tm;    // 256-column tiles in whole rounds
    const int64_t rest = 2 * tm * (tn - nt1);           // 128 x 256 tiles left
    if (nt1 > 0 && nt1 < tn && rest <= cus) {
      const int64_t n1 = 256 * nt1;
      const hipError_t e = launch_tile<256, 256, 2, 4>(a_codes, a_scales, a_ts, w_codes, w_scales,
                                                       w_ts, m, n1, k, c, n, stream);
      if (e != hipSuccess) return e;
      return launch_tile<128, 256, 2, 4>(a_codes, a_scales, a_ts, w_codes + n1 * (k / 2),
                                         w_scales + n1 * (k / kBlock), w_ts, m, n - n1, k,
                                         c + n1, n, stream);
    }
    return launch_tile<256, 256, 2, 4>(a_codes, a_scales, a_ts, w_codes, w_scales, w_ts, m, n, k,
                                       c, n, stream);
  }
  if (4 * tiles128x256 >= 3 * cus)
    return launch_tile<128, 256, 2, 4>(a_codes, a_scales, a_ts, w_codes, w_scales, w_ts, m, n, k,
                                       c, n, stream);
  return launch_tile<128, 128, 2, 2>(a_codes, a_scales, a_ts, w_codes, w_scales, w_ts, m, n, k,
                                     c, n, stream);
}

}  // namespace mixfp4
