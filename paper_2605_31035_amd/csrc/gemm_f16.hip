// Two-pass MixFP4 GEMM for compute-bound shapes: C = s32_A s32_W A W^T.
//
// Pass 1 (decode_operand.hip) decodes each operand once into the exact
// 16-bit values s8 * v (Sec. 3.3, App. B.5) in a blocked layout in the
// caller's workspace.  Pass 2 is a GEMM on those fp16 operands with fp32 accumulation
// (Sec. 3.3 keeps the accumulation unchanged) whose main loop issues nothing
// but matrix instructions, LDS reads and direct global -> LDS loads.
//
// Why two passes.  Measured on MI355X, the matrix core's throughput under a
// sustained fp16 MFMA load is power-limited (the clock settles near 1.6-1.8
// GHz), and every VALU instruction issued between MFMAs lowers it further: a
// decode fused into the MFMA loop costs ~6 VALU instructions per 32x32x16
// MFMA (each element decoded once per 256 x 256 tile), which held the fused
// kernel below ~0.47 of the fp16 peak.  Decoding once per element instead
// (16 B of fp16 written and read back per 4.5 bits stored) moves that work to
// an HBM-bound pass that takes ~4% of the GEMM's time at the large shapes.
//
// The operands arrive in the blocked layout of blocked_layout.h.
//
// GEMM kernel.  A workgroup of 4 waves (one per SIMD) owns a 256 x 256 tile
// of C; wave w computes rows 128 (w / 2) and columns 128 (w % 2) of it as
// 4 x 4 v_mfma_f32_32x32x16_f16 tiles (256 accumulator registers), with W as
// the first operand so that each lane ends up holding runs of four
// consecutive columns of one C row (16-byte stores in the epilogue).  The K loop
// steps 32; four LDS stages of 32 KB (A block then W block) hold the steps
// t .. t+3, filled by 16-byte buffer loads straight into LDS three steps
// ahead, so global latency hides under three steps of MFMAs.  Each step is
// two halves of 16 MFMAs (one 16-K slice each): the first half reads the
// second slice's fragments, a barrier then makes step t+1 visible, and the
// second half reads step t+1's first slice, so no LDS latency and no barrier
// sits in front of an MFMA that has nothing else to wait for.  The eight
// loads a wave issues per step are spread one per four MFMAs.
#include <mutex>

#include "blocked_layout.h"
#include "internal.h"
#include "tile_order.h"

typedef int mixfp4_i32x4 __attribute__((ext_vector_type(4)));
// The 16-byte buffer load that writes straight into LDS (the LLVM intrinsic;
// its LDS destination is M0 + offset + 16 * lane).
__device__ void raw_buffer_load_lds(mixfp4_i32x4 rsrc,
                                    __attribute__((address_space(3))) uint32_t* lds, int size,
                                    int voffset, int soffset, int offset,
                                    int aux) __asm("llvm.amdgcn.raw.buffer.load.lds");

namespace mixfp4 {
namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef mixfp4_i32x4 i32x4;

constexpr int kStages = 4;

// ---------------------------------------------------------------------------
// Pass 2: the fp16 GEMM on blocked operands.

// Buffer resource of a raw byte range (stride 0, 32-bit data format word of
// the gfx9 descriptor); loads past `bytes` return zeros.
__device__ __forceinline__ i32x4 make_rsrc(const void* base, uint32_t bytes) {
  const uint64_t b = reinterpret_cast<uint64_t>(base);
  i32x4 r;
  r[0] = (int)(uint32_t)b;
  r[1] = (int)(uint32_t)(b >> 32);
  r[2] = (int)bytes;
  r[3] = 0x00020000;
  return r;
}

__global__ __launch_bounds__(256, 1) void gemm_f16_kernel(const uint8_t* __restrict__ ablk,
                                                         const uint8_t* __restrict__ wblk,
                                                         const float* __restrict__ a_ts,
                                                         const float* __restrict__ w_ts,
                                                         int64_t m, int64_t n, int64_t k,
                                                         float* __restrict__ c, int64_t ldc) {
  typedef _Float16 f16x8v __attribute__((ext_vector_type(8)));
  __shared__ __attribute__((aligned(1024))) uint8_t lds[kStages * kStageBytes];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int64_t steps = k / kStepK;
  const int64_t ntm = (m + kTileRows - 1) / kTileRows, ntn = (n + kTileRows - 1) / kTileRows;
  const int64_t tile = grouped_tile(xcd_item(blockIdx.x, gridDim.x), ntm, ntn);
  const int64_t tm = tile / ntn, tn = tile % ntn;

  // Waves 0-1 copy halves (8 KB) of the A block of each step, waves 2-3 of
  // the W block: 8 loads of 1 KB per wave and step.
  const bool is_a = wave < 2;
  const uint8_t* src = (is_a ? ablk + tm * steps * kBlkBytes : wblk + tn * steps * kBlkBytes) +
                       (wave & 1) * (kBlkBytes / 2);
  const i32x4 rsrc = make_rsrc(src, (uint32_t)(steps * kBlkBytes));
  const int ldst = (is_a ? 0 : kBlkBytes) + (wave & 1) * (kBlkBytes / 2);
  // Part p (0-7) of this wave's share of step st: 1 KB into `stage`.
  auto issue = [&](int stage, int64_t st, int p) {
    const int hoff = (p >> 2) * 4096;
    auto* l = (__attribute__((address_space(3))) uint32_t*)(uintptr_t)(
        reinterpret_cast<uintptr_t>(lds) + stage * kStageBytes + ldst + hoff);
    raw_buffer_load_lds(rsrc, l, 16, lane * 16, (int)(st * kBlkBytes) + hoff, (p & 3) * 1024, 0);
  };

  const int wm = (wave >> 1) * 128, wn = (wave & 1) * 128;
  const int half = lane >> 5, lrow = lane & 31;
  f32x16 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int q = 0; q < 16; ++q) acc[i][j][q] = 0.0f;

  // Fragments of one 16-K slice: 4 A and 4 W 32-row tiles.  Lane (lrow,
  // half) takes the 8-element group 2 sl + half of its row.  read_pair
  // fetches the A and W fragments of 32-row tile c.
  typedef f16x8v Frag[4];
  auto read_pair = [&](Frag& fa, Frag& fw, int stage, int sl, int c) {
    const uint8_t* b = lds + stage * kStageBytes;
    const int g = 2 * sl + half;
    const int ra = wm + 32 * c + lrow, rw = wn + 32 * c + lrow;
    fa[c] = *reinterpret_cast<const f16x8v*>(b + ra * 64 + slot_of(ra, g) * 16);
    fw[c] = *reinterpret_cast<const f16x8v*>(b + kBlkBytes + rw * 64 + slot_of(rw, g) * 16);
  };
  // The four MFMAs of A tile i.  W fragments are the first operand, so the
  // accumulator tile is C^T: a lane holds row m of C and each register quad
  // four consecutive columns.
  auto mfma_row = [&](const Frag& fa, const Frag& fw, int i) {
#pragma unroll
    for (int j = 0; j < 4; ++j)
      acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(fw[j], fa[i], acc[i][j], 0, 0, 0);
  };

  const int64_t last = steps - 1;
#pragma unroll
  for (int s0 = 0; s0 < kStages - 1; ++s0)
#pragma unroll
    for (int p = 0; p < 8; ++p) issue(s0, s0 < last ? s0 : last, p);
  // step 0 landed (the two later steps' 16 loads may be in flight)
  asm volatile("s_waitcnt vmcnt(16)" ::: "memory");
  __builtin_amdgcn_s_barrier();
  Frag pa, pw, qa, qw;
#pragma unroll
  for (int c = 0; c < 4; ++c) read_pair(pa, pw, 0, 0, c);
  // Invariant at the top of step t: P holds slice 0 of step t; the loads of
  // steps t+1 and t+2 are in flight or landed.  Each half of a step runs in
  // four chunks of one A tile's four MFMAs, each followed by one of the
  // wave's eight 1 KB loads of step t+3 (into the stage of step t-1, which
  // every wave finished reading before the barrier of step t-1).  Issued
  // together, the loads fill the texture unit's address queue (the reads
  // wait ~350 cycles on L2 and beyond), and a wave that cannot issue its
  // next load cannot issue its next MFMA either; spread like this they
  // measured 7% faster on 16384 x 8192 x 8192.  Loads and reads past the
  // last step are clamped to it (they refill a stage never read again).
  for (int64_t t = 0; t < steps; ++t) {
    const int cur = (int)(t % kStages), ls = (int)((t + kStages - 1) % kStages);
    const int64_t tl = t + kStages - 1 < last ? t + kStages - 1 : last;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      read_pair(qa, qw, cur, 1, c);
      mfma_row(pa, pw, c);
      __builtin_amdgcn_sched_barrier(0);
      issue(ls, tl, c);
      __builtin_amdgcn_sched_barrier(0);
    }
    // step t+1 landed: after its loads this wave issued the 8 of step t+2
    // and 4 of step t+3.  The reads of slice 1 are complete too.
    asm volatile("s_waitcnt vmcnt(12) lgkmcnt(0)" ::: "memory");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      read_pair(pa, pw, (int)((t + 1) % kStages), 0, c);
      mfma_row(qa, qw, c);
      __builtin_amdgcn_sched_barrier(0);
      issue(ls, tl, 4 + c);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");

  const float scale = (a_ts ? *a_ts : 1.0f) * (w_ts ? *w_ts : 1.0f);
  const int64_t m0 = tm * kTileRows + wm, n0 = tn * kTileRows + wn;
  // 32 x 32 accumulator layout of C^T: lane holds row m0 + 32 i + lane%32;
  // register q holds column 32 j + 8*(q/4) + 4*(lane/32) + q%4.  Four
  // consecutive registers are four consecutive columns: one 16-byte store
  // when C's rows keep 16-byte alignment (n % 4 == 0, C 16-byte aligned).
  const bool vec = (ldc % 4) == 0 && (reinterpret_cast<uintptr_t>(c) & 15u) == 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int64_t row = m0 + i * 32 + lrow;
    if (row >= m) continue;
    float* crow = c + row * ldc;
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int qq = 0; qq < 4; ++qq) {
        const int64_t col = n0 + j * 32 + 8 * qq + 4 * half;
        const f32x16& v = acc[i][j];
        if (vec) {
          if (col < n)
            *reinterpret_cast<float4*>(crow + col) =
                make_float4(v[4 * qq] * scale, v[4 * qq + 1] * scale, v[4 * qq + 2] * scale,
                            v[4 * qq + 3] * scale);
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (col + e < n) crow[col + e] = v[4 * qq + e] * scale;
        }
      }
  }
}


// The same GEMM on 128 x 256 tiles, for the columns of a short last round
// of 256 x 256 tiles and for products of at most half a round
// (launch_gemm_decoded): a tile does half the work, so such columns fill one
// round of 128 x 256 tiles in half a tile time.  Wave w computes rows 64 (w / 2) and columns 128 (w % 2)
// of the tile as 2 x 4 MFMA tiles; an A tile is one half (8 KB, contiguous)
// of each 256-row step block.  Each step's 24 KB are 24 loads of 1 KB, six
// per wave, spread one per four MFMAs; the pipeline, stages and barriers are
// those of gemm_f16_kernel, and every output sums its K steps in the same
// order, so C is bit-identical to the 256 x 256 tiles'.
constexpr int kHalfRows = 128;
constexpr int kHalfStageBytes = kBlkBytes / 2 + kBlkBytes;       // A half block, W block

__global__ __launch_bounds__(256, 1) void gemm_f16_half_kernel(
    const uint8_t* __restrict__ ablk, const uint8_t* __restrict__ wblk,
    const float* __restrict__ a_ts, const float* __restrict__ w_ts, int64_t m, int64_t n,
    int64_t k, float* __restrict__ c, int64_t ldc) {
  typedef _Float16 f16x8v __attribute__((ext_vector_type(8)));
  __shared__ __attribute__((aligned(1024))) uint8_t lds[kStages * kHalfStageBytes];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int64_t steps = k / kStepK;
  // both halves of every 256-row block of A (the blocked layout pads the
  // rows to 256; a half past m reads padding and stores nothing)
  const int64_t ntm = 2 * ((m + kTileRows - 1) / kTileRows), ntn = (n + kTileRows - 1) / kTileRows;
  const int64_t tile = grouped_tile(xcd_item(blockIdx.x, gridDim.x), ntm, ntn);
  const int64_t tm = tile / ntn, tn = tile % ntn;

  // part q (0-23) of a step: q < 8 is KB q of the A tile's half block, else
  // KB q - 8 of the W block; wave w issues parts 6 w .. 6 w + 5
  const i32x4 rsrc_a = make_rsrc(ablk + (tm >> 1) * steps * kBlkBytes, (uint32_t)(steps * kBlkBytes));
  const i32x4 rsrc_w = make_rsrc(wblk + tn * steps * kBlkBytes, (uint32_t)(steps * kBlkBytes));
  const int a_half = (int)(tm & 1) * (kBlkBytes / 2);
  auto issue = [&](int stage, int64_t st, int j) {
    const int q = 6 * wave + j;
    const bool is_a = q < 8;
    const int lofs = is_a ? q * 1024 : kBlkBytes / 2 + (q - 8) * 1024;
    const int gofs = (int)(st * kBlkBytes) + (is_a ? a_half + q * 1024 : (q - 8) * 1024);
    auto* l = (__attribute__((address_space(3))) uint32_t*)(uintptr_t)(
        reinterpret_cast<uintptr_t>(lds) + stage * kHalfStageBytes + lofs);
    raw_buffer_load_lds(is_a ? rsrc_a : rsrc_w, l, 16, lane * 16, gofs, 0, 0);
  };

  const int wm = (wave >> 1) * 64, wn = (wave & 1) * 128;
  const int half = lane >> 5, lrow = lane & 31;
  f32x16 acc[2][4];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int q = 0; q < 16; ++q) acc[i][j][q] = 0.0f;

  // Fragments of one 16-K slice: 2 A and 4 W 32-row tiles.  The A half
  // block's rows keep their swizzle (128 is a multiple of 16).
  struct Frags {
    f16x8v a[2], w[4];
  };
  auto read_a = [&](Frags& f, int stage, int sl, int cc) {
    const uint8_t* b = lds + stage * kHalfStageBytes;
    const int g = 2 * sl + half, ra = wm + 32 * cc + lrow;
    f.a[cc] = *reinterpret_cast<const f16x8v*>(b + ra * 64 + slot_of(ra, g) * 16);
  };
  auto read_w = [&](Frags& f, int stage, int sl, int cc) {
    const uint8_t* b = lds + stage * kHalfStageBytes + kBlkBytes / 2;
    const int g = 2 * sl + half, rw = wn + 32 * cc + lrow;
    f.w[cc] = *reinterpret_cast<const f16x8v*>(b + rw * 64 + slot_of(rw, g) * 16);
  };
  auto mfma_row = [&](const Frags& f, int i) {
#pragma unroll
    for (int j = 0; j < 4; ++j)
      acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(f.w[j], f.a[i], acc[i][j], 0, 0, 0);
  };
  // One half step: read the next slice's fragments while the current
  // slice's 8 MFMAs run, with three of the wave's six loads of step t + 3.
  auto half_step = [&](Frags& cur, Frags& nxt, int stage, int sl, int ls, int64_t tl, int j0) {
    read_a(nxt, stage, sl, 0);
    read_w(nxt, stage, sl, 0);
    read_w(nxt, stage, sl, 1);
    mfma_row(cur, 0);
    __builtin_amdgcn_sched_barrier(0);
    issue(ls, tl, j0);
    __builtin_amdgcn_sched_barrier(0);
    read_a(nxt, stage, sl, 1);
    read_w(nxt, stage, sl, 2);
    read_w(nxt, stage, sl, 3);
    mfma_row(cur, 1);
    __builtin_amdgcn_sched_barrier(0);
    issue(ls, tl, j0 + 1);
    issue(ls, tl, j0 + 2);
    __builtin_amdgcn_sched_barrier(0);
  };

  const int64_t last = steps - 1;
#pragma unroll
  for (int s0 = 0; s0 < kStages - 1; ++s0)
#pragma unroll
    for (int j = 0; j < 6; ++j) issue(s0, s0 < last ? s0 : last, j);
  // step 0 landed (the two later steps' 12 loads may be in flight)
  asm volatile("s_waitcnt vmcnt(12)" ::: "memory");
  __builtin_amdgcn_s_barrier();
  Frags p, q;
  read_a(p, 0, 0, 0);
  read_a(p, 0, 0, 1);
#pragma unroll
  for (int cc = 0; cc < 4; ++cc) read_w(p, 0, 0, cc);
  // Invariant at the top of step t as in gemm_f16_kernel: P holds slice 0 of
  // step t; the loads of steps t+1 and t+2 are in flight or landed.
  for (int64_t t = 0; t < steps; ++t) {
    const int cur = (int)(t % kStages), ls = (int)((t + kStages - 1) % kStages);
    const int64_t tl = t + kStages - 1 < last ? t + kStages - 1 : last;
    half_step(p, q, cur, 1, ls, tl, 0);
    // step t+1 landed: after its loads this wave issued the 6 of step t+2
    // and 3 of step t+3.  The reads of slice 1 are complete too.
    asm volatile("s_waitcnt vmcnt(9) lgkmcnt(0)" ::: "memory");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    half_step(q, p, (int)((t + 1) % kStages), 0, ls, tl, 3);
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");

  const float scale = (a_ts ? *a_ts : 1.0f) * (w_ts ? *w_ts : 1.0f);
  const int64_t m0 = tm * kHalfRows + wm, n0 = tn * kTileRows + wn;
  const bool vec = (ldc % 4) == 0 && (reinterpret_cast<uintptr_t>(c) & 15u) == 0;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int64_t row = m0 + i * 32 + lrow;
    if (row >= m) continue;
    float* crow = c + row * ldc;
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int qq = 0; qq < 4; ++qq) {
        const int64_t col = n0 + j * 32 + 8 * qq + 4 * half;
        const f32x16& v = acc[i][j];
        if (vec) {
          if (col < n)
            *reinterpret_cast<float4*>(crow + col) =
                make_float4(v[4 * qq] * scale, v[4 * qq + 1] * scale, v[4 * qq + 2] * scale,
                            v[4 * qq + 3] * scale);
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (col + e < n) crow[col + e] = v[4 * qq + e] * scale;
        }
      }
  }
}

}  // namespace

bool gemm_two_pass_applies(int64_t m, int64_t n, int64_t k) {
  // k <= 2^22 keeps a tile-row's blocks (k/32 x 16 KB) inside a 32-bit buffer range
  return m > 16 && n > 0 && k > 0 && k % kStepK == 0 && k <= (int64_t(1) << 22);
}

int64_t gemm_two_pass_workspace(int64_t m, int64_t n, int64_t k) {
  if (!gemm_two_pass_applies(m, n, k)) return 0;
  return (padded_rows(m) + padded_rows(n)) * k * 2;
}

hipError_t launch_gemm_decoded(const uint8_t* ablk, const float* a_ts, const uint8_t* wblk,
                               const float* w_ts, int64_t m, int64_t n, int64_t k, float* c,
                               hipStream_t stream) {
  const int64_t tm = padded_rows(m) / kTileRows, tn = padded_rows(n) / kTileRows;
  const int64_t tiles = tm * tn;
  // A short last round of 256 x 256 tiles keeps a few CUs busy for a whole
  // tile time: its columns go to 128 x 256 tiles (half the work each) when
  // those fit in one round, and so does the whole product when it is half a
  // round or less.  Each output sums its K steps in the same order either
  // way, so C is bit-identical.
  const int64_t cus = compute_units();
  if (2 * tiles <= cus) {
    // at most half a round of 256 x 256 tiles: 128 x 256 tiles fill (at most)
    // one round in half the time
    gemm_f16_half_kernel<<<(unsigned)(2 * tiles), 256, 0, stream>>>(ablk, wblk, a_ts, w_ts, m, n,
                                                                     k, c, n);
    return hipGetLastError();
  }
  const int64_t nt1 = tiles > cus ? (tiles / cus) * cus / tm : 0;   // tile columns in whole rounds
  const int64_t rest = 2 * tm * (tn - nt1);                          // 128 x 256 tiles left
  if (nt1 > 0 && nt1 < tn && rest <= cus) {
    const int64_t n1 = kTileRows * nt1;
    gemm_f16_kernel<<<(unsigned)(tm * nt1), 256, 0, stream>>>(ablk, wblk, a_ts, w_ts, m, n1, k,
                                                               c, n);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    gemm_f16_half_kernel<<<(unsigned)rest, 256, 0, stream>>>(
        ablk, wblk + nt1 * (k / kStepK) * kBlkBytes, a_ts, w_ts, m, n - n1, k, c + n1, n);
    return hipGetLastError();
  }
  gemm_f16_kernel<<<(unsigned)tiles, 256, 0, stream>>>(ablk, wblk, a_ts, w_ts, m, n, k, c, n);
  return hipGetLastError();
}

hipError_t launch_gemm_two_pass(const uint8_t* a_codes, const uint8_t* a_scales, const float* a_ts,
                                const uint8_t* w_codes, const uint8_t* w_scales, const float* w_ts,
                                int64_t m, int64_t n, int64_t k, float* c, uint8_t* workspace,
                                hipStream_t stream) {
  uint8_t* ablk = workspace;
  uint8_t* wblk = workspace + decoded_bytes(m, k);
  hipError_t e = launch_decode_blocked(a_codes, a_scales, m, k, ablk, stream);
  if (e != hipSuccess) return e;
  e = launch_decode_blocked(w_codes, w_scales, n, k, wblk, stream);
  if (e != hipSuccess) return e;
  return launch_gemm_decoded(ablk, a_ts, wblk, w_ts, m, n, k, c, stream);
}

// ---------------------------------------------------------------------------
// Workspace for callers that cannot allocate: a file-scope device array that
// each GPU the library runs on holds until the process ends.  Host code never
// passes `scratch` itself (on the host the name is only a stand-in for the
// symbol): it takes the array's device address once per device with
// hipGetSymbolAddress and passes that pointer to the kernels.
namespace {
static __device__ __align__(256) uint8_t scratch[kStaticScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void* g_scratch_ptr[kMaxDevices] = {};
}  // namespace

hipError_t static_scratch(void** ptr) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace mixfp4
