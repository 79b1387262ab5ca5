// Pass 1 of the two-pass GEMM: each element of a MixFP4 operand decoded once
// into its exact 16-bit value s8 * v (Sec. 3.3, App. B.5; see decode.h), in
// the blocked layout of blocked_layout.h.  HBM-bound: 0.5625 B read and 2 B
// written per element.
#include "blocked_layout.h"
#include "decode.h"
#include "internal.h"
#include "quant_block.h"

namespace mixfp4 {
namespace {

// Pass 1: decode a MixFP4 operand [rows, k] into the blocked layout.
// A workgroup takes items of 32 rows x 8 steps.  Thread (row rl, step j)
// reads 16 code bytes and two scale bytes (eight lanes cover 128 contiguous
// code bytes of a row) and decodes them into the row's 64 output bytes in an
// LDS tile [step][32 rows x 64 B]; after a barrier the tile leaves as eight
// runs of 2 KB, one per step block (the item's rows are consecutive there),
// so every store instruction writes contiguous memory.  Each step plane of the
// tile is padded by 16 bytes, so the eight steps that a row's threads write
// fall on different LDS banks.  The next item's loads
// are issued before the current item's stores.  Rows beyond `rows` decode as
// zeros into padding rows of the last tile; nothing beyond the padded layout
// is written.
constexpr int kDecRows = 32, kDecSteps = 8;
constexpr int kPlane = kDecRows * 4 + 1;     // 16-byte chunks per step plane, padded

__global__ __launch_bounds__(256) void decode_blocked_kernel(const uint8_t* __restrict__ codes,
                                                             const uint8_t* __restrict__ scales,
                                                             int64_t rows, int64_t k,
                                                             uint8_t* __restrict__ out) {
  __shared__ uint4 tile[kDecSteps * kPlane];
  const int64_t steps = k / kStepK;
  const int64_t sgroups = (steps + kDecSteps - 1) / kDecSteps;
  const int64_t items = ((rows + kDecRows - 1) / kDecRows) * sgroups;
  const int tid = threadIdx.x;
  const int j = tid & 7, rl = tid >> 3;
  struct In { uint4 c; uint32_t s0, s1; bool ok; };
  auto load = [&](In& in, int64_t it) {
    const int64_t row = (it / sgroups) * kDecRows + rl;
    const int64_t s = (it % sgroups) * kDecSteps + j;
    in.ok = it < items && row < rows && s < steps;
    if (in.ok) {
      in.c = *reinterpret_cast<const uint4*>(codes + row * (k / 2) + s * 16);
      const uint8_t* sp = scales + row * (k / kBlock) + 2 * s;
      in.s0 = sp[0];
      in.s1 = sp[1];
    } else {
      in.c = make_uint4(0u, 0u, 0u, 0u);
      in.s0 = in.s1 = 0u;
    }
  };
  In cur;
  int64_t it = blockIdx.x;
  load(cur, it);
  for (; it < items; it += gridDim.x) {
    In nxt;
    load(nxt, it + gridDim.x);
    {
      const BlockDec d0 = block_dec(cur.s0), d1 = block_dec(cur.s1);
      const int r = (int)(((it / sgroups) * kDecRows + rl) % kTileRows);
      uint4* t = tile + j * kPlane + rl * 4;
      t[slot_of(r, 0)] = decode8(cur.c.x, d0);
      t[slot_of(r, 1)] = decode8(cur.c.y, d0);
      t[slot_of(r, 2)] = decode8(cur.c.z, d1);
      t[slot_of(r, 3)] = decode8(cur.c.w, d1);
    }
    __syncthreads();
    const int64_t row0 = (it / sgroups) * kDecRows;
    const int64_t s0 = (it % sgroups) * kDecSteps;
    uint8_t* ob = out + (row0 / kTileRows) * steps * kBlkBytes + (row0 % kTileRows) * 64;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int ch = tid + 256 * q;          // 16-byte chunk of the tile
      const int sj = ch >> 7;                // step within the item (128 chunks each)
      if (s0 + sj < steps)
        *reinterpret_cast<uint4*>(ob + (s0 + sj) * kBlkBytes + (ch & 127) * 16) =
            tile[sj * kPlane + (ch & 127)];
    }
    __syncthreads();
    cur = nxt;
  }
}

// Activation quantization fused with pass 1 (Sec. 3.2 / Fig. 7: the
// activation is quantized on the fly before the block-scaled GEMM): one pass
// over X [rows, k] writes its MixFP4 codes and scales (Algorithm 1, tensor
// scale given on the device) and the blocked fp16 decode of those codes, the
// operand of pass 2.  Same items as decode_blocked_kernel (32 rows x 8
// steps of 32 K); thread (row rl, step j) reads the step's 32 elements of
// its row (eight threads cover 512 contiguous bytes of a row), quantizes
// them as two blocks with the quantizer's per-block code (quantize_xs: the
// codes, scales and format bits are mixfp4_quantize's), stores the 16 code
// bytes and two scale bytes, and decodes its own codes into the LDS tile
// that leaves as eight 2 KB runs.  x = fl32(X / s32) takes Markstein's step
// (exact for every tensor scale, with X and s32 rescaled by 2^+-64 outside
// [2^-90, 2^120]).  Measured on A[16384, 8192]: about 120 us, against 76 us
// for the quantizer and 72 us for the decode pass run one after the other.
template <int kMode>
__global__ __launch_bounds__(256) void quantize_decode_kernel(
    const uint16_t* __restrict__ x, int64_t rows, int64_t k, int64_t ldx,
    uint8_t* __restrict__ codes, uint8_t* __restrict__ scales,
    const float* __restrict__ tensor_scale, uint8_t* __restrict__ out) {
  __shared__ uint4 tile[kDecSteps * kPlane];
  __shared__ ScaleRecip tab[128];
  fill_scale_table(tab);
  const float s32 = *tensor_scale;
  const bool direct = s32 >= 0x1p-90f && s32 <= 0x1p120f;
  const float xmul = direct ? 1.0f : (s32 < 1.0f ? 0x1p64f : 0x1p-64f);
  const float sx = s32 * xmul, rx = __fdiv_rn(1.0f, sx);
  const int64_t steps = k / kStepK;
  const int64_t sgroups = (steps + kDecSteps - 1) / kDecSteps;
  const int64_t items = ((rows + kDecRows - 1) / kDecRows) * sgroups;
  const int tid = threadIdx.x;
  const int j = tid & 7, rl = tid >> 3;
  struct In { uint4 v[4]; bool ok; };
  auto load = [&](In& in, int64_t it) {
    const int64_t row = (it / sgroups) * kDecRows + rl;
    const int64_t st = (it % sgroups) * kDecSteps + j;
    in.ok = it < items && row < rows && st < steps;
    if (in.ok) {
      const uint4* src = reinterpret_cast<const uint4*>(x + row * ldx + st * kStepK);
#pragma unroll
      for (int q = 0; q < 4; ++q) in.v[q] = src[q];
    } else {
#pragma unroll
      for (int q = 0; q < 4; ++q) in.v[q] = make_uint4(0u, 0u, 0u, 0u);
    }
  };
  __syncthreads();                                  // the scale table
  In cur;
  int64_t it = blockIdx.x;
  load(cur, it);
  for (; it < items; it += gridDim.x) {
    In nxt;
    load(nxt, it + gridDim.x);
    {
      uint2 c0 = make_uint2(0u, 0u), c1 = c0;
      uint32_t sb0 = 0u, sb1 = 0u;
      if (cur.ok) {
        float xs[16];
        if (direct) to_fp8_domain<false>(cur.v[0], cur.v[1], 1.0f, sx, rx, xs);
        else to_fp8_domain<true>(cur.v[0], cur.v[1], xmul, sx, rx, xs);
        quantize_xs<kMode, false>(xs, tab, c0, sb0, make_uint4(0, 0, 0, 0));
        if (direct) to_fp8_domain<false>(cur.v[2], cur.v[3], 1.0f, sx, rx, xs);
        else to_fp8_domain<true>(cur.v[2], cur.v[3], xmul, sx, rx, xs);
        quantize_xs<kMode, false>(xs, tab, c1, sb1, make_uint4(0, 0, 0, 0));
        const int64_t row = (it / sgroups) * kDecRows + rl;
        const int64_t st = (it % sgroups) * kDecSteps + j;
        *reinterpret_cast<uint4*>(codes + row * (k / 2) + st * 16) = make_uint4(c0.x, c0.y, c1.x, c1.y);
        uint8_t* sp = scales + row * (k / kBlock) + 2 * st;
        sp[0] = (uint8_t)sb0;
        sp[1] = (uint8_t)sb1;
      }
      const BlockDec d0 = block_dec(sb0), d1 = block_dec(sb1);
      const int r = (int)(((it / sgroups) * kDecRows + rl) % kTileRows);
      uint4* t = tile + j * kPlane + rl * 4;
      t[slot_of(r, 0)] = decode8(c0.x, d0);
      t[slot_of(r, 1)] = decode8(c0.y, d0);
      t[slot_of(r, 2)] = decode8(c1.x, d1);
      t[slot_of(r, 3)] = decode8(c1.y, d1);
    }
    __syncthreads();
    const int64_t row0 = (it / sgroups) * kDecRows;
    const int64_t s0 = (it % sgroups) * kDecSteps;
    uint8_t* ob = out + (row0 / kTileRows) * steps * kBlkBytes + (row0 % kTileRows) * 64;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int ch = tid + 256 * q;
      const int sj = ch >> 7;
      if (s0 + sj < steps)
        *reinterpret_cast<uint4*>(ob + (s0 + sj) * kBlkBytes + (ch & 127) * 16) =
            tile[sj * kPlane + (ch & 127)];
    }
    __syncthreads();
    cur = nxt;
  }
}

}  // namespace

hipError_t launch_quantize_decode(const uint16_t* x, int64_t rows, int64_t k, int64_t ldx,
                                  uint8_t* codes, uint8_t* scales, const float* tensor_scale,
                                  int mode, uint8_t* out, hipStream_t stream) {
  static ResidentCache cache{};
  const int64_t items = ((rows + kDecRows - 1) / kDecRows) * ((k / kStepK + kDecSteps - 1) / kDecSteps);
  int64_t grid = resident_groups(quantize_decode_kernel<kSelect>, cache, 8, 256);
  if (grid > items) grid = items;
  if (grid < 1) grid = 1;
  switch (mode) {
    case kSelect: quantize_decode_kernel<kSelect><<<(unsigned)grid, 256, 0, stream>>>(x, rows, k, ldx, codes, scales, tensor_scale, out); break;
    case kForceE2M1: quantize_decode_kernel<kForceE2M1><<<(unsigned)grid, 256, 0, stream>>>(x, rows, k, ldx, codes, scales, tensor_scale, out); break;
    case kForceE1M2: quantize_decode_kernel<kForceE1M2><<<(unsigned)grid, 256, 0, stream>>>(x, rows, k, ldx, codes, scales, tensor_scale, out); break;
    case kFourSix: quantize_decode_kernel<kFourSix><<<(unsigned)grid, 256, 0, stream>>>(x, rows, k, ldx, codes, scales, tensor_scale, out); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_decode_blocked(const uint8_t* codes, const uint8_t* scales, int64_t rows,
                                 int64_t k, uint8_t* out, hipStream_t stream) {
  static ResidentCache cache{};
  const int64_t items = ((rows + kDecRows - 1) / kDecRows) * ((k / kStepK + kDecSteps - 1) / kDecSteps);
  int64_t grid = resident_groups(decode_blocked_kernel, cache, 8, 256);
  if (grid > items) grid = items;
  if (grid < 1) grid = 1;
  decode_blocked_kernel<<<(unsigned)grid, 256, 0, stream>>>(codes, scales, rows, k, out);
  return hipGetLastError();
}

int64_t decoded_bytes(int64_t rows, int64_t k) { return padded_rows(rows) * k * 2; }

}  // namespace mixfp4
