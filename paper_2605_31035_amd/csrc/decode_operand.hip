// Pass 1 of the two-pass GEMM: each element of a MixFP4 operand decoded once
// into its exact 16-bit value s8 * v (Sec. 3.3, App. B.5; see decode.h), in
// the blocked layout of blocked_layout.h.  HBM-bound: 0.5625 B read and 2 B
// written per element.
#include "blocked_layout.h"
#include "decode.h"
#include "internal.h"

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

}  // namespace

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
