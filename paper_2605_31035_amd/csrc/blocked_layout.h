// The blocked layout of a decoded operand (exact 16-bit values s8 * v),
// written by the decode pass and read by the decoded-operand GEMM.
//
// Blocked operand layout (rows padded to a multiple of 256, K % 32 == 0):
// block (t, s) = rows [256 t, 256 t + 256) x K [32 s, 32 s + 32) is 16 KB at
// byte offset (t * K/32 + s) * 16384.  Row r of a block takes 64 bytes at
// 64 r; its 8-element group g (K 32 s + 8 g ..) is stored at 16-byte slot
// g ^ ((r >> 2) & 3), in the order [e0 e2 e4 e6 e1 e3 e5 e7] that decode8
// produces (A and W share the order; a dot product does not depend on it).
// A whole block is then one contiguous copy into LDS, and the swizzle keeps
// the 16 lanes of each LDS read pass on distinct banks.
//
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mixfp4 {

constexpr int kTileRows = 256;                // rows of A or W per tile
constexpr int kStepK = 32;                    // K per step (two 16-K MFMA slices)
constexpr int kBlkBytes = kTileRows * kStepK * 2;   // 16 KB per (tile, step) block
constexpr int kStageBytes = 2 * kBlkBytes;    // A block then W block

__host__ __device__ __forceinline__ int slot_of(int r, int g) { return g ^ ((r >> 2) & 3); }

inline int64_t padded_rows(int64_t rows) { return (rows + kTileRows - 1) / kTileRows * kTileRows; }

}  // namespace mixfp4
