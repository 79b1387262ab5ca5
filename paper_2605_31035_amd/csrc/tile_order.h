// Work-item order of the tiled GEMM kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mixfp4 {

// Work-item order.  The hardware deals workgroups round-robin over the 8 XCDs,
// each with its own L2.  xcd_item() turns the launch index into an item index
// such that every XCD receives one contiguous range of items (a bijection for
// any count), and grouped_tile() walks tiles in groups of four tile-rows,
// column by column, so the workgroups resident on one XCD share A and W
// tiles in that XCD's L2.
__device__ __forceinline__ int64_t xcd_item(int64_t b, int64_t count) {
  const int64_t q = count / 8, r = count % 8, x = b % 8, j = b / 8;
  return x * q + (x < r ? x : r) + j;
}
__device__ __forceinline__ int64_t grouped_tile(int64_t i, int64_t ntm, int64_t ntn) {
  constexpr int64_t kGroup = 4;
  const int64_t per_group = kGroup * ntn;
  const int64_t first = (i / per_group) * kGroup;
  const int64_t rows = ntm - first < kGroup ? ntm - first : kGroup;
  const int64_t local = i % per_group;
  return (first + local % rows) * ntn + local / rows;
}

}  // namespace mixfp4
