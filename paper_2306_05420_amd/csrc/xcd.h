// XCD-aware block numbering.
//
// An MI355X has 8 accelerator complex dies (XCDs), each with its own L2, and
// the dispatcher hands the blocks of a 1-D grid to them round-robin: block p
// runs on XCD p % 8, and each XCD takes its blocks in increasing p.  Kernels
// launch a grid padded to a multiple of 8 and work on
//   logical = (p % 8) * (grid / 8) + p / 8,
// so each XCD receives one contiguous range of logical blocks, in order.
// Tiles that read the same operand data are numbered next to each other and
// so share one L2 at about the same time.
#pragma once

#include <hip/hip_runtime.h>

namespace swsft {

constexpr int kNumXcd = 8;

inline unsigned xcd_grid(long long nblocks) {
  return (unsigned)((nblocks + kNumXcd - 1) / kNumXcd * kNumXcd);
}

__device__ __forceinline__ int xcd_logical_block() {
  const int p = blockIdx.x;
  return (p % kNumXcd) * (gridDim.x / kNumXcd) + p / kNumXcd;
}

// Order in which the 2L-1 orders m are numbered: q -> mi = q * L mod (2L-1)
// alternates between large and small |m| (L and 2L-1 are coprime), so a
// contiguous range of logical blocks mixes cheap and expensive orders.
__device__ __forceinline__ int mixed_order(int q, int L) { return (int)(((long long)q * L) % (2 * L - 1)); }

}  // namespace swsft
