// Small device helpers shared by the kernel files.
#pragma once

#include <hip/hip_runtime.h>

namespace fdc {

// Blocks are dispatched round-robin over the 8 XCDs; renumber them so that
// neighbouring tiles (which share cache lines) run on the same XCD and its L2.
__device__ __forceinline__ int xcd_remap(int bid, int nblocks) {
  const int q = nblocks >> 3, rem = nblocks & 7;
  const int x = bid & 7, i = bid >> 3;
  return x * q + (x < rem ? x : rem) + i;
}

}  // namespace fdc
