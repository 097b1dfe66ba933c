// Workgroup-to-XCD mapping shared by the kernels.
#pragma once

#include <hip/hip_runtime.h>

namespace dconv {

// Blocks are dispatched round-robin over the 8 XCDs of an MI355X, each with
// its own L2.  Remapping the linear block id so that consecutive ids of one
// XCD get consecutive tiles keeps neighbouring tiles (which share halo rows
// and filter slices) in the same L2.
__device__ __forceinline__ int xcd_remap(int b, int n) {
  constexpr int kXcd = 8;
  const int per = n / kXcd;
  const int full = per * kXcd;
  if (b >= full) return b;
  return (b % kXcd) * per + b / kXcd;
}

}  // namespace dconv
