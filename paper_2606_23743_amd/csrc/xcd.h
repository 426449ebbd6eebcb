// Workgroup-to-XCD placement shared by the kernels.
#pragma once

#include <hip/hip_runtime.h>

namespace sva {

// Workgroup order: the hardware hands consecutive workgroup ids to the 8 XCDs
// round-robin.  Mapping id -> (id % 8) * ceil(n/8) + id / 8 gives each XCD a
// contiguous range of logical work items, so neighbouring query blocks of a
// head (which read overlapping key/value blocks) share one XCD's L2.
__device__ __forceinline__ int xcd_remap(int id, int n) {
  constexpr int kXcd = 8;
  const int per = (n + kXcd - 1) / kXcd;
  const int xcd = id % kXcd;
  const int slot = id / kXcd;
  // the first (n % 8) XCDs (or all, if n is a multiple of 8) own `per` items,
  // the rest own per-1; compute the start of this XCD's range accordingly
  const int full = (n % kXcd == 0) ? kXcd : (n % kXcd);
  const int start = (xcd < full) ? xcd * per : full * per + (xcd - full) * (per - 1);
  return start + slot;
}

}  // namespace sva
