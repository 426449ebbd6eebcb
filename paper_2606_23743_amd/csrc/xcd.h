// Workgroup-to-XCD placement shared by the kernels.
#pragma once

#include <hip/hip_runtime.h>

namespace sva {

// Workgroup order: the hardware hands consecutive workgroup ids to the 8 XCDs
// round-robin.  Mapping id -> (id % 8) * ceil(n/8) + id / 8 gives each XCD a
// contiguous range of logical work items, so neighbouring query blocks of a
// head (which read overlapping key/value blocks) share one XCD's L2.
__host__ __device__ __forceinline__ int xcd_remap(int id, int n) {
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

// Segment order: rows are cut into segments of 8*c consecutive items, and XCD x
// takes the x-th run of c items of each segment in turn, so the eight XCDs work
// through the same segment (one head's query blocks, for c*8 <= nB) at the same
// time while each still holds c neighbouring rows.  Items past the last whole
// segment keep their own id.  A bijection on [0, n) for every c >= 1.
__host__ __device__ __forceinline__ int xcd_remap_segments(int id, int n, int c) {
  constexpr int kXcd = 8;
  const int seg = kXcd * c;
  const int whole = (n / seg) * seg;
  if (id >= whole) return id;
  const int slot = id / kXcd, xcd = id % kXcd;
  const int k = slot / c;
  return k * seg + xcd * c + (slot - k * c);
}

}  // namespace sva
