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

// Row order inside a head for sparse lists: frame tiles.  With F query blocks
// per frame (rounded), logical rows are cut into super-rows of FPT frames
// (F * FPT rows) and each super-row is walked tile by tile, a tile being BPT
// consecutive blocks of each of the FPT frames (the last tile of a super-row
// is the F % BPT blocks left over).  So a run of BPT * FPT consecutive logical
// rows is a (frames) x (blocks) patch of the video whose blocks keep mostly
// the same key blocks.  The last partial super-row is tiled with the whole
// frames it holds; rows past those keep their own index.  A bijection on
// [0, nB) for every F, FPT, BPT >= 1.
__host__ __device__ __forceinline__ int frame_tile_in(int r, int F, int fpt, int bpt) {
  const int tsz = fpt * bpt, fullc = F / bpt;
  if (r < fullc * tsz) {
    const int tc = r / tsz, u = r - tc * tsz, f = u / bpt, d = u - f * bpt;
    return f * F + tc * bpt + d;
  }
  const int rem = F - fullc * bpt, u = r - fullc * tsz, f = u / rem, d = u - f * rem;
  return f * F + fullc * bpt + d;
}

__host__ __device__ __forceinline__ int frame_tile_order(int l, int nB, int F, int fpt, int bpt) {
  const int span = F * fpt;
  const int whole = (nB / span) * span;
  if (l < whole) {
    const int sr = l / span;
    return sr * span + frame_tile_in(l - sr * span, F, fpt, bpt);
  }
  const int ft = (nB - whole) / F;   // whole frames in the tail
  if (ft > 0 && l < whole + ft * F) return whole + frame_tile_in(l - whole, F, ft, bpt);
  return l;
}

}  // namespace sva
