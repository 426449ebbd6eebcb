// Device helpers shared by the attention kernels (types, the LDS tile
// geometry and swizzles, lane exchanges, explicit waits).
#pragma once

#include "sva_internal.h"

namespace sva {
namespace attn {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) __bf16 bf16x4;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;
typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(2))) float f32x2;
typedef __attribute__((ext_vector_type(4))) short i16x4;
typedef __attribute__((ext_vector_type(2))) unsigned u32x2;
typedef __attribute__((ext_vector_type(4))) unsigned u32x4;
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
typedef __attribute__((address_space(4))) const int32_t const_i32;


template <int D>
struct Geo {
  static constexpr int RB = (D > 64) ? 256 : 128;   // LDS row pitch, bytes
  static constexpr int NCH = RB / 16;               // 16-byte chunks per LDS row
  static constexpr int DCH = D / 8;                 // chunks that hold data
  static constexpr int RPI = 1024 / RB;             // rows per 1 KB direct load
  static constexpr int DQ = D / 16;                 // k-steps of QK^T
  static constexpr int DP = (D + 31) / 32 * 32;     // head dim padded to PV tiles
  static constexpr int DT = DP / 32;                // 32-row d tiles of O^T
};

// LDS position of 16-byte piece c of tile row r.  LDS serves 256 bytes per
// clock from 64 four-byte banks: a b128 read in groups of 16 consecutive lanes,
// a b64 (transpose) read in groups of 32.  K operand reads put 16 consecutive
// rows at one piece in a group, so the K swizzle spreads any 16 consecutive
// rows over all 64 banks; V transpose reads put 4 consecutive rows x 4 pieces
// in a group, so the V swizzle moves those 4 rows to disjoint 4-piece groups.
// Both are XORs (involutions): the same function maps position to piece.
template <int NCH>
__device__ __forceinline__ int swz_k(int r, int c) {
  return NCH == 16 ? c ^ (r & 15) : c ^ ((r >> 1) & 7);
}
template <int NCH>
__device__ __forceinline__ int swz_v(int r, int c) {
  return NCH == 16 ? c ^ (4 * (r & 3)) : c ^ (4 * ((r >> 1) & 1));
}

// V tiles of the 16x16 kernels (attn_w16.h): a 32-lane transpose-read group
// takes pieces 2dt and 2dt+1 of 8 consecutive rows.  Piece c of row r at
// c ^ 2(r & 7) (256-byte rows) or c ^ 2((r >> 1) & 3) (128-byte rows, two per
// 256-byte bank window) puts those 16 reads on disjoint banks.
template <int NCH>
__device__ __forceinline__ int swz_v16(int r, int c) {
  return NCH == 16 ? c ^ (2 * (r & 7)) : c ^ (2 * ((r >> 1) & 3));
}

__device__ __forceinline__ bf16x2 cvt2(float a, float b) {
  f32x2 f = {a, b};
  return __builtin_convertvector(f, bf16x2);
}

__device__ __forceinline__ float swap_halves_max(float x) {
  const u32x2 r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

__device__ __forceinline__ float swap_halves_sum(float x) {
  const u32x2 r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// s_waitcnt vmcnt(n) leaving the other counters alone (gfx9 encoding).
template <int n>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(n >= 0 && n < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((n & 15) | (7 << 4) | (15 << 8) | ((n >> 4) << 14));
  asm volatile("" ::: "memory");
}

// s_waitcnt vmcnt(n) lgkmcnt(0): also every LDS read of this wave has returned
// (and any scalar load), so a stage it was reading may be refilled once every
// wave has passed the following barrier.
template <int n>
__device__ __forceinline__ void wait_vmcnt_lds_idle() {
  static_assert(n >= 0 && n < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((n & 15) | (7 << 4) | (0 << 8) | ((n >> 4) << 14));
  asm volatile("" ::: "memory");
}

// Workgroup barrier without the release/acquire fences of __syncthreads (which
// would wait for every in-flight direct load); LDS visibility is handled by the
// explicit vmcnt waits and by MFMAs having consumed their LDS operands.
__device__ __forceinline__ void wg_barrier() {
  asm volatile("s_barrier" ::: "memory");
}

}  // namespace attn
}  // namespace sva
