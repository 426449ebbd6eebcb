// Building blocks of the bf16 attention kernels: the direct global -> LDS
// chunk loads every kernel uses, the NaN mark of a block left to the
// recompute pass, and the operand reads of the 32x32x16 form (per-lane LDS
// offsets of the K operand and of the V transpose reads) that the
// remainder's moment, weight and GEMM kernels (remainder.hip) use.  The
// attention kernels' own arithmetic is the 16x16 form (attn_w16.h).
#pragma once

#include "attn_common.h"

namespace sva {
namespace attn {

typedef __attribute__((address_space(3))) unsigned char lds_u8;

// Direct global -> LDS loads of one 32-key chunk (K or V tile of CT bytes):
// the NUW 1 KB pieces this wave fills.  Piece u covers tile rows u*RPI ..;
// lane L fills row u*RPI + L/NCH at position L % NCH with the global piece the
// swizzle maps there, so a wave's per-lane byte offsets are fixed and the
// chunk's key offset is the scalar offset.  Every address lies inside the
// head's rows: full chunks by construction, the sequence's last partial chunk
// by clamping rows past the end to its first row, and a chunk wholly past the
// end by reading chunk 0 instead.  V16 selects the V tile swizzle of the 16x16
// kernels (swz_v16) in place of the one of the transpose reads below.
template <int D, int NUW, int CT, bool V16 = false>
struct ChunkLoader {
  __amdgpu_buffer_rsrc_t krs, vrs;
  int kgv[NUW], vgv[NUW];
  unsigned ks_base, vs_base;
  int w, lane, N;
};

template <int D, int NUW, int CT, bool V16>
__device__ __forceinline__ void loader_init(ChunkLoader<D, NUW, CT, V16>& f, const uint16_t* Kh, const uint16_t* Vh,
                                            int N, const unsigned char* ks, const unsigned char* vs, int w,
                                            int lane) {
  using G = Geo<D>;
  f.krs = __builtin_amdgcn_make_buffer_rsrc((void*)Kh, (short)0, N * D * 2, 0x00020000);
  f.vrs = __builtin_amdgcn_make_buffer_rsrc((void*)Vh, (short)0, N * D * 2, 0x00020000);
#pragma unroll
  for (int v = 0; v < NUW; ++v) {
    const int r = (w * NUW + v) * G::RPI + lane / G::NCH;
    const int p = lane % G::NCH;
    int ck = swz_k<G::NCH>(r, p), cv = V16 ? swz_v16<G::NCH>(r, p) : swz_v<G::NCH>(r, p);
    if (ck >= G::DCH) ck = 0;                        // padding pieces: any in-row address
    if (cv >= G::DCH) cv = 0;
    f.kgv[v] = (r * D + ck * 8) * 2;
    f.vgv[v] = (r * D + cv * 8) * 2;
  }
  f.ks_base = __builtin_amdgcn_readfirstlane((unsigned)(size_t)(const lds_u8*)ks);
  f.vs_base = __builtin_amdgcn_readfirstlane((unsigned)(size_t)(const lds_u8*)vs);
  f.w = w;
  f.lane = lane;
  f.N = N;
}

__device__ __forceinline__ void buffer_to_lds(const __amdgpu_buffer_rsrc_t& rs, unsigned lds_addr, int voff, int soff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_u8*)(size_t)__builtin_amdgcn_readfirstlane(lds_addr), 16, voff,
                                           __builtin_amdgcn_readfirstlane(soff), 0, 0);
}

// one tensor's pieces (TK: K, else V) of the chunk starting at key0 into stage st
template <bool TK, int D, int NUW, int CT, bool V16>
__device__ __forceinline__ void load_tile(const ChunkLoader<D, NUW, CT, V16>& f, int st, int key0) {
  using G = Geo<D>;
  const __amdgpu_buffer_rsrc_t& rs = TK ? f.krs : f.vrs;
  const unsigned base = (TK ? f.ks_base : f.vs_base) + st * CT;
  key0 = __builtin_amdgcn_readfirstlane(key0);
  if (key0 + 32 <= f.N) {
#pragma unroll
    for (int v = 0; v < NUW; ++v) buffer_to_lds(rs, base + (f.w * NUW + v) * 1024, TK ? f.kgv[v] : f.vgv[v], key0 * D * 2);
  } else {
    // The lane id goes through an empty asm so this rare path's per-lane
    // values are recomputed here rather than hoisted and kept live.
    if (key0 >= f.N) key0 = 0;
    const int valid = f.N - key0;
    int ln = f.lane;
    asm volatile("" : "+v"(ln));
    const int p = ln % G::NCH;
#pragma unroll
    for (int v = 0; v < NUW; ++v) {
      const int u = f.w * NUW + v;
      const int r = u * G::RPI + ln / G::NCH;
      const int rs_ = r < valid ? r : 0;
      int c = TK ? swz_k<G::NCH>(r, p) : (V16 ? swz_v16<G::NCH>(r, p) : swz_v<G::NCH>(r, p));
      if (c >= G::DCH) c = 0;
      buffer_to_lds(rs, base + u * 1024, (rs_ * D + c * 8) * 2, key0 * D * 2);
    }
  }
}

template <int D, int NUW, int CT, bool V16>
__device__ __forceinline__ void load_chunk(const ChunkLoader<D, NUW, CT, V16>& f, int st, int key0) {
  load_tile<true>(f, st, key0);
  load_tile<false>(f, st, key0);
}

// Per-lane LDS offset of the transpose reads of column tile dt (columns
// dt*32 ..) of a V-swizzled tile: row (kk*16 + hf*4 + n16/4 [+8]), piece
// dt*4 + (g16&1)*2 + (n16&3)/2; only dt interacts with the swizzle.  The
// stage and the kk / +8 row offsets are immediates.
template <int D>
__device__ __forceinline__ int tr_offset(int lane, int dt) {
  using G = Geo<D>;
  const int hf = lane >> 5, g16 = lane >> 4, n16 = lane & 15;
  const int vr = hf * 4 + (n16 >> 2);
  const int c = dt * 4 + (g16 & 1) * 2 + ((n16 & 3) >> 1);
  return vr * G::RB + (swz_v<G::NCH>(vr, c) << 4) + (n16 & 1) * 8;
}

// Per-lane LDS offsets.  K operand, step s: row l32 of the tile, piece
// 2s + hf.  V transpose reads: tr_offset.
template <int D>
__device__ __forceinline__ void operand_offsets(int lane, int (&koff)[Geo<D>::DQ], int (&voff)[Geo<D>::DT]) {
  using G = Geo<D>;
  const int hf = lane >> 5, l32 = lane & 31;
#pragma unroll
  for (int s = 0; s < G::DQ; ++s) koff[s] = l32 * G::RB + (swz_k<G::NCH>(l32, 2 * s + hf) << 4);
#pragma unroll
  for (int dt = 0; dt < G::DT; ++dt) voff[dt] = tr_offset<D>(lane, dt);
}

// Transpose read of a V-swizzled [32 rows][RB] tile: lane l gets column
// dt*32 + l%32 (through voff = tr_offset(lane, dt)) at the 8 rows of key half
// kk in the order rows kk*16 + hf*4 + 0..3, then kk*16 + 8 + hf*4 + 0..3 (the
// key order of a 32x32x16 S^T register group).  The same register serves as the A operand
// (row m = the column) or the B operand (column n = the column) of an MFMA
// whose contraction runs over the tile's rows.
template <int D>
__device__ __forceinline__ bf16x8 tr_operand(const unsigned char* tile, int voff, int kk) {
  using G = Geo<D>;
  // rows r and r + 8 have the same swizzle, so one offset serves both
  const unsigned char* p = tile + voff + kk * 16 * G::RB;
  const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p));
  const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p + 8 * G::RB));
  const u32x2 lw = __builtin_bit_cast(u32x2, lo);
  const u32x2 hw = __builtin_bit_cast(u32x2, hi);
  const u32x4 vw = {lw[0], lw[1], hw[0], hw[1]};
  return __builtin_bit_cast(bf16x8, vw);
}

// the NaN mark on a query block's first output element (recomputed later)
template <bool OUT_F32>
__device__ __forceinline__ void mark_block(void* out, size_t first) {
  if constexpr (OUT_F32) static_cast<float*>(out)[first] = __builtin_nanf("");
  else static_cast<uint16_t*>(out)[first] = 0x7FC0;
}

}  // namespace attn
}  // namespace sva
