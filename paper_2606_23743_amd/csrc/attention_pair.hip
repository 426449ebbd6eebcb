// Block-sparse attention for 64-token blocks, two neighbouring query blocks
// per workgroup (Section 4.2.2: kept blocks computed exactly).
//
// Neighbouring query blocks of a video keep almost the same key blocks (for
// the block-64 layers the union of two neighbours' lists is 55-70% of their
// combined length).  A workgroup takes query blocks 2p and 2p+1 with four
// waves of 32 queries (waves 0, 1: block 2p; waves 2, 3: block 2p+1) and walks
// the union of the two kept lists: every key chunk is staged in LDS once for
// both blocks, and each wave computes only on the key blocks its own query
// block keeps.  The stage pipeline is the one of the 128-token kernel: 32-key
// chunks, four LDS stages, loads three chunks ahead, so one loop iteration
// covers two union entries (four chunks) and every stage index is a constant.
//
// The union is built in LDS from two bitmaps over the key blocks, which needs
// lists that are strictly increasing and in range, as the selection kernel
// writes them.  A pair with any other list (out-of-range entries, repeats,
// another order) is marked (NaN first output element of both blocks) and the
// per-iteration rescaling kernel that runs next recomputes it with the general
// list semantics.  Per chunk, the arithmetic of a wave is that of the
// 32-query kernel (attn_w16.h: Sᵀ = K·Qᵀ on 16x16x32 products, fixed reference
// maximum from the wave's first chunk, P rounded to bf16 with l summed from
// it, Oᵀ += Vᵀ·Pᵀ), so keep-all lists give dense attention bit for bit.
#include "attn_w16.h"

namespace sva {
namespace {

using namespace attn;

constexpr int kPairMaxBlocks = 4096;         // key blocks a pair's bitmaps and union hold

template <int D, bool OUT_F32>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2)))
void attn_pair_kernel(AttnArgs a, int n_pairs) {
  using G = Geo<D>;
  using G16 = Geo16<D>;
  constexpr int S = 64;                      // tokens per (query and key) block
  constexpr int NW = 4;                      // waves per workgroup
  constexpr int CK = 32;                     // keys per staged chunk
  constexpr int NST = 4;                     // LDS stages (two union entries)
  constexpr int PD = NST - 1;                // prefetch distance, in chunks
  constexpr int CT = CK * G::RB;             // bytes of one chunk tile (K or V)
  constexpr int NUW = CT / 1024 / NW;        // direct-load pieces per wave per tile
  constexpr int kWords = kPairMaxBlocks / 32;
  static_assert(NUW >= 1, "tile split");

  __shared__ __attribute__((aligned(1024))) unsigned char Ks[NST][CT];
  __shared__ __attribute__((aligned(1024))) unsigned char Vs[NST][CT];
  __shared__ uint16_t ulist[kPairMaxBlocks];  // (block << 2) | (kept by 2p) | (kept by 2p+1) << 1
  __shared__ uint32_t bm[2][kWords];
  __shared__ int n_union, list_bad, wg_bad;

  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int N = a.N, nB = a.nB;
  const float sl2 = a.scale_log2;

  const int npb = (nB + 1) / 2;              // pairs per (b, h)
  // segments of 8 x 64 pairs (the eight XCDs on one head at a time), and
  // inside a head frame tiles of 2 pairs x 8 frames
  const int pr = __builtin_amdgcn_readfirstlane(xcd_remap_segments(blockIdx.x, n_pairs, 64));
  const int bh = pr / npb;
  const int pairs_per_frame = max(1, (a.frame_blocks + 1) / 2);
  const int p = frame_tile_order(pr - bh * npb, npb, pairs_per_frame, 8, 2);
  const int qsel = w >> 1;                   // 0: block 2p, 1: block 2p+1
  const int qb = 2 * p + qsel;               // this wave's query block (may be nB: none)
  const bool has_b = 2 * p + 1 < nB;
  const int row0 = bh * nB + 2 * p;          // row of block 2p; 2p+1 is row0 + 1
  const size_t head = (size_t)bh * N * D;
  const uint16_t* Qh = a.q + head;
  const uint16_t* Kh = a.k + head;
  const uint16_t* Vh = a.v + head;

  // ---- the union of the two kept lists ----
  const int words = (nB + 31) >> 5;
  for (int t = threadIdx.x; t < 2 * kWords; t += 256) (&bm[0][0])[t] = 0u;
  if (threadIdx.x == 0) {
    list_bad = 0;
    wg_bad = 0;
  }
  __syncthreads();
  int cnt2[2];
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    cnt2[s] = 0;
    if (s == 0 || has_b) cnt2[s] = min(max(a.kv_count[row0 + s], 0), a.kmax);
  }
  bool bad = false;
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    const int32_t* idx = a.kv_idx + (size_t)(row0 + s) * a.kmax;
    for (int t = threadIdx.x; t < cnt2[s]; t += 256) {
      const int j = idx[t];
      const bool ok = j >= 0 && j < nB && (t + 1 == cnt2[s] || j < idx[t + 1]);
      if (ok) atomicOr(&bm[s][j >> 5], 1u << (j & 31));
      else bad = true;
    }
  }
  if (__builtin_amdgcn_ballot_w64(bad) != 0 && lane == 0) atomicOr(&list_bad, 1);
  __syncthreads();
  if (list_bad) {                            // general lists: recomputed by the rescaling kernel
    if (threadIdx.x < 2 && (threadIdx.x == 0 || has_b))
      mark_block<OUT_F32>(a.out, head + (size_t)(2 * p + threadIdx.x) * S * D);
    return;
  }
  if (w == 0) {                              // compaction in block order, 64 words per step
    int base = 0;
    for (int w0 = 0; w0 < words; w0 += 64) {
      const int wd = w0 + lane;
      const uint32_t ba = wd < words ? bm[0][wd] : 0u;
      const uint32_t bb = wd < words ? bm[1][wd] : 0u;
      uint32_t u = ba | bb;
      const int c = __builtin_popcount(u);
      int incl = c;                          // inclusive prefix over the lanes
#pragma unroll
      for (int off = 1; off < 64; off <<= 1) {
        const int y = __shfl_up(incl, off, 64);
        if (lane >= off) incl += y;
      }
      int pos = base + incl - c;
      while (u != 0) {
        const int k = __builtin_ctz(u);
        u &= u - 1;
        const int j = wd * 32 + k;
        ulist[pos++] = (uint16_t)((j << 2) | ((ba >> k) & 1u) | (((bb >> k) & 1u) << 1));
      }
      base += __shfl(incl, 63, 64);
    }
    if (lane == 0) n_union = base;
  }
  __syncthreads();
  const int U = n_union;
  auto ent = [&](int e) -> int {             // union entry e (block 0, kept by neither, past the end)
    return __builtin_amdgcn_readfirstlane(e < U ? (int)ulist[e] : 0);
  };
  auto active = [&](int u) -> bool { return ((u >> qsel) & 1) != 0; };
  auto key0_of = [&](int u, int c2) -> int { return (u >> 2) * S + c2 * CK; };

  // ---- Q^T operands: queries qb*S + (w&1)*32 + 0..31 ----
  const int qbase = qb * S + (w & 1) * 32;
  bf16x8 qop[2][G16::KS];
  load_q16<D>(qop, Qh, qbase, qb < nB ? N : 0, lane);

  // direct global -> LDS loads of this wave's pieces of a chunk
  ChunkLoader<D, NUW, CT, true> ld;
  loader_init(ld, Kh, Vh, N, &Ks[0][0], &Vs[0][0], w, lane);
  auto fetch = [&](int st, int key0) { load_chunk(ld, st, key0); };

  int koff[G16::KS], voff[G16::DT];
  operand_offsets16<D>(lane, koff, voff);

  float m_ref[2] = {0.0f, 0.0f};
  float l_part[2] = {0.0f, 0.0f};
  bool ref_set = false;                      // wave-uniform: the reference is taken
  f32x4 oacc[G16::DT][2];
#pragma unroll
  for (int dt = 0; dt < G16::DT; ++dt) oacc[dt][0] = oacc[dt][1] = f32x4{};

  auto qk = [&](f32x4 (&s)[2][2], const unsigned char* kt) { qk16<D>(s, kt, koff, qop); };
  auto softmax = [&](const f32x4 (&s)[2][2], bf16x8 (&pop)[2]) { softmax16(s, pop, l_part, m_ref, sl2); };
  auto pv = [&](const bf16x8 (&pop)[2], const unsigned char* vt) { pv16<D>(pop, vt, voff, oacc); };
  auto take = [](f32x4 (&dst)[2][2], const f32x4 (&src)[2][2]) {
#pragma unroll
    for (int x = 0; x < 2; ++x) {
      dst[x][0] = src[x][0];
      dst[x][1] = src[x][1];
    }
  };

  // ---- pipeline over the union, two entries (four chunks) per iteration ----
  // Chunk c of an iteration: entry u0 (c = 0, 1) or u1 (c = 2, 3), half c % 2,
  // in stage c.  After the barrier of chunk c the stage of chunk c-1 is free
  // and receives the chunk three ahead (u1's second half, then u2's halves and
  // u3's first).  Each chunk issues one load group (past the end: block 0, in
  // bounds), so the wait count is a constant, as in the 32-query kernel.
  int u0 = ent(0), u1 = ent(1), u2 = ent(2), u3 = ent(3);
  f32x4 sacc[2][2];
#pragma unroll
  for (int x = 0; x < 2; ++x) sacc[x][0] = sacc[x][1] = f32x4{};
  if (U > 0) {
    fetch(0, key0_of(u0, 0));
    fetch(1, key0_of(u0, 1));
    fetch(2, key0_of(u1, 0));
    wait_vmcnt<2 * NUW * (PD - 1)>();
    wg_barrier();
    if (active(u0)) {
      qk(sacc, &Ks[0][0]);
      const int valid = __builtin_amdgcn_readfirstlane(N - key0_of(u0, 0));
      if (valid < CK) mask_tail16(sacc, valid, lane);
      chunk_reference16(sacc, sl2, m_ref);   // chunk 0 of a block holds a valid key
      ref_set = true;
    }
  }
  for (int e = 0; e < U; e += 2) {
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      wait_vmcnt_lds_idle<2 * NUW * (PD - 2)>();     // chunk c+1 landed
      wg_barrier();
      if (c == 0) fetch(3, key0_of(u1, 1));
      else if (c == 1) fetch(0, key0_of(u2, 0));
      else if (c == 2) fetch(1, key0_of(u2, 1));
      else fetch(2, key0_of(u3, 0));
      const int uc = c < 2 ? u0 : u1;                 // this chunk's entry
      const int un = c == 0 ? u0 : (c < 3 ? u1 : u2); // the next chunk's entry
      const int nkey0 = key0_of(un, (c + 1) & 1);
      f32x4 snext[2][2];
#pragma unroll
      for (int x = 0; x < 2; ++x) snext[x][0] = snext[x][1] = f32x4{};
      bf16x8 pop[2];
      if (active(uc) && !ref_set) {                    // the wave's first chunk
        chunk_reference16(sacc, sl2, m_ref);
        ref_set = true;
      }
      if (active(un) && active(uc)) {
        // the common case in one basic block, so that the next chunk's S
        // products interleave with this chunk's softmax
        qk(snext, &Ks[(c + 1) & 3][0]);
        softmax(sacc, pop);
        pv(pop, &Vs[c][0]);
      } else {
        if (active(un)) qk(snext, &Ks[(c + 1) & 3][0]);
        if (active(uc)) {
          softmax(sacc, pop);
          pv(pop, &Vs[c][0]);
        }
      }
      const int nvalid = __builtin_amdgcn_readfirstlane(N - nkey0);
      if (nvalid < CK && active(un)) {
        asm volatile("");
        mask_tail16(snext, nvalid, lane);
      }
      take(sacc, snext);
      if (c & 1) rescale_if_large16<D>(l_part, m_ref, oacc);               // after each 64-key block
    }
    u0 = u2;
    u1 = u3;
    u2 = ent(e + 4);
    u3 = ent(e + 5);
  }
  wait_vmcnt<0>();           // no load may still target this workgroup's LDS

  // ---- epilogue: overflow check, then O = O^T / l and LSE ----
  float l_tot[2];
  l_tot[0] = quad_sum(l_part[0]);
  l_tot[1] = quad_sum(l_part[1]);
  const bool over = overflowed16<D>(l_tot, oacc);
  if (__builtin_amdgcn_ballot_w64(over) != 0 && lane == 0) atomicOr(&wg_bad, 1);
  __syncthreads();
  if (wg_bad) {
    if (threadIdx.x < 2 && (threadIdx.x == 0 || has_b))
      mark_block<OUT_F32>(a.out, head + (size_t)(2 * p + threadIdx.x) * S * D);
    return;
  }
  const bool has[2] = {ref_set && l_tot[0] > 0.0f, ref_set && l_tot[1] > 0.0f};
  if (qb < nB) store_query16<D, OUT_F32>(a.out, a.lse, head, (size_t)bh * N, qbase, N, oacc, l_tot, m_ref, has, lane);
}

template <int D>
hipError_t launch_pair(const Dims& d, const AttnArgs& a, hipStream_t stream) {
  const int n_pairs = d.B * d.H * ((d.nB + 1) / 2);
  dim3 grid(n_pairs), block(256);
  if (d.out_f32) hipLaunchKernelGGL((attn_pair_kernel<D, true>), grid, block, 0, stream, a, n_pairs);
  else hipLaunchKernelGGL((attn_pair_kernel<D, false>), grid, block, 0, stream, a, n_pairs);
  return hipGetLastError();
}

}  // namespace

// Pairs pay off when neighbours share enough of their blocks, which goes with
// denser lists.  Measured at D = 128 on the block-64 layers: rows of 18-100%
// of the blocks ran 6-33% faster in pairs, 12% ran 2.5% slower and 10% 8%
// slower (the waves of a block that does not keep an entry sit idle while it
// is staged).  At D = 112 (the 2B-class layer) the single-block kernel already
// runs near the dense rate and pairs were level or slower at every density.
bool pair_attention_fits(const Dims& d, int kmax) {
  return d.S == 64 && d.D == 128 && d.nB <= kPairMaxBlocks && 20LL * kmax >= 3LL * d.nB;
}

hipError_t launch_attention_pair(const Dims& d, const AttnArgs& a, hipStream_t stream) {
  if (d.D != 128) return hipErrorInvalidValue;
  return launch_pair<128>(d, a, stream);
}

}  // namespace sva
