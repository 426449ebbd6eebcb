// Block-sparse (and dense) flash attention on mfma_f32_16x16x32_bf16, 32
// queries per wave, two waves per SIMD (Section 4.2.2: kept blocks computed
// exactly; Appendix A.2.2: dense FlashAttention fallback).
//
// A workgroup is one query block of S tokens with S/32 waves of 32 queries.
// Each wave's state (O^T 4*D/16*2 registers, Q^T, S^T and P of a key chunk)
// fits in 256 registers, so two workgroups share a CU with two waves on every
// SIMD.
//
// Keys are processed in 32-key chunks staged in LDS, chunk c of a kept block
// in stage c (S/32 stages), filled by buffer_load ... lds straight from global
// memory ahead of use (S = 128: three chunks ahead; S = 64: K two chunks and
// V one chunk ahead).  Tiles are unpadded and XOR-swizzled on 16-byte pieces
// so that the ds_read_b128 K operand reads and the ds_read_b64_tr_b16 V
// transpose reads are free of bank conflicts.  Each wave overlaps the next
// chunk's S^T products with the current chunk's softmax, then issues the
// current chunk's PV products.  The per-chunk arithmetic (attn_w16.h):
//   S^T = K Q^T                Q^T in registers
//   p   = exp2(c*log2e*s - m)  m is the reference maximum taken from the
//                              query's first chunk, so O is not rescaled per
//                              chunk
//   l  += sum of the bf16 p    v_dot2 with (1, 1)
//   O^T += V^T P^T             P^T from the S^T registers, V^T by transpose reads
// After each kept block a query whose sum has passed 2^64 moves its reference
// up by a power of two (O and l scaled exactly).  A block with a query that
// still overflows (its logits jump by more than ~2^63 over the running sum
// inside one block) is marked (NaN first element) and recomputed by the
// per-iteration rescaling kernel that runs next.
//
// Workgroup order: sparse lists run, inside a head, in frame tiles of 4
// consecutive query blocks x 8 frames (frame_tile_order), so the query blocks
// an XCD runs at once are neighbours in (t, y, x) and keep mostly the same key
// blocks.  At S = 128 the rows are also cut into segments of 8 x 128
// (xcd_remap_segments: the eight XCDs work through one head at a time); at
// S = 64, and for dense walks, each XCD takes a whole range of rows
// (xcd_remap).
#include "attn_w16.h"

namespace sva {
namespace {

using namespace attn;

template <int D, int S, bool SPARSE, bool OUT_F32>
__global__ __launch_bounds__(2 * S) __attribute__((amdgpu_waves_per_eu(2, 2)))
void attn_q16_kernel(AttnArgs a) {
  using G = Geo<D>;
  using G16 = Geo16<D>;
  constexpr int NW = S / 32;                 // waves per workgroup
  constexpr int CK = 32;                     // keys per staged chunk
  constexpr int NCK = S / CK;                // chunks per block
  constexpr int NST = NCK;                   // LDS stages: chunk c of a block in stage c
  constexpr int PD = NST - 1;                // prefetch distance, in chunks
  constexpr bool PIPE = NST >= 4;            // four stages (S = 128); else two (S = 64)
  constexpr int CT = CK * G::RB;             // bytes of one chunk tile (K or V)
  constexpr int NUW = CT / 1024 / NW;        // direct-load pieces per wave per tile
  static_assert(NUW >= 1 && PD >= 1, "tile split");

  __shared__ __attribute__((aligned(1024))) unsigned char Ks[NST][CT];
  __shared__ __attribute__((aligned(1024))) unsigned char Vs[NST][CT];
  __shared__ int wg_bad;

  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int N = a.N, nB = a.nB;
  const float sl2 = a.scale_log2;

  constexpr bool kSegments = SPARSE && S == 128;
  const int wg = kSegments ? xcd_remap_segments(blockIdx.x, a.n_rows, 128) : xcd_remap(blockIdx.x, a.n_rows);
  const int rowl = __builtin_amdgcn_readfirstlane(wg);   // (b*H + h)*nB + logical block
  const int bh = rowl / nB;
  const int i = SPARSE ? frame_tile_order(rowl - bh * nB, nB, a.frame_blocks, 8, 4) : rowl - bh * nB;
  const int row = bh * nB + i;
  const size_t head = (size_t)bh * N * D;
  const uint16_t* Qh = a.q + head;
  const uint16_t* Kh = a.k + head;
  const uint16_t* Vh = a.v + head;

  // ---- Q^T operands: queries i*S + w*32 + 0..31 ----
  const int qbase = i * S + w * 32;
  bf16x8 qop[2][G16::KS];
  load_q16<D>(qop, Qh, qbase, N, lane);

  // ---- the kept-block list ----
  // Read through the constant address space: uniform reads become scalar
  // loads (lgkmcnt), so they never wait on the in-flight tile loads.
  int count;
  const_i32* idxrow = nullptr;
  if constexpr (SPARSE) {
    count = __builtin_amdgcn_readfirstlane(min(max(((const_i32*)a.kv_count)[row], 0), a.kmax));
    idxrow = (const_i32*)a.kv_idx + (size_t)row * a.kmax;
  } else {
    count = nB;
  }
  auto raw_at = [&](int it) -> int {
    return __builtin_amdgcn_readfirstlane(SPARSE ? idxrow[it] : it);
  };
  auto in_range = [&](int j) -> bool { return j >= 0 && j < nB; };
  auto seek = [&](int it) -> int {         // first usable entry at or after it
    while (it < count && !in_range(raw_at(it))) ++it;
    return it;
  };

  // direct global -> LDS loads of this wave's pieces of a chunk
  ChunkLoader<D, NUW, CT, true> ld;
  loader_init(ld, Kh, Vh, N, &Ks[0][0], &Vs[0][0], w, lane);
  auto fetch_k = [&](int st, int key0) { load_tile<true>(ld, st, key0); };
  auto fetch_v = [&](int st, int key0) { load_tile<false>(ld, st, key0); };
  auto fetch = [&](int st, int key0) { load_chunk(ld, st, key0); };

  int koff[G16::KS], voff[G16::DT];
  operand_offsets16<D>(lane, koff, voff);

  float m_ref[2] = {0.0f, 0.0f};     // reference max (log2 units) per query tile
  float l_part[2] = {0.0f, 0.0f};    // this lane's quarter of each row sum
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

  // ---- pipeline over (kept block, chunk) ----
  // Chunk c of every block lives in stage c (NST = NCK stages), so stages and
  // LDS offsets are compile-time in the unrolled chunk loop.  At chunk c a
  // wave waits for its own loads of that chunk and for its own LDS reads of
  // chunk c-1; after the barrier every wave's loads have landed and every wave
  // is done reading chunk c-1, so the loads of the chunk PD = NST-1 positions
  // ahead go into chunk c-1's stage.  Each chunk issues exactly one load group
  // (a dummy past the end of the list), so the wait count is a constant.  The
  // block index after the next is read one block ahead, after chunk 0's
  // barrier so that its scalar load has a whole chunk to land before the next
  // LDS-idle wait.
  int it = seek(0);
  int j = it < count ? raw_at(it) : 0;
  int itn = it < count ? seek(it + 1) : count;
  int jn = itn < count ? raw_at(itn) : -1;
  if (it < count) {
#pragma unroll
    for (int c = 0; c < PD; ++c) fetch(c, j * S + c * CK);
    if constexpr (!PIPE) fetch_k(1, j * S + CK);
  }
  auto advance_block = [&](int itnn, int jnn) {
    it = itn;
    j = jn;
    if (itnn >= count || in_range(jnn)) {
      itn = itnn;
      jn = jnn;
    } else {
      itn = seek(itnn + 1);
      jn = itn < count ? raw_at(itn) : -1;
    }
  };
  f32x4 sacc[2][2];
#pragma unroll
  for (int x = 0; x < 2; ++x) sacc[x][0] = sacc[x][1] = f32x4{};
  if (it < count) {
    if constexpr (PIPE) wait_vmcnt<2 * NUW * (PD - 1)>();
    else wait_vmcnt<0>();
    wg_barrier();
    qk(sacc, &Ks[0][0]);
    const int valid = __builtin_amdgcn_readfirstlane(N - j * S);
    if (valid < CK) mask_tail16(sacc, valid, lane);
    chunk_reference16(sacc, sl2, m_ref);   // chunk 0 holds a valid key: finite
  }
  if constexpr (PIPE) {
    // Software pipeline inside the wave: the S products of the next chunk are
    // issued alongside the softmax of this one, then this chunk's PV.  At
    // iteration c the wave needs K of chunk c+1 and V of chunk c; after
    // iteration c's barrier chunk c-1's stage is free (its K was read at
    // iteration c-2, its V at c-1), and it receives chunk c+PD.  The last
    // chunk of the list computes S for a dummy next chunk (stage 0 holds
    // in-bounds data then), which is dropped.
    while (it < count) {
      const int itnn = itn + 1;
      int jnn = -1;
#pragma unroll
      for (int c = 0; c < NCK; ++c) {
        wait_vmcnt_lds_idle<2 * NUW * (PD - 2)>();     // chunk c+1 landed
        wg_barrier();
        if (c + PD < NCK) fetch((c + PD) % NST, j * S + (c + PD) * CK);
        else fetch((c + PD) % NST, jn >= 0 ? jn * S + (c + PD - NCK) * CK : 0);
        if (c == 0) jnn = itnn < count ? raw_at(itnn) : -1;
        const int nkey0 = c + 1 < NCK ? j * S + (c + 1) * CK : (jn >= 0 ? jn * S : 0);
        f32x4 snext[2][2];
        bf16x8 pop[2];
        qk(snext, &Ks[(c + 1) % NST][0]);
        softmax(sacc, pop);
        // The PV products issue at raised wave priority, ahead of the other
        // wave's softmax on the SIMD (measured 1.6% faster at the 64B-class
        // layer than the default priority).
        __builtin_amdgcn_s_setprio(1);
        pv(pop, &Vs[c][0]);
        __builtin_amdgcn_s_setprio(0);
        const int nvalid = __builtin_amdgcn_readfirstlane(N - nkey0);
        if (nvalid < CK) {
          asm volatile("");        // keep this a real (rarely taken) branch, not select code
          mask_tail16(snext, nvalid, lane);
        }
        take(sacc, snext);
      }
      rescale_if_large16<D>(l_part, m_ref, oacc);
      advance_block(itnn, jnn);
    }
  } else {
    // Two stages (S = 64): the same overlap with K and V prefetched at
    // different distances.  At iteration c the wave reads K of chunk c+1 and
    // V of chunk c; after the barrier K stage c (last read by the S products
    // of iteration c-1) receives K of chunk c+2, i.e. chunk c of the next
    // block, and V stage c+1 (last read by the PV of iteration c-1) receives
    // V of chunk c+1.  Each iteration issues one K and one V group and waits
    // for the previous iteration's, so the wait is for everything.
    static_assert(NST == 2 && NCK == 2, "two-stage pipeline");
    while (it < count) {
      const int itnn = itn + 1;
      int jnn = -1;
#pragma unroll
      for (int c = 0; c < NCK; ++c) {
        wait_vmcnt_lds_idle<0>();          // K of chunk c+1 and V of chunk c landed
        wg_barrier();
        fetch_k(c, jn >= 0 ? jn * S + c * CK : 0);
        if (c + 1 < NCK) fetch_v(c + 1, j * S + (c + 1) * CK);
        else fetch_v(0, jn >= 0 ? jn * S : 0);
        if (c == 0) jnn = itnn < count ? raw_at(itnn) : -1;
        const int nkey0 = c + 1 < NCK ? j * S + (c + 1) * CK : (jn >= 0 ? jn * S : 0);
        f32x4 snext[2][2];
        bf16x8 pop[2];
        qk(snext, &Ks[(c + 1) % NST][0]);
        softmax(sacc, pop);
        pv(pop, &Vs[c][0]);
        const int nvalid = __builtin_amdgcn_readfirstlane(N - nkey0);
        if (nvalid < CK) {
          asm volatile("");        // keep this a real (rarely taken) branch, not select code
          mask_tail16(snext, nvalid, lane);
        }
        take(sacc, snext);
      }
      rescale_if_large16<D>(l_part, m_ref, oacc);
      advance_block(itnn, jnn);
    }
  }
  wait_vmcnt<0>();           // no load may still target this workgroup's LDS

  // ---- epilogue: overflow check, then O = O^T / l and LSE ----
  if (threadIdx.x == 0) wg_bad = 0;
  float l_tot[2];
  l_tot[0] = quad_sum(l_part[0]);
  l_tot[1] = quad_sum(l_part[1]);
  const bool bad = overflowed16<D>(l_tot, oacc);
  __syncthreads();
  if (__builtin_amdgcn_ballot_w64(bad) != 0 && lane == 0) atomicOr(&wg_bad, 1);
  __syncthreads();
  if (wg_bad) {
    if (threadIdx.x == 0 && i * S < N) mark_block<OUT_F32>(a.out, head + (size_t)i * S * D);
    return;
  }
  const bool has[2] = {count > 0 && l_tot[0] > 0.0f, count > 0 && l_tot[1] > 0.0f};
  store_query16<D, OUT_F32>(a.out, a.lse, head, (size_t)bh * N, qbase, N, oacc, l_tot, m_ref, has, lane);
}

template <int D, int S>
hipError_t launch_q16(const Dims& d, bool sparse, const AttnArgs& a, hipStream_t stream) {
  dim3 grid(a.n_rows), block(2 * S);
  if (sparse) {
    if (d.out_f32) hipLaunchKernelGGL((attn_q16_kernel<D, S, true, true>), grid, block, 0, stream, a);
    else hipLaunchKernelGGL((attn_q16_kernel<D, S, true, false>), grid, block, 0, stream, a);
  } else {
    if (d.out_f32) hipLaunchKernelGGL((attn_q16_kernel<D, S, false, true>), grid, block, 0, stream, a);
    else hipLaunchKernelGGL((attn_q16_kernel<D, S, false, false>), grid, block, 0, stream, a);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attention_q16(const Dims& d, bool sparse, const AttnArgs& a, hipStream_t stream) {
  switch (d.D * 1000 + d.S) {
    case 64128: return launch_q16<64, 128>(d, sparse, a, stream);
    case 112128: return launch_q16<112, 128>(d, sparse, a, stream);
    case 128128: return launch_q16<128, 128>(d, sparse, a, stream);
    case 64064: return launch_q16<64, 64>(d, sparse, a, stream);
    case 112064: return launch_q16<112, 64>(d, sparse, a, stream);
    case 128064: return launch_q16<128, 64>(d, sparse, a, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace sva
