// Block-sparse (and dense) flash attention, 32 queries per wave, two waves per
// SIMD (Section 4.2.2: kept blocks computed exactly; Appendix A.2.2: dense
// FlashAttention fallback).
//
// A workgroup is one query block of S tokens with S/32 waves of 32 queries.
// Each wave's state (O^T 64 registers, Q^T 32, S^T and P of a key chunk) fits
// in 256 registers, so two workgroups share a CU with two waves on every SIMD.
//
// Keys are processed in 32-key chunks staged in LDS, chunk c of a kept block
// in stage c (S/32 stages), filled by buffer_load ... lds straight from global
// memory ahead of use (S = 128: three chunks ahead; S = 64: K two chunks and
// V one chunk ahead).  Tiles are unpadded and XOR-swizzled on 16-byte pieces
// so that both the ds_read_b128 K operand reads and the ds_read_b64_tr_b16 V
// transpose reads are free of bank conflicts.  Each wave overlaps the next
// chunk's S^T MFMAs with the current chunk's softmax.
//
// Per 32-key sub-chunk (lane = one query; its 16 S^T registers are keys
// (r/4)*8 + half*4 + r%4):
//   S^T = K Q^T                mfma_f32_32x32x16_bf16, Q^T in registers
//   p   = exp2(c*log2e*s - m)  m is the reference maximum taken from the first
//                              chunk of the row, so O is not rescaled per chunk
//   l  += sum of the bf16 p    v_dot2 with (1, 1)
//   O^T += V^T P^T             P^T from the S^T registers, V^T by transpose reads
// After each kept block a row whose sum has passed 2^64 moves its reference up
// by a power of two (O and l scaled exactly).  A row that still overflows (its
// logits jump by more than ~2^63 over the running sum inside one block) is
// marked (NaN first element) and recomputed by the per-iteration rescaling
// kernel that runs next.
#include "attn_wave32.h"

namespace sva {
namespace {

using namespace attn;

template <int D, int S, bool SPARSE, bool OUT_F32>
__global__ __launch_bounds__(2 * S) __attribute__((amdgpu_waves_per_eu(2, 2)))
void attn_q32_kernel(AttnArgs a) {
  using G = Geo<D>;
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
  const int hf = lane >> 5;
  const int l32 = lane & 31;
  const int N = a.N, nB = a.nB;
  const float sl2 = a.scale_log2;

  // Sparse lists at S=128 run about 4% faster with the eight XCDs sharing one
  // head at a time (128 query blocks each); at S=64, and for dense walks, whole
  // ranges of heads per XCD are as fast or faster.
  constexpr int kSegRows = (SPARSE && S == 128) ? 128 : 0;
  const int wg = kSegRows ? xcd_remap_segments(blockIdx.x, a.n_rows, kSegRows) : xcd_remap(blockIdx.x, a.n_rows);
  const int row = __builtin_amdgcn_readfirstlane(wg);   // (b*H + h)*nB + i
  const int bh = row / nB;
  const int i = row - bh * nB;
  const size_t head = (size_t)bh * N * D;
  const uint16_t* Qh = a.q + head;
  const uint16_t* Kh = a.k + head;
  const uint16_t* Vh = a.v + head;

  // ---- Q^T operand: query i*S + w*32 + l32 ----
  const int qr = i * S + w * 32 + l32;
  bf16x8 qop[G::DQ];
  load_q<D>(qop, Qh, qr, qr < N, hf);

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
  ChunkLoader<D, NUW, CT> ld;
  loader_init(ld, Kh, Vh, N, &Ks[0][0], &Vs[0][0], w, lane);
  auto fetch_k = [&](int st, int key0) { load_tile<true>(ld, st, key0); };
  auto fetch_v = [&](int st, int key0) { load_tile<false>(ld, st, key0); };
  auto fetch = [&](int st, int key0) { load_chunk(ld, st, key0); };

  int koff[G::DQ], voff[G::DT];
  operand_offsets<D>(lane, koff, voff);

  float m_ref = 0.0f;        // reference max (log2 units), fixed by the first chunk
  float l_part = 0.0f;       // this lane's half of the row sum
  f32x16 oacc[G::DT];
#pragma unroll
  for (int dt = 0; dt < G::DT; ++dt) oacc[dt] = f32x16{};

  auto qk = [&](f32x16& sacc, const unsigned char* kt) { qk_chunk<D>(sacc, kt, koff, qop); };
  auto softmax = [&](const f32x16& sacc, bf16x8 (&pop)[2]) { softmax_chunk(sacc, pop, l_part, m_ref, sl2); };
  auto pv = [&](const bf16x8 (&pop)[2], const unsigned char* vt) { pv_chunk<D>(pop, vt, voff, oacc); };

  // ---- pipeline over (kept block, chunk) ----
  // Chunk c of every block lives in stage c (NST = NCK stages), so stages and
  // LDS offsets are compile-time in the unrolled chunk loop.  At chunk c a
  // wave waits for its own loads of that chunk and for its own LDS reads of
  // chunk c-1 (the compiler may leave the last V reads in flight, their MFMAs
  // sunk below the barrier); after the barrier every wave's loads have landed
  // and every wave is done reading chunk c-1, so the loads of the chunk
  // PD = NST-1 positions ahead go into chunk c-1's stage.  Each chunk issues
  // exactly one load group (a dummy past the end of the list), so the wait
  // count is a constant.  The block index after the next is read one block
  // ahead, after chunk 0's barrier so that its scalar load has a whole chunk
  // to land before the next LDS-idle wait.
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
  if constexpr (PIPE) {
    // Software pipeline inside the wave: the S MFMAs of the next chunk are
    // issued alongside the softmax of this one, then this chunk's PV.  At
    // iteration c the wave needs K of chunk c+1 and V of chunk c; after
    // iteration c's barrier chunk c-1's stage is free (its K was read at
    // iteration c-2, its V at c-1), and it receives chunk c+PD.  The last
    // chunk of the list computes S for a dummy next chunk (stage 0 holds
    // in-bounds data then), which is dropped.
    f32x16 sacc = f32x16{};
    if (it < count) {
      wait_vmcnt<2 * NUW * (PD - 1)>();
      wg_barrier();
      qk(sacc, &Ks[0][0]);
      const int valid = __builtin_amdgcn_readfirstlane(N - j * S);
      if (valid < CK) mask_tail(sacc, valid, hf);
      m_ref = chunk_reference(sacc, sl2);   // chunk 0 holds a valid key: finite
    }
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
        f32x16 snext;
        bf16x8 pop[2];
        qk(snext, &Ks[(c + 1) % NST][0]);
        softmax(sacc, pop);
        // The PV products issue at raised wave priority, ahead of the other
        // wave's softmax on the SIMD: measured 1.5-2.5% faster at the 64B-class
        // layer (raising it for the S products or the softmax was slower).
        __builtin_amdgcn_s_setprio(1);
        pv(pop, &Vs[c][0]);
        __builtin_amdgcn_s_setprio(0);
        const int nvalid = __builtin_amdgcn_readfirstlane(N - nkey0);
        if (nvalid < CK) {
          asm volatile("");        // keep this a real (rarely taken) branch, not select code
          mask_tail(snext, nvalid, hf);
        }
        sacc = snext;
      }
      rescale_if_large<D>(l_part, m_ref, oacc);
      advance_block(itnn, jnn);
    }
  } else {
    // Two stages (S = 64): the same overlap with K and V prefetched at
    // different distances.  At iteration c the wave reads K of chunk c+1 and
    // V of chunk c; after the barrier K stage c (last read by the S MFMAs of
    // iteration c-1) receives K of chunk c+2, i.e. chunk c of the next block,
    // and V stage c+1 (last read by the PV of iteration c-1) receives V of
    // chunk c+1.  Each iteration issues one K and one V group and waits for
    // the previous iteration's, so the wait is for everything.
    static_assert(NST == 2 && NCK == 2, "two-stage pipeline");
    f32x16 sacc = f32x16{};
    if (it < count) {
      wait_vmcnt<0>();
      wg_barrier();
      qk(sacc, &Ks[0][0]);
      const int valid = __builtin_amdgcn_readfirstlane(N - j * S);
      if (valid < CK) mask_tail(sacc, valid, hf);
      m_ref = chunk_reference(sacc, sl2);   // chunk 0 holds a valid key: finite
    }
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
        f32x16 snext;
        bf16x8 pop[2];
        qk(snext, &Ks[(c + 1) % NST][0]);
        softmax(sacc, pop);
        pv(pop, &Vs[c][0]);
        const int nvalid = __builtin_amdgcn_readfirstlane(N - nkey0);
        if (nvalid < CK) {
          asm volatile("");        // keep this a real (rarely taken) branch, not select code
          mask_tail(snext, nvalid, hf);
        }
        sacc = snext;
      }
      rescale_if_large<D>(l_part, m_ref, oacc);
      advance_block(itnn, jnn);
    }
  }
  wait_vmcnt<0>();           // no load may still target this workgroup's LDS

  // ---- epilogue: overflow check, then O = O^T / l and LSE ----
  if (threadIdx.x == 0) wg_bad = 0;
  const float l_tot = swap_halves_sum(l_part);
  const bool bad = overflowed<D>(l_tot, oacc);
  __syncthreads();
  if (__builtin_amdgcn_ballot_w64(bad) != 0 && lane == 0) atomicOr(&wg_bad, 1);
  __syncthreads();
  if (wg_bad) {
    if (threadIdx.x == 0 && i * S < N) mark_block<OUT_F32>(a.out, head + (size_t)i * S * D);
    return;
  }
  const bool has = count > 0 && l_tot > 0.0f;
  if (qr < N)
    store_query<D, OUT_F32>(a.out, a.lse, head + (size_t)qr * D, (size_t)bh * N + qr, oacc, l_tot, m_ref, has, hf);
}

template <int D, int S>
hipError_t launch_q32(const Dims& d, bool sparse, const AttnArgs& a, hipStream_t stream) {
  dim3 grid(a.n_rows), block(2 * S);
  if (sparse) {
    if (d.out_f32) hipLaunchKernelGGL((attn_q32_kernel<D, S, true, true>), grid, block, 0, stream, a);
    else hipLaunchKernelGGL((attn_q32_kernel<D, S, true, false>), grid, block, 0, stream, a);
  } else {
    if (d.out_f32) hipLaunchKernelGGL((attn_q32_kernel<D, S, false, true>), grid, block, 0, stream, a);
    else hipLaunchKernelGGL((attn_q32_kernel<D, S, false, false>), grid, block, 0, stream, a);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attention_q32(const Dims& d, bool sparse, const AttnArgs& a, hipStream_t stream) {
  switch (d.D * 1000 + d.S) {
    case 64128: return launch_q32<64, 128>(d, sparse, a, stream);
    case 112128: return launch_q32<112, 128>(d, sparse, a, stream);
    case 128128: return launch_q32<128, 128>(d, sparse, a, stream);
    case 64064: return launch_q32<64, 64>(d, sparse, a, stream);
    case 112064: return launch_q32<112, 64>(d, sparse, a, stream);
    case 128064: return launch_q32<128, 64>(d, sparse, a, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace sva
