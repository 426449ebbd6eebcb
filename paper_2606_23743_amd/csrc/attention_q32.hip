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
#include <type_traits>

#include "attn_common.h"

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
  const int g16 = lane >> 4;
  const int n16 = lane & 15;
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

  // ---- Q^T operand: query i*S + w*32 + l32, d = s*16 + hf*8 + 0..7 ----
  const int qr = i * S + w * 32 + l32;
  bf16x8 qop[G::DQ];
#pragma unroll
  for (int s = 0; s < G::DQ; ++s) {
    if (qr < N) qop[s] = *reinterpret_cast<const bf16x8*>(Qh + (size_t)qr * D + s * 16 + hf * 8);
    else qop[s] = bf16x8{};
  }

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

  // ---- direct global -> LDS fetch of one chunk (this wave's 1 KB pieces) ----
  // Piece u covers chunk rows u*RPI .. u*RPI + RPI - 1; lane L fills row
  // u*RPI + L/NCH at position L % NCH, i.e. global piece (L % NCH) ^ swizzle(row).
  // A wave always loads the same pieces, so its per-lane byte offsets are
  // fixed and the chunk's key offset is the scalar offset.  Every address
  // formed lies inside the head's rows: full chunks by construction, the
  // sequence's last partial chunk by clamping rows past the end to its first
  // row, and a chunk wholly past the end (the rest of a partial block, or a
  // pipeline slot with nothing left to load) by reading chunk 0 instead.
  const __amdgpu_buffer_rsrc_t krs = __builtin_amdgcn_make_buffer_rsrc((void*)Kh, (short)0, N * D * 2, 0x00020000);
  const __amdgpu_buffer_rsrc_t vrs = __builtin_amdgcn_make_buffer_rsrc((void*)Vh, (short)0, N * D * 2, 0x00020000);
  int kgv[NUW], vgv[NUW];
#pragma unroll
  for (int v = 0; v < NUW; ++v) {
    const int r = (w * NUW + v) * G::RPI + lane / G::NCH;
    const int p = lane % G::NCH;
    int ck = swz_k<G::NCH>(r, p), cv = swz_v<G::NCH>(r, p);
    if (ck >= G::DCH) ck = 0;                        // padding pieces: any in-row address
    if (cv >= G::DCH) cv = 0;
    kgv[v] = (r * D + ck * 8) * 2;
    vgv[v] = (r * D + cv * 8) * 2;
  }
  typedef __attribute__((address_space(3))) unsigned char lds_u8;
  const unsigned ks_base = __builtin_amdgcn_readfirstlane((unsigned)(size_t)(lds_u8*)&Ks[0][0]);
  const unsigned vs_base = __builtin_amdgcn_readfirstlane((unsigned)(size_t)(lds_u8*)&Vs[0][0]);
  auto bll = [&](const __amdgpu_buffer_rsrc_t& rs, unsigned lds_addr, int voff, int soff) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_u8*)(size_t)__builtin_amdgcn_readfirstlane(lds_addr), 16,
                                             voff, __builtin_amdgcn_readfirstlane(soff), 0, 0);
  };
  // One tensor's pieces of one chunk into stage st (TK: K, else V).
  auto fetch_one = [&](auto tk, int st, int key0) {
    constexpr bool TK = decltype(tk)::value;
    const __amdgpu_buffer_rsrc_t& rs = TK ? krs : vrs;
    const unsigned base = (TK ? ks_base : vs_base) + st * CT;
    key0 = __builtin_amdgcn_readfirstlane(key0);
    if (key0 + CK <= N) {
#pragma unroll
      for (int v = 0; v < NUW; ++v)
        bll(rs, base + (w * NUW + v) * 1024, TK ? kgv[v] : vgv[v], key0 * D * 2);
    } else {
      // The lane id goes through an empty asm so this rare path's per-lane
      // values are recomputed here rather than hoisted and kept live.
      if (key0 >= N) key0 = 0;
      const int valid = N - key0;
      int ln = lane;
      asm volatile("" : "+v"(ln));
      const int p = ln % G::NCH;
#pragma unroll
      for (int v = 0; v < NUW; ++v) {
        const int u = w * NUW + v;
        const int r = u * G::RPI + ln / G::NCH;
        const int rs_ = r < valid ? r : 0;
        int c = TK ? swz_k<G::NCH>(r, p) : swz_v<G::NCH>(r, p);
        if (c >= G::DCH) c = 0;
        bll(rs, base + u * 1024, (rs_ * D + c * 8) * 2, key0 * D * 2);
      }
    }
  };
  auto fetch_k = [&](int st, int key0) { fetch_one(std::true_type{}, st, key0); };
  auto fetch_v = [&](int st, int key0) { fetch_one(std::false_type{}, st, key0); };
  auto fetch = [&](int st, int key0) {
    fetch_k(st, key0);
    fetch_v(st, key0);
  };

  // Per-lane LDS offsets.  K operand, step s: row l32 of the tile, piece
  // 2s + hf.  V transpose reads: row (kk*16 + hf*4 + n16/4 [+8]), piece
  // dt*4 + (g16&1)*2 + (n16&3)/2; only dt interacts with the swizzle.  The
  // stage and the kk / +8 row offsets are immediates.
  int koff[G::DQ];
#pragma unroll
  for (int s = 0; s < G::DQ; ++s) koff[s] = l32 * G::RB + (swz_k<G::NCH>(l32, 2 * s + hf) << 4);
  int voff[G::DT];
  {
    const int vr = hf * 4 + (n16 >> 2);
#pragma unroll
    for (int dt = 0; dt < G::DT; ++dt) {
      const int c = dt * 4 + (g16 & 1) * 2 + ((n16 & 3) >> 1);
      voff[dt] = vr * G::RB + (swz_v<G::NCH>(vr, c) << 4) + (n16 & 1) * 8;
    }
  }

  float m_ref = 0.0f;        // reference max (log2 units), fixed by the first chunk
  float l_part = 0.0f;       // this lane's half of the row sum
  f32x16 oacc[G::DT];
#pragma unroll
  for (int dt = 0; dt < G::DT; ++dt) oacc[dt] = f32x16{};

  auto qk = [&](f32x16& sacc, const unsigned char* kt) {
    sacc = f32x16{};
#pragma unroll
    for (int s = 0; s < G::DQ; ++s) {
      const bf16x8 kop = *reinterpret_cast<const bf16x8*>(kt + koff[s]);
      sacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kop, qop[s], sacc, 0, 0, 0);
    }
  };
  auto mask_tail = [&](f32x16& sacc, int valid) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int key = (r >> 2) * 8 + hf * 4 + (r & 3);
      if (key >= valid) sacc[r] = -INFINITY;
    }
  };
  auto softmax = [&](const f32x16& sacc, bf16x8 (&pop)[2]) {
    const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
    float lsum = l_part;
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      u32x4 wv;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[kk * 8 + 2 * e], sl2, -m_ref));
        const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[kk * 8 + 2 * e + 1], sl2, -m_ref));
        const bf16x2 pb = cvt2(p0, p1);
        lsum = __builtin_amdgcn_fdot2_f32_bf16(pb, ones, lsum, false);
        wv[e] = __builtin_bit_cast(unsigned, pb);
      }
      pop[kk] = __builtin_bit_cast(bf16x8, wv);
    }
    l_part = lsum;
  };
  auto pv = [&](const bf16x8 (&pop)[2], const unsigned char* vt) {
#pragma unroll
    for (int dt = 0; dt < G::DT; ++dt) {
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
        // rows r and r + 8 have the same swizzle, so one offset serves both
        const unsigned char* p = vt + voff[dt] + kk * 16 * G::RB;
        const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p));
        const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p + 8 * G::RB));
        const u32x2 lw = __builtin_bit_cast(u32x2, lo);
        const u32x2 hw = __builtin_bit_cast(u32x2, hi);
        const u32x4 vw = {lw[0], lw[1], hw[0], hw[1]};
        oacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, vw), pop[kk], oacc[dt], 0, 0, 0);
      }
    }
  };

  // After every kept block: if a row sum has grown past 2^64 (the reference
  // maximum was far below this row's logits), move the reference up by the
  // sum's binary exponent and scale that query's O and l by the same power of
  // two (exact).  p = exp2(s - m) can then only overflow if one block raises
  // the logits by more than ~2^63 over the running sum; that rare case is
  // caught by the final check.  Rows never come near 2^64 in practice, so this
  // is one compare and a branch per block.
  auto rescale_if_large = [&]() {
    if (__builtin_amdgcn_ballot_w64(l_part > 0x1p64f) != 0) {
      asm volatile("");
      const float l_tot = swap_halves_sum(l_part);
      const int e = l_tot > 0x1p64f ? __builtin_amdgcn_frexp_expf(l_tot) : 0;
      const float f = __builtin_amdgcn_ldexpf(1.0f, -e);
      l_part *= f;
#pragma unroll
      for (int dt = 0; dt < G::DT; ++dt)
#pragma unroll
        for (int r = 0; r < 16; ++r) oacc[dt][r] *= f;
      m_ref += (float)e;
    }
  };

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
      if (valid < CK) mask_tail(sacc, valid);
      float mx = sacc[0];                 // chunk 0 holds a valid key: finite
#pragma unroll
      for (int r = 1; r < 16; ++r) mx = fmaxf(mx, sacc[r]);
      m_ref = swap_halves_max(mx) * sl2;
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
        pv(pop, &Vs[c][0]);
        const int nvalid = __builtin_amdgcn_readfirstlane(N - nkey0);
        if (nvalid < CK) {
          asm volatile("");        // keep this a real (rarely taken) branch, not select code
          mask_tail(snext, nvalid);
        }
        sacc = snext;
      }
      rescale_if_large();
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
      if (valid < CK) mask_tail(sacc, valid);
      float mx = sacc[0];                 // chunk 0 holds a valid key: finite
#pragma unroll
      for (int r = 1; r < 16; ++r) mx = fmaxf(mx, sacc[r]);
      m_ref = swap_halves_max(mx) * sl2;
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
          mask_tail(snext, nvalid);
        }
        sacc = snext;
      }
      rescale_if_large();
      advance_block(itnn, jnn);
    }
  }
  wait_vmcnt<0>();           // no load may still target this workgroup's LDS

  // ---- epilogue: overflow check, then O = O^T / l and LSE ----
  if (threadIdx.x == 0) wg_bad = 0;
  const float l_tot = swap_halves_sum(l_part);
  bool bad = !(l_tot < 0x1p100f);
#pragma unroll
  for (int dt = 0; dt < G::DT; ++dt)
#pragma unroll
    for (int r = 0; r < 16; ++r) bad |= !__builtin_isfinite(oacc[dt][r]);
  __syncthreads();
  if (__builtin_amdgcn_ballot_w64(bad) != 0 && lane == 0) atomicOr(&wg_bad, 1);
  __syncthreads();
  if (wg_bad) {
    if (threadIdx.x == 0 && i * S < N) {
      if constexpr (OUT_F32) static_cast<float*>(a.out)[head + (size_t)i * S * D] = __builtin_nanf("");
      else static_cast<uint16_t*>(a.out)[head + (size_t)i * S * D] = 0x7FC0;
    }
    return;
  }
  const bool has = count > 0 && l_tot > 0.0f;
  const float inv = has ? 1.0f / l_tot : 0.0f;
  if (qr < N) {
    const size_t obase = head + (size_t)qr * D;
#pragma unroll
    for (int dt = 0; dt < G::DT; ++dt)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        const int d = dt * 32 + r4 * 8 + hf * 4;
        if (d < D) {
          const float o0 = oacc[dt][r4 * 4 + 0] * inv, o1 = oacc[dt][r4 * 4 + 1] * inv;
          const float o2 = oacc[dt][r4 * 4 + 2] * inv, o3 = oacc[dt][r4 * 4 + 3] * inv;
          if constexpr (OUT_F32) {
            *reinterpret_cast<float4*>(static_cast<float*>(a.out) + obase + d) = make_float4(o0, o1, o2, o3);
          } else {
            const bf16x2 x = cvt2(o0, o1), y = cvt2(o2, o3);
            const bf16x4 o = {x[0], x[1], y[0], y[1]};
            *reinterpret_cast<bf16x4*>(static_cast<uint16_t*>(a.out) + obase + d) = o;
          }
        }
      }
    if (a.lse && hf == 0) {
      a.lse[(size_t)bh * N + qr] = has ? (m_ref + __log2f(l_tot)) * 0.69314718055994530942f : -INFINITY;
    }
  }
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
