// Block-sparse (and dense) flash attention, 64 queries per wave (Section 4.2.2:
// kept blocks computed exactly; Appendix A.2.2: dense FlashAttention fallback).
//
// Layout of the work.  A workgroup is one query block of S tokens with S/64
// waves; each wave owns 64 queries as two 32-query MFMA tiles, so every K or
// V^T operand read from LDS feeds two MFMAs.  That halves LDS bytes per FLOP
// relative to 32 queries per wave (LDS reads run near 128 B/clk/CU on gfx950;
// the b64 transpose read near 72 B/clk/CU).  Keys are processed in 64-key
// chunks.
//
// Memory path.  Each kept block's K and V tiles (S x D bf16) are fetched with
// global_load_lds_dwordx4 straight into LDS (no VGPR staging).  The tiles are
// unpadded with an XOR swizzle on 16-byte chunks: K chunk c of row r sits at
// c ^ (r & 7) (conflict-free for the ds_read_b128 K operand reads); V chunk c
// of row r sits at c ^ 2(r & 7) (conflict-free for the transpose reads, which
// touch 4 consecutive rows x 32 bytes per 16 lanes).  K and V have one buffer
// each and separate waits: the next block's K is fetched while this block's
// softmax and PV run, its V while the next QK runs.
//
// Math per 64-key chunk (lane = one query of each tile; its 16 registers per
// 32-key subtile are keys (r/4)*8 + half*4 + r%4):
//   S^T = K Q^T                 mfma_f32_32x32x16_bf16, Q^T in registers
//   m   = max over keys         v_max3 + one permlane32 swap
//   lazy rescale                the running max moves only if the chunk max
//                               exceeds it by more than 8 (log2 units); then
//                               O and l are rescaled, otherwise p <= 2^8
//   p   = exp2(c*log2e*s - m)   one FMA + v_exp_f32, rounded to bf16
//   l  += sum of the bf16 p     v_dot2 with (1, 1): the sum the MFMA sees
//   O^T += V^T P^T              P^T straight from the S^T registers, V^T via
//                               ds_read_b64_tr_b16 from the row-major tile
// Code order places the softmax of chunk c next to independent MFMAs (QK of
// chunk c+1, PV of chunk c-1) so the scheduler can overlap VALU and MFMA.
#include <type_traits>

#include "attn_common.h"

namespace sva {
namespace {

using namespace attn;

template <int D, int S, bool SPARSE, bool OUT_F32>
__global__ __launch_bounds__(S) __attribute__((amdgpu_waves_per_eu(1, 1)))
void attn_q64_kernel(AttnArgs a) {
  using G = Geo<D>;
  constexpr int NW = S / 64;                 // waves per workgroup
  constexpr int NCK = S / 64;                // 64-key chunks per block
  constexpr int CT = 64 * G::RB;             // bytes of one chunk tile (K or V)
  constexpr int NUW = CT / 1024 / NW;        // direct-load instructions per wave per tile
  static_assert(NCK == 1 || NCK == 2, "block size 64 or 128");

  __shared__ __attribute__((aligned(1024))) unsigned char Ks[2][CT];
  __shared__ __attribute__((aligned(1024))) unsigned char Vs[2][CT];

  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  const int hf = lane >> 5;
  const int l32 = lane & 31;
  const int g16 = lane >> 4;
  const int n16 = lane & 15;
  const int N = a.N, nB = a.nB;
  const float sl2 = a.scale_log2;

  const int row = __builtin_amdgcn_readfirstlane(xcd_remap(blockIdx.x, a.n_rows));  // (b*H + h)*nB + i
  const int bh = row / nB;
  const int i = row - bh * nB;
  const size_t head = (size_t)bh * N * D;
  const uint16_t* Qh = a.q + head;
  const uint16_t* Kh = a.k + head;
  const uint16_t* Vh = a.v + head;

  // ---- Q^T operands: tile t holds queries i*S + w*64 + t*32 + l32 ----
  const int q0 = i * S + w * 64;
  bf16x8 qop[2][G::DQ];
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    const int qr = q0 + t * 32 + l32;
#pragma unroll
    for (int s = 0; s < G::DQ; ++s) {
      if (qr < N) qop[t][s] = *reinterpret_cast<const bf16x8*>(Qh + (size_t)qr * D + s * 16 + hf * 8);
      else qop[t][s] = bf16x8{};
    }
  }

  // index list through the constant address space: uniform reads become
  // scalar loads (lgkmcnt), so they never wait on the in-flight tile loads
  int count;
  const_i32* idxrow = nullptr;
  if constexpr (SPARSE) {
    count = __builtin_amdgcn_readfirstlane(min(max(((const_i32*)a.kv_count)[row], 0), a.kmax));
    idxrow = (const_i32*)a.kv_idx + (size_t)row * a.kmax;
  } else {
    count = nB;
  }
  auto block_at = [&](int it) -> int {
    return __builtin_amdgcn_readfirstlane(SPARSE ? idxrow[it] : it);
  };
  auto next_valid = [&](int it) -> int {
    while (it < count) {
      const int j = block_at(it);
      if (j >= 0 && j < nB) break;
      ++it;
    }
    return it;
  };
  // position in the flattened (kept block, 64-key chunk) sequence; chunks that
  // lie wholly past the end of the sequence are skipped
  struct Pos { int it, ch, key0; };
  auto make = [&](int it, int ch) -> Pos {
    return Pos{it, ch, it < count ? block_at(it) * S + ch * 64 : 0};
  };
  auto advance = [&](const Pos& p) -> Pos {
    if (NCK == 2 && p.ch == 0 && p.key0 + 64 < N) return make(p.it, 1);
    return make(next_valid(p.it + 1), 0);
  };

  // ---- direct global -> LDS fetch of one chunk (this wave's 1 KB pieces) ----
  // Piece u covers LDS rows u*RPI .. u*RPI + RPI - 1; lane L fills row
  // u*RPI + L/NCH at position L % NCH, i.e. global chunk (L % NCH) ^ swizzle(row).
  // The swizzle depends on the row only through (row & 7), which for a given
  // lane depends on u only through its parity (RPI = 4) or not at all (RPI = 8),
  // so two per-lane byte offsets per tensor serve every full chunk; the uniform
  // part (chunk start + u * RPI rows) is the scalar offset of buffer_load ... lds.
  // Every address formed here lies inside the head's K or V rows (full chunks
  // by construction, the last chunk by clamping), so nothing relies on the
  // descriptor's range check.
  const __amdgpu_buffer_rsrc_t krs = __builtin_amdgcn_make_buffer_rsrc((void*)Kh, (short)0, N * D * 2, 0x00020000);
  const __amdgpu_buffer_rsrc_t vrs = __builtin_amdgcn_make_buffer_rsrc((void*)Vh, (short)0, N * D * 2, 0x00020000);
  int kgo[2], vgo[2];
  {
    const int p = lane % G::NCH;
    const int rl = lane / G::NCH;
#pragma unroll
    for (int par = 0; par < 2; ++par) {
      const int r = par * G::RPI + rl;
      int ck = swz_k(r, p), cv = swz_v<G::NCH>(r, p);   // the swizzle is an involution
      if (ck >= G::DCH) ck = 0;                          // padding chunks: any in-row address
      if (cv >= G::DCH) cv = 0;
      kgo[par] = (rl * D + ck * 8) * 2;
      vgo[par] = (rl * D + cv * 8) * 2;
    }
  }
  // both the LDS destination (M0) and the scalar offset are wave-uniform; say so
  auto bll = [&](const __amdgpu_buffer_rsrc_t& rs, unsigned char* dst, int voff, int soff) {
    typedef __attribute__((address_space(3))) void lds_void;
    const unsigned la = __builtin_amdgcn_readfirstlane((unsigned)(size_t)(lds_void*)dst);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void*)(size_t)la, 16, voff,
                                             __builtin_amdgcn_readfirstlane(soff), 0, 0);
  };
  auto fetch = [&](int st, int key0) {
    st = __builtin_amdgcn_readfirstlane(st);
    key0 = __builtin_amdgcn_readfirstlane(key0);
    const int base = key0 * D * 2;
    const int valid = N - key0;
    if (valid >= 64) {
#pragma unroll
      for (int v = 0; v < NUW; ++v) {
        const int u = w * NUW + v;
        bll(krs, &Ks[st][u * 1024], kgo[u & 1], base + u * G::RPI * D * 2);
      }
#pragma unroll
      for (int v = 0; v < NUW; ++v) {
        const int u = w * NUW + v;
        bll(vrs, &Vs[st][u * 1024], vgo[u & 1], base + u * G::RPI * D * 2);
      }
    } else {
      // last, partial chunk: rows past the sequence read row 0 of the chunk
      // (finite data; those keys are masked out of the softmax).  The lane id
      // goes through an empty asm so this rare path's per-lane values are
      // recomputed here rather than hoisted (and kept live) across the loop.
      int ln = lane;
      asm volatile("" : "+v"(ln));
      const int p = ln % G::NCH;
#pragma unroll
      for (int v = 0; v < NUW; ++v) {
        const int u = w * NUW + v;
        const int r = u * G::RPI + ln / G::NCH;
        const int rs = r < valid ? r : 0;
        int ck = swz_k(r, p), cv = swz_v<G::NCH>(r, p);
        if (ck >= G::DCH) ck = 0;
        if (cv >= G::DCH) cv = 0;
        bll(krs, &Ks[st][u * 1024], (rs * D + ck * 8) * 2, base);
        bll(vrs, &Vs[st][u * 1024], (rs * D + cv * 8) * 2, base);
      }
    }
  };

  // ---- per-lane softmax state for its two queries ----
  // m_ref: the reference maximum, fixed from the first chunk this workgroup
  // processes and never moved afterwards, so O is never rescaled in the loop.
  float m_ref[2] = {0.0f, 0.0f};
  float l_part[2] = {0.0f, 0.0f};
  f32x16 oacc[2][G::DT];
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int dt = 0; dt < G::DT; ++dt) oacc[t][dt] = f32x16{};

  // Per-lane LDS offsets.  K operand, step s: row (sc*32 + l32), chunk 2s + hf
  // at position (2s + hf) ^ (l32 & 7); positions of steps s and s + 4 differ by
  // exactly 8 chunks, so four offsets cover all steps and the rest is an
  // immediate.  V transpose reads: row (sc*32 + kk*16 + hf*4 + n16/4 [+8]),
  // chunk dt*4 + (g16&1)*2 + (n16&3)/2; only dt interacts with the swizzle.
  int koff[4];
#pragma unroll
  for (int s = 0; s < 4; ++s) koff[s] = l32 * G::RB + (swz_k(l32, 2 * s + hf) << 4);
  int voff[G::DT];
  {
    const int vr = hf * 4 + (n16 >> 2);
#pragma unroll
    for (int dt = 0; dt < G::DT; ++dt) {
      const int c = dt * 4 + (g16 & 1) * 2 + ((n16 & 3) >> 1);
      voff[dt] = vr * G::RB + (swz_v<G::NCH>(vr, c) << 4) + (n16 & 1) * 8;
    }
  }

  // S^T of one 32-key sub-chunk sc (keys sc*32 + row-of-C), both query tiles
  auto qk = [&](f32x16 (&sacc)[2], const unsigned char* kt, int sc) {
    sacc[0] = f32x16{};
    sacc[1] = f32x16{};
#pragma unroll
    for (int s = 0; s < G::DQ; ++s) {
      const bf16x8 kop = *reinterpret_cast<const bf16x8*>(kt + koff[s & 3] + (s >> 2) * 128 + sc * 32 * G::RB);
#pragma unroll
      for (int t = 0; t < 2; ++t)
        sacc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kop, qop[t][s], sacc[t], 0, 0, 0);
    }
  };

  // keys at or past `valid` (within the chunk) get -inf before the softmax
  auto mask_tail = [&](f32x16 (&sacc)[2], int sc, int valid) {
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = sc * 32 + (r >> 2) * 8 + hf * 4 + (r & 3);
        if (key >= valid) sacc[t][r] = -INFINITY;
      }
  };

  // max over this lane's query of both sub-chunks (first chunk only)
  auto set_reference = [&](const f32x16 (&sa)[2], const f32x16 (&sb)[2]) {
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      float mx = fmaxf(sa[t][0], sb[t][0]);
#pragma unroll
      for (int r = 1; r < 16; ++r) mx = fmaxf(mx, fmaxf(sa[t][r], sb[t][r]));
      mx = swap_halves_max(mx) * sl2;
      // the first chunk holds at least one valid key, so mx is finite
      m_ref[t] = mx;
    }
  };

  // p = exp2(c*log2e*s - m_ref) rounded to bf16 -> P operands pop[t][kk]
  // (two 16-key MFMA steps); the row sum adds exactly the bf16 values
  auto softmax = [&](const f32x16 (&sacc)[2], bf16x8 (&pop)[2][2]) {
    const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      float lsum = l_part[t];
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
        // the operand is built as four packed dwords so each v_cvt_pk_bf16_f32
        // can write its final register directly
        u32x4 w;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[t][kk * 8 + 2 * e], sl2, -m_ref[t]));
          const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[t][kk * 8 + 2 * e + 1], sl2, -m_ref[t]));
          const bf16x2 pb = cvt2(p0, p1);
          lsum = __builtin_amdgcn_fdot2_f32_bf16(pb, ones, lsum, false);
          w[e] = __builtin_bit_cast(unsigned, pb);
        }
        pop[t][kk] = __builtin_bit_cast(bf16x8, w);
      }
      l_part[t] = lsum;
    }
  };

  // O^T += V^T P^T for one 32-key sub-chunk
  auto pv = [&](const bf16x8 (&pop)[2][2], const unsigned char* vt, int sc) {
#pragma unroll
    for (int dt = 0; dt < G::DT; ++dt) {
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
        // rows r and r + 8 share (r & 7), hence the swizzle
        const unsigned char* p = vt + voff[dt] + (sc * 32 + kk * 16) * G::RB;
        const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p));
        const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p + 8 * G::RB));
        const u32x2 lw = __builtin_bit_cast(u32x2, lo);
        const u32x2 hw = __builtin_bit_cast(u32x2, hi);
        const u32x4 vw = {lw[0], lw[1], hw[0], hw[1]};
        const bf16x8 vop = __builtin_bit_cast(bf16x8, vw);
#pragma unroll
        for (int t = 0; t < 2; ++t)
          oacc[t][dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vop, pop[t][kk], oacc[t][dt], 0, 0, 0);
      }
    }
  };

  // one 64-key chunk: QK of both sub-chunks, the softmax of sub-chunk a next
  // to nothing dependent, PV(a) beside the softmax of b, then PV(b)
  auto chunk = [&](const unsigned char* kt, const unsigned char* vt, int valid, bool first,
                   auto tail) {
    f32x16 sa[2], sb[2];
    bf16x8 pa[2][2], pb[2][2];
    qk(sa, kt, 0);
    qk(sb, kt, 1);
    if constexpr (decltype(tail)::value) {
      mask_tail(sa, 0, valid);
      mask_tail(sb, 1, valid);
    }
    if (first) set_reference(sa, sb);
    softmax(sa, pa);
    pv(pa, vt, 0);
    softmax(sb, pb);
    pv(pb, vt, 1);
  };

  Pos cur = make(next_valid(0), 0);
  if (cur.it < count) fetch(0, cur.key0);
  int st = 0;
  bool first = true;
  while (cur.it < count) {
    const Pos nxt = advance(cur);
    const bool more = nxt.it < count;
    if (more) {
      fetch(st ^ 1, nxt.key0);   // that stage was released by the last iteration's barrier
      wait_vmcnt<2 * NUW>();     // this chunk landed; the next one may still be in flight
    } else {
      wait_vmcnt<0>();
    }
    wg_barrier();
    st = __builtin_amdgcn_readfirstlane(st);
    const int valid = __builtin_amdgcn_readfirstlane(N - cur.key0);
    if (valid >= 64) chunk(Ks[st], Vs[st], valid, first, std::false_type{});
    else chunk(Ks[st], Vs[st], valid, first, std::true_type{});
    first = false;
    wg_barrier();                // every wave is done with this stage
    st ^= 1;
    cur = nxt;
  }

  // ---- epilogue: O = O^T / l, LSE ----
  // With the reference max fixed from the first chunk, p = 2^(x - m_ref) may
  // exceed 1 for later keys.  That is exact in fp32/bf16 unless the logits grow
  // by ~100 (log2 units) past the first chunk's maximum.  If any row sum
  // reaches 2^100 or any accumulator is not finite, the whole query block is
  // marked with a NaN in its first output element and left for the
  // rescaling kernel that runs next on the same stream.
  __shared__ int wg_bad;
  if (threadIdx.x == 0) wg_bad = 0;
  // O is read out of the accumulation registers (AGPRs) explicitly: with every
  // use of O being an MFMA or this read, O stays in AGPRs for the whole loop
  // instead of being copied in and out around each PV step.
  float ov[2][G::DT][16];
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int dt = 0; dt < G::DT; ++dt)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        asm volatile("v_accvgpr_read_b32 %0, %1" : "=v"(ov[t][dt][r]) : "a"(oacc[t][dt][r]));
  float l_tot[2];
  bool bad = false;
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    l_tot[t] = swap_halves_sum(l_part[t]);
    bad |= !(l_tot[t] < 0x1p100f);
#pragma unroll
    for (int dt = 0; dt < G::DT; ++dt)
#pragma unroll
      for (int r = 0; r < 16; ++r) bad |= !__builtin_isfinite(ov[t][dt][r]);
  }
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
  const bool has_keys = count > 0;
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    const float inv = (has_keys && l_tot[t] > 0.0f) ? 1.0f / l_tot[t] : 0.0f;
    const int qr = q0 + t * 32 + l32;
    if (qr < N) {
      const size_t obase = head + (size_t)qr * D;
#pragma unroll
      for (int dt = 0; dt < G::DT; ++dt)
#pragma unroll
        for (int r4 = 0; r4 < 4; ++r4) {
          const int d = dt * 32 + r4 * 8 + hf * 4;
          if (d < D) {
            const float o0 = ov[t][dt][r4 * 4 + 0] * inv, o1 = ov[t][dt][r4 * 4 + 1] * inv;
            const float o2 = ov[t][dt][r4 * 4 + 2] * inv, o3 = ov[t][dt][r4 * 4 + 3] * inv;
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
        a.lse[(size_t)bh * N + qr] = (has_keys && l_tot[t] > 0.0f)
                                         ? (m_ref[t] + __log2f(l_tot[t])) * 0.69314718055994530942f
                                         : -INFINITY;
      }
    }
  }
}

template <int D, int S>
hipError_t launch_q64(const Dims& d, bool sparse, const AttnArgs& a, hipStream_t stream) {
  dim3 grid(a.n_rows), block(S);
  if (sparse) {
    if (d.out_f32) hipLaunchKernelGGL((attn_q64_kernel<D, S, true, true>), grid, block, 0, stream, a);
    else hipLaunchKernelGGL((attn_q64_kernel<D, S, true, false>), grid, block, 0, stream, a);
  } else {
    if (d.out_f32) hipLaunchKernelGGL((attn_q64_kernel<D, S, false, true>), grid, block, 0, stream, a);
    else hipLaunchKernelGGL((attn_q64_kernel<D, S, false, false>), grid, block, 0, stream, a);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attention_q64(const Dims& d, bool sparse, const AttnArgs& a, hipStream_t stream) {
  switch (d.D * 1000 + d.S) {
    case 64128: return launch_q64<64, 128>(d, sparse, a, stream);
    case 112128: return launch_q64<112, 128>(d, sparse, a, stream);
    case 128128: return launch_q64<128, 128>(d, sparse, a, stream);
    case 64064: return launch_q64<64, 64>(d, sparse, a, stream);
    case 112064: return launch_q64<112, 64>(d, sparse, a, stream);
    case 128064: return launch_q64<128, 64>(d, sparse, a, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace sva
