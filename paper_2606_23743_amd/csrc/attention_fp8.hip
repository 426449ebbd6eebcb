// 8-bit (fp8 e4m3) block-sparse attention (Section 4.2.4 points to 8-bit
// attention with outlier smoothing; Section 4.2.2 / Appendix A.2.2 the
// block-sparse pattern it runs under).  Inputs come from the fp8 quantiser:
// Q and K codes [B, H, Np, DP] with one power-of-two exponent per block, V
// codes in 64-key tiles [B, H, Np/64, DP, 64] with one exponent per channel
// (DP = D rounded up to a multiple of 64; the padding channels are zero and
// are not written out).
//
// A workgroup is one query block of S tokens, S/32 waves of 32 queries (one
// query per lane pair, as in the bf16 kernel).  Keys go in 64-key chunks, one
// PV matrix instruction each:
//   S^T = K Q^T   mfma_scale_f32_32x32x64_f8f6f4, two 32-key tiles, the block
//                 exponents of K and Q applied by the instruction's scales.
//                 Q carries the softmax scale in base 2 (the quantiser folds
//                 c*log2(e) into it), so s is the logit in base-2 units.
//                 K rows are read in the order pi(r) = 16*((r>>2)&1) +
//                 4*(r>>3) + (r&3), so register j of tile t of lane (n, h) is
//                 key 32t + 16h + j: the lane's 32 probabilities are two runs
//                 of 16 consecutive keys.
//   p = exp2(s - m + 6)   with m the floor of the first chunk's row maximum,
//                 moved up to the floor of a chunk's maximum (O and l scaled
//                 by the power of two, exactly) before any chunk whose maximum
//                 exceeds it by more than 2.75.  m is an integer, so the
//                 offset rides on the conversion: exp2(s) is converted with
//                 v_cvt_scalef32_pk_fp8_f32, which divides by the power of two
//                 2^(m - 6) before rounding, and no per-element subtraction is
//                 needed.  (A wave with a row whose |m| exceeds 100, where
//                 exp2(s) could leave float32's range, subtracts instead.)
//                 So p <= 2^8.75 < 448 fits e4m3, and the offset puts
//                 the weights near the maximum high in e4m3's range: only
//                 weights below 2^-16 of the maximum fall under its smallest
//                 subnormal (with no offset every weight below 2^-10 would
//                 vanish, a one-sided error that grows with the number of
//                 keys).  Offsets of 5 to 8 (guards 3.75 to 0.5) measured within
//                 2% of each other; larger guards rescale less often.  p is
//                 converted to e4m3 (round to nearest even).
//   O^T += V^T P^T  the same instruction, V^T rows (channels) read straight
//                 from the d-major tile, the channel exponents applied as the
//                 per-row scales.
//   l  += 1^T P^T   one more instruction with an all-ones operand: l is exactly
//                 the sum of the e4m3 weights the PV product applied.
// Chunks stream through four LDS stages (K and V tiles of 64 x D bytes)
// filled three chunks ahead by buffer_load ... lds (two stages, K two chunks
// and V one chunk ahead, at D = 128 with S = 64); the stage is the chunk
// counter mod the stage count.  Each wave overlaps the next chunk's S^T with the current
// chunk's softmax and PV, as in the bf16 kernel.  The kept-block list is
// compacted into LDS at the start (entries outside [0, nB) dropped), packed
// with each block's K exponent.
#include "attn_common.h"

namespace sva {
namespace {

using namespace attn;

typedef __attribute__((ext_vector_type(8))) int i32x8;
typedef __attribute__((ext_vector_type(4))) int i32x4;
typedef __attribute__((ext_vector_type(2))) short s16x2;

constexpr int kListSlots = kFp8MaxList + 1;  // LDS list entries; the last slot holds the count
constexpr int kShift = 6;                // log2 offset of the probabilities (see above)
constexpr float kGuard = 2.75f;          // allowed excess of a chunk maximum over m
constexpr float kFastRange = 100.0f;     // |m| up to this: exp2(s) stays normal float32

__device__ __forceinline__ int pi_row(int r) { return 16 * ((r >> 2) & 1) + 4 * (r >> 3) + (r & 3); }

// LDS slot of 16-byte piece p of K tile row q (row = key); D/16 pieces per row.
// 16 lanes of a b128 read take rows pi(r) for 16 consecutive r: the XOR makes
// their (row parity, slot) pairs distinct, i.e. all 64 banks.
template <int D>
__device__ __forceinline__ int k_slot(int q, int p) {
  if constexpr (D == 128) return p ^ (((q >> 1) & 3) | (((q >> 4) & 1) << 2));
  else return p ^ (((q >> 2) & 1) | (((q >> 4) & 1) << 1));
}
// LDS slot of piece p (of 4) of V tile row d (row = channel, 64 keys).
__device__ __forceinline__ int v_slot(int d, int p) { return p ^ ((d >> 2) & 3); }

template <int D, int S, bool SPARSE, bool OUT_F32>
__global__ __launch_bounds__(2 * S) __attribute__((amdgpu_waves_per_eu(2, 2)))
void attn_fp8_kernel(Fp8AttnArgs a) {
  constexpr int DP = (D + 63) / 64 * 64;     // code channels (D = 112: 128, the last 16 zero)
  constexpr int NW = S / 32;                 // waves per workgroup
  constexpr int CK = 64;                     // keys per chunk
  constexpr int NCK = S / CK;                // chunks per block
  // LDS stages: four (loads three chunks ahead), or two at D = 128, S = 64 so
  // that four two-wave workgroups (two waves per SIMD) fit a CU's 160 KB
  constexpr int NST = (DP == 128 && S == 64) ? 2 : 4;
  constexpr int TB = CK * DP;                // bytes of one K (or V) tile
  constexpr int NPC = DP / 16;               // 16-byte pieces per K row
  constexpr int NUK = TB / 1024 / NW;        // direct-load pieces per wave per tile
  constexpr int DQ = DP / 64;                // k-steps of S^T
  constexpr int DT = DP / 32;                // 32-channel tiles of O^T
  constexpr int GL = 2 * NUK;                // loads per wave per chunk
  static_assert(NUK >= 1, "tile split");

  __shared__ __attribute__((aligned(1024))) unsigned char Ks[NST][TB];
  __shared__ __attribute__((aligned(1024))) unsigned char Vs[NST][TB];
  __shared__ int list[kListSlots];           // (block << 8) | (K exponent + 127); count last

  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int hf = lane >> 5;
  const int l32 = lane & 31;
  const int N = a.N, nB = a.nB, Np = a.Np;

  // workgroup order as in the bf16 kernel: sparse lists in frame tiles of 4
  // query blocks x 8 frames inside a head, at S = 128 also in segments of
  // 8 x 128 rows (the eight XCDs on one head at a time)
  constexpr bool kSegments = SPARSE && S == 128;
  const int wg = kSegments ? xcd_remap_segments(blockIdx.x, a.n_rows, 128) : xcd_remap(blockIdx.x, a.n_rows);
  const int rowl = __builtin_amdgcn_readfirstlane(wg);   // (b*H + h)*nB + logical block
  const int bh = rowl / nB;
  const int i = SPARSE ? frame_tile_order(rowl - bh * nB, nB, a.frame_blocks, 8, 4) : rowl - bh * nB;
  const int row = bh * nB + i;
  const size_t head = (size_t)bh * Np * DP;

  // ---- the block list: compacted, with each block's K exponent ----
  if constexpr (SPARSE) {
    if (w == 0) {
      const int count = min(max(a.kv_count[row], 0), a.kmax);
      const int32_t* idx = a.kv_idx + (size_t)row * a.kmax;
      int n = 0;
      for (int t0 = 0; t0 < count; t0 += 64) {
        const int t = t0 + lane;
        const int j = t < count ? idx[t] : -1;
        const bool ok = j >= 0 && j < nB;
        const unsigned long long m = __builtin_amdgcn_ballot_w64(ok);
        const int pos = n + __builtin_amdgcn_mbcnt_hi((unsigned)(m >> 32), __builtin_amdgcn_mbcnt_lo((unsigned)m, 0));
        if (ok && pos < kFp8MaxList) list[pos] = (j << 8) | (a.k_exp[(size_t)bh * nB + j] + 127);
        n += __builtin_popcountll(m);
      }
      if (lane == 0) list[kFp8MaxList] = min(n, kFp8MaxList);
    }
  } else {
    for (int t = threadIdx.x; t < nB; t += 2 * S) list[t] = (t << 8) | (a.k_exp[(size_t)bh * nB + t] + 127);
    if (threadIdx.x == 0) list[kFp8MaxList] = nB;
  }
  __syncthreads();
  const int nblk = list[kFp8MaxList];
  const int G = nblk * NCK;                  // chunks to process
  auto entry = [&](int g) -> int {           // list entry of chunk g (block 0 past the end)
    return g < G ? list[g / NCK] : 127;
  };

  // ---- Q^T operand: query i*S + w*32 + l32; per k-step two 16-byte runs ----
  const int qr = i * S + w * 32 + l32;       // < Np: padded rows are zero codes
  const uint8_t* Qh = a.q8 + head;
  i32x8 qop[DQ];
#pragma unroll
  for (int s = 0; s < DQ; ++s) {
    const i32x4 lo = *reinterpret_cast<const i32x4*>(Qh + (size_t)qr * DP + s * 64 + hf * 16);
    const i32x4 hi = *reinterpret_cast<const i32x4*>(Qh + (size_t)qr * DP + s * 64 + 32 + hf * 16);
    qop[s] = i32x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  }
  const int q_scale = a.q_exp[row] + 127;
  int v_scale[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) v_scale[dt] = a.v_exp[(size_t)bh * DP + dt * 32 + l32] + 127;

  // ---- direct global -> LDS fetch of one chunk (this wave's 1 KB pieces) ----
  // K piece u: rows u*RPK .. (RPK = 1024/D), lane L -> row u*RPK + L/NPC, slot
  // L%NPC, holding global piece k_slot(row, L%NPC).  V piece u: channels
  // u*16 .. u*16+15, lane L -> channel u*16 + L/4, slot L%4.  Both tiles of the
  // chunk starting at key key0 begin at byte key0*D of their head.
  constexpr int RPK = 1024 / DP;
  const __amdgpu_buffer_rsrc_t krs = __builtin_amdgcn_make_buffer_rsrc((void*)(a.k8 + head), (short)0, Np * DP, 0x00020000);
  const __amdgpu_buffer_rsrc_t vrs = __builtin_amdgcn_make_buffer_rsrc((void*)(a.v8 + head), (short)0, Np * DP, 0x00020000);
  int kgv[NUK], vgv[NUK];
#pragma unroll
  for (int v = 0; v < NUK; ++v) {
    const int u = w * NUK + v;
    const int kr = u * RPK + lane / NPC;
    kgv[v] = kr * DP + k_slot<DP>(kr, lane % NPC) * 16;
    const int vd = u * 16 + lane / 4;
    vgv[v] = vd * CK + v_slot(vd, lane % 4) * 16;
  }
  typedef __attribute__((address_space(3))) unsigned char lds_u8;
  const unsigned ks_base = __builtin_amdgcn_readfirstlane((unsigned)(size_t)(lds_u8*)&Ks[0][0]);
  const unsigned vs_base = __builtin_amdgcn_readfirstlane((unsigned)(size_t)(lds_u8*)&Vs[0][0]);
  // (the load goes through this helper: written inline in fetch_chunk, the
  // host compilation pass dropped the kernel's launch stub)
  auto bll = [&](const __amdgpu_buffer_rsrc_t& rs, unsigned lds_addr, int voff, int soff) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_u8*)(size_t)__builtin_amdgcn_readfirstlane(lds_addr), 16,
                                             voff, __builtin_amdgcn_readfirstlane(soff), 0, 0);
  };
  // K (tk) or V of chunk g (list entry e) into stage g % NST
  auto fetch_half = [&](bool tk, int g, int e) {
    e = __builtin_amdgcn_readfirstlane(e);
    const int key0 = __builtin_amdgcn_readfirstlane((e >> 8) * S + (g < G ? (g % NCK) * CK : 0));
    const int st = g & (NST - 1);
#pragma unroll
    for (int v = 0; v < NUK; ++v) {
      if (tk) bll(krs, ks_base + st * TB + (w * NUK + v) * 1024, kgv[v], key0 * DP);
      else bll(vrs, vs_base + st * TB + (w * NUK + v) * 1024, vgv[v], key0 * DP);
    }
  };
  auto fetch_chunk = [&](int g, int e) {
    fetch_half(true, g, e);
    fetch_half(false, g, e);
  };

  // per-lane LDS read offsets (the stage and the tile/row offsets are added)
  int koff[DQ][2];
#pragma unroll
  for (int s = 0; s < DQ; ++s) {
    const int q = pi_row(l32);
    koff[s][0] = q * DP + k_slot<DP>(q, s * 4 + hf) * 16;
    koff[s][1] = q * DP + k_slot<DP>(q, s * 4 + 2 + hf) * 16;
  }
  const int voff0 = l32 * CK + v_slot(l32, hf) * 16;        // channel l32 (+32*dt: same slot pattern)
  const int voff1 = l32 * CK + v_slot(l32, 2 + hf) * 16;

  float m_ref = 0.0f;                        // reference max (log2 units, an integer)
  float cvt_scale = 1.0f;                    // 2^(m_ref - kShift): the conversion divides by it
  bool fast = true;                          // every row of the wave has |m_ref| <= kFastRange
  auto set_ref = [&](float m) {
    m_ref = m;
    // (clamped: a row beyond the fast range never uses its scale)
    cvt_scale = __builtin_amdgcn_ldexpf(1.0f, (int)__builtin_fminf(__builtin_fmaxf(m, -120.0f), 120.0f) - kShift);
    fast = __builtin_amdgcn_ballot_w64(!(__builtin_fabsf(m) <= kFastRange)) == 0;
  };
  f32x16 oacc[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) oacc[dt] = f32x16{};
  f32x16 lacc = f32x16{};
  const i32x8 ones = {0x38383838, 0x38383838, 0x38383838, 0x38383838,
                      0x38383838, 0x38383838, 0x38383838, 0x38383838};   // e4m3 1.0

  auto qk = [&](f32x16 (&sc)[2], int st, int kscale) {
    const unsigned char* kt = &Ks[0][0] + st * TB;
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      sc[t] = f32x16{};
#pragma unroll
      for (int s = 0; s < DQ; ++s) {
        const i32x4 lo = *reinterpret_cast<const i32x4*>(kt + koff[s][0] + t * 32 * DP);
        const i32x4 hi = *reinterpret_cast<const i32x4*>(kt + koff[s][1] + t * 32 * DP);
        const i32x8 kop = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
        sc[t] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(kop, qop[s], sc[t], 0, 0, 0, kscale, 0, q_scale);
      }
    }
  };
  auto mask_tail = [&](f32x16 (&sc)[2], int valid) {     // keys >= valid of the chunk
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        if (32 * t + 16 * hf + r >= valid) sc[t][r] = -INFINITY;
  };
  // Row maximum of a chunk.  The logits are never NaN (finite or -inf), so the
  // maxima are taken with v_max3_f32 directly: fmaxf would first canonicalise
  // every operand, tripling the instruction count of this per-chunk step.
  auto max3 = [](float a, float b, float c) -> float {
    float r;
    asm("v_max3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
    return r;
  };
  auto row_max = [&](const f32x16 (&sc)[2]) -> float {
    float mx = max3(sc[0][0], sc[0][1], sc[0][2]);
#pragma unroll
    for (int r = 3; r < 15; r += 2) mx = max3(mx, sc[0][r], sc[0][r + 1]);
    mx = max3(mx, sc[0][15], sc[1][0]);
#pragma unroll
    for (int r = 1; r < 15; r += 2) mx = max3(mx, sc[1][r], sc[1][r + 1]);
    mx = max3(mx, sc[1][15], sc[1][15]);
    // both halves of the row: lanes l and l ^ 32
    const u32x2 sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx), false, false);
    return max3(__uint_as_float(sw[0]), __uint_as_float(sw[1]), __uint_as_float(sw[1]));
  };
  // before a chunk's probabilities: keep p = exp2(s - m_ref + kShift) <= 2^(kShift + kGuard)
  auto guard = [&](const f32x16 (&sc)[2]) {
    const float over = row_max(sc) - m_ref;
    if (__builtin_amdgcn_ballot_w64(over > kGuard) != 0) {
      asm volatile("");
      const float mn = over > kGuard ? __builtin_floorf(m_ref + over) : m_ref;
      // exact power of two (below 2^-256 it is zero, as exp2 would give)
      const float f = __builtin_amdgcn_ldexpf(1.0f, (int)__builtin_fmaxf(m_ref - mn, -256.0f));
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int r = 0; r < 16; ++r) oacc[dt][r] *= f;
#pragma unroll
      for (int r = 0; r < 16; ++r) lacc[r] *= f;
      set_ref(mn);
    }
  };
  // e4m3 weights of a chunk.  Fast form: exp2(s), divided by 2^(m_ref - kShift)
  // inside the conversion.  Otherwise exp2(s - m_ref + kShift), converted.
  // The first conversion's other half is overwritten by the second, so any
  // register serves as its old value: one of its own inputs, so that no move
  // is needed.
  auto softmax = [&](const f32x16 (&sc)[2], i32x8& pop) {
    if (fast) {
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float p0 = __builtin_amdgcn_exp2f(sc[t][4 * e + 0]);
          const float p1 = __builtin_amdgcn_exp2f(sc[t][4 * e + 1]);
          const float p2 = __builtin_amdgcn_exp2f(sc[t][4 * e + 2]);
          const float p3 = __builtin_amdgcn_exp2f(sc[t][4 * e + 3]);
          s16x2 wv = __builtin_bit_cast(s16x2, __float_as_uint(p0));
          wv = __builtin_amdgcn_cvt_scalef32_pk_fp8_f32(wv, p0, p1, cvt_scale, false);
          wv = __builtin_amdgcn_cvt_scalef32_pk_fp8_f32(wv, p2, p3, cvt_scale, true);
          pop[4 * t + e] = __builtin_bit_cast(int, wv);
        }
    } else {
      const float off = (float)kShift - m_ref;
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float p0 = __builtin_amdgcn_exp2f(sc[t][4 * e + 0] + off);
          const float p1 = __builtin_amdgcn_exp2f(sc[t][4 * e + 1] + off);
          const float p2 = __builtin_amdgcn_exp2f(sc[t][4 * e + 2] + off);
          const float p3 = __builtin_amdgcn_exp2f(sc[t][4 * e + 3] + off);
          int wv = __builtin_amdgcn_cvt_pk_fp8_f32(p0, p1, (int)__float_as_uint(p2), false);
          wv = __builtin_amdgcn_cvt_pk_fp8_f32(p2, p3, wv, true);
          pop[4 * t + e] = wv;
        }
    }
  };
  auto pv = [&](const i32x8& pop, int st) {
    const unsigned char* vt = &Vs[0][0] + st * TB;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
      const i32x4 lo = *reinterpret_cast<const i32x4*>(vt + voff0 + dt * 32 * CK);
      const i32x4 hi = *reinterpret_cast<const i32x4*>(vt + voff1 + dt * 32 * CK);
      const i32x8 vop = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
      oacc[dt] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(vop, pop, oacc[dt], 0, 0, 0, v_scale[dt], 0, 127);
    }
    lacc = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(ones, pop, lacc, 0, 0, 0, 127, 0, 127);
  };

  // ---- pipeline over chunks: chunk g in stage g % 4, loads three ahead ----
  // At iteration g the wave needs K of chunk g+1 and V of chunk g.  After the
  // barrier of iteration g, chunk g-1's stage is free (its K was read at
  // iteration g-2, its V at g-1) and receives chunk g+3.  Every iteration
  // issues one load group (past the end: block 0's first chunk, in bounds),
  // so the wait count is a constant.
  // The loop body is written twice (chunks g and g+1) so the S^T tiles of the
  // current and next chunk swap roles without register copies.  The list
  // entries a chunk step needs are read from LDS one step earlier, so their
  // latency is hidden.
  if (G > 0) {
    f32x16 sa[2], sb[2];
    if constexpr (NST == 4) {
      fetch_chunk(0, entry(0));
      fetch_chunk(1, entry(1));
      fetch_chunk(2, entry(2));
      wait_vmcnt<2 * GL>();
    } else {
      fetch_chunk(0, entry(0));
      fetch_half(true, 1, entry(1));
      wait_vmcnt<0>();
    }
    wg_barrier();
    {
      const int e0 = __builtin_amdgcn_readfirstlane(entry(0));
      qk(sa, 0, e0 & 255);
      const int valid = __builtin_amdgcn_readfirstlane(N - (e0 >> 8) * S);
      if (valid < CK) mask_tail(sa, valid);
      set_ref(__builtin_floorf(row_max(sa)));   // chunk 0 of a block holds a valid key
    }
    // Four stages: after the barrier of step g, chunk g-1's stage is free (its
    // K was read at step g-2, its V at g-1) and receives chunk g+3; the wait is
    // for chunk g+1.  Two stages: K stage g (read by the S^T of step g-1)
    // receives K of chunk g+2 and V stage g+1 (read by the PV of step g-1)
    // receives V of chunk g+1; every load of the previous step is waited for.
    // Each step issues the same loads (past the end: block 0, in bounds), so
    // the wait counts are constants.
    int ent1 = entry(1), ent2 = entry(2), ent3 = entry(3);
    auto step = [&](int g, f32x16 (&scur)[2], f32x16 (&snxt)[2]) {
      if constexpr (NST == 4) {
        wait_vmcnt_lds_idle<GL>();           // chunk g+1 landed, this wave's LDS reads done
        wg_barrier();
        fetch_chunk(g + 3, ent3);
      } else {
        wait_vmcnt_lds_idle<0>();            // K of chunk g+1 and V of chunk g landed
        wg_barrier();
        fetch_half(true, g + 2, ent2);
        fetch_half(false, g + 1, ent1);
      }
      const int e1 = __builtin_amdgcn_readfirstlane(ent1);
      ent1 = entry(g + 2);
      ent2 = entry(g + 3);
      ent3 = entry(g + 4);
      const int nkey0 = __builtin_amdgcn_readfirstlane((e1 >> 8) * S + (g + 1 < G ? ((g + 1) % NCK) * CK : 0));
      i32x8 pop;
      qk(snxt, (g + 1) & (NST - 1), e1 & 255);
      guard(scur);
      softmax(scur, pop);
      pv(pop, g & (NST - 1));
      const int nvalid = __builtin_amdgcn_readfirstlane(N - nkey0);
      if (nvalid < CK) {
        asm volatile("");
        mask_tail(snxt, nvalid);
      }
    };
    for (int g = 0; g < G; g += 2) {
      step(g, sa, sb);
      if (g + 1 >= G) break;
      step(g + 1, sb, sa);
    }
  }
  wait_vmcnt<0>();                           // no load may still target this workgroup's LDS

  // ---- epilogue: O = O^T / l and LSE ----
  const float l_tot = lacc[0];               // every row of the ones tile holds l
  const bool has = G > 0 && l_tot > 0.0f;
  const float inv = has ? 1.0f / l_tot : 0.0f;
  if (qr < N) {
    const size_t obase = ((size_t)bh * N + qr) * D;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        const int d = dt * 32 + r4 * 8 + hf * 4;
        if (DP != D && d >= D) continue;     // padding channels
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
    if (a.lse && hf == 0)
      a.lse[(size_t)bh * N + qr] = has ? (m_ref - (float)kShift + __log2f(l_tot)) * 0.69314718055994530942f : -INFINITY;
  }
}

template <int D, int S>
hipError_t launch_fp8_ds(const Dims& d, bool sparse, const Fp8AttnArgs& a, hipStream_t stream) {
  dim3 grid(a.n_rows), block(2 * S);
  if (sparse) {
    if (d.out_f32) hipLaunchKernelGGL((attn_fp8_kernel<D, S, true, true>), grid, block, 0, stream, a);
    else hipLaunchKernelGGL((attn_fp8_kernel<D, S, true, false>), grid, block, 0, stream, a);
  } else {
    if (d.out_f32) hipLaunchKernelGGL((attn_fp8_kernel<D, S, false, true>), grid, block, 0, stream, a);
    else hipLaunchKernelGGL((attn_fp8_kernel<D, S, false, false>), grid, block, 0, stream, a);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attention_fp8(const Dims& d, bool sparse, const Fp8AttnArgs& args, hipStream_t stream) {
  Fp8AttnArgs a = args;
  a.N = d.N;
  a.nB = d.nB;
  a.Np = d.nB * d.S;
  a.n_rows = d.B * d.H * d.nB;
  const int64_t fb = ((int64_t)d.frame_tokens + d.S / 2) / d.S;
  a.frame_blocks = fb < 1 ? 1 : (fb > d.nB ? d.nB : (int)fb);
  switch (d.D * 1000 + d.S) {
    case 64064: return launch_fp8_ds<64, 64>(d, sparse, a, stream);
    case 64128: return launch_fp8_ds<64, 128>(d, sparse, a, stream);
    case 112064: return launch_fp8_ds<112, 64>(d, sparse, a, stream);
    case 112128: return launch_fp8_ds<112, 128>(d, sparse, a, stream);
    case 128064: return launch_fp8_ds<128, 64>(d, sparse, a, stream);
    case 128128: return launch_fp8_ds<128, 128>(d, sparse, a, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace sva
