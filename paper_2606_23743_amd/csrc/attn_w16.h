// Per-chunk arithmetic of the bf16 attention kernels on mfma_f32_16x16x32_bf16
// (attention_q16.hip, attention_pair.hip): QT tiles of 16 queries per wave
// (two: 32 queries), one staged 32-key chunk at a time.
//
// Lane l = 16g + i (group g = 0..3, column i = 0..15).  For query tile qt the
// lane holds query qt*16 + i:
//   S^T tile (kt, qt) = K_kt Q_qt^T over d in KS steps of 32: the A operand is
//     K row kt*16 + i at d = 32s + 8g .. +8 (one ds_read_b128, shared by both
//     query tiles), the B operand Q^T of the same d range, kept in registers;
//     the result puts keys kt*16 + 4g + r (r = 0..3) of the lane's query in
//     its four registers.
//   P = exp2(c*log2e*s - m) in float32, rounded to bf16; l sums the rounded
//     values (v_dot2 with (1, 1)), so l is exactly the weight the PV product
//     applied.  m is the reference maximum taken from the query's first chunk.
//   O^T tile (dt, qt) += V^T_dt P^T_qt with the contraction over the 32 keys in
//     the order kappa = 8g + e <-> key (e < 4 ? 4g + e : 16 + 4g + e - 4): the
//     lane's eight P values of a query (key tile 0, then 1) are its B operand
//     as they stand, and the A operand (d = 16dt + i at those keys) is two
//     ds_read_b64_tr_b16 at rows 4g.. and 16 + 4g.. of the V tile (swz_v16).
// Against the 32x32x16 form this moves half the accumulator registers per
// multiply: fewer register-file bytes per FLOP, the larger part of the power
// a matrix-bound kernel draws.
#pragma once

#include "attn_wave32.h"

namespace sva {
namespace attn {

template <int D>
struct Geo16 {
  static constexpr int KS = (D + 31) / 32;   // 32-wide d steps of the S products (zero-padded Q)
  static constexpr int DT = D / 16;          // 16-row d tiles of O^T
  static_assert(D % 16 == 0, "head dim multiple of 16");
};

// Per-lane LDS offsets: K operand of step s (key tile 0; tile 1 is 16 rows
// further, the same swizzle) and the first transpose read of d tile dt (the
// second is 16 rows further, the same swizzle).
template <int D>
__device__ __forceinline__ void operand_offsets16(int lane, int (&koff)[Geo16<D>::KS], int (&voff)[Geo16<D>::DT]) {
  using G = Geo<D>;
  const int g = lane >> 4, i = lane & 15;
#pragma unroll
  for (int s = 0; s < Geo16<D>::KS; ++s) koff[s] = i * G::RB + (swz_k<G::NCH>(i, 4 * s + g) << 4);
  const int r1 = 4 * g + (i >> 2);
#pragma unroll
  for (int dt = 0; dt < Geo16<D>::DT; ++dt)
    voff[dt] = r1 * G::RB + (swz_v16<G::NCH>(r1, 2 * dt + ((i & 3) >> 1)) << 4) + (i & 1) * 8;
}

// Q^T operands of queries qbase + qt*16 + i at d = 32s + 8g .. +8; zero for an
// absent query or d >= D
template <int D, int QT>
__device__ __forceinline__ void load_q16(bf16x8 (&qop)[QT][Geo16<D>::KS], const uint16_t* Qh, int qbase, int N,
                                         int lane) {
  const int g = lane >> 4, i = lane & 15;
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    const int q = qbase + qt * 16 + i;
#pragma unroll
    for (int s = 0; s < Geo16<D>::KS; ++s) {
      const int d0 = s * 32 + g * 8;
      if (q < N && d0 < D) qop[qt][s] = *reinterpret_cast<const bf16x8*>(Qh + (size_t)q * D + d0);
      else qop[qt][s] = bf16x8{};
    }
  }
}

template <int D, int QT>
__device__ __forceinline__ void qk16(f32x4 (&sacc)[2][QT], const unsigned char* kt, const int (&koff)[Geo16<D>::KS],
                                     const bf16x8 (&qop)[QT][Geo16<D>::KS]) {
  using G = Geo<D>;
#pragma unroll
  for (int k2 = 0; k2 < 2; ++k2)
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) sacc[k2][qt] = f32x4{};
#pragma unroll
  for (int s = 0; s < Geo16<D>::KS; ++s)
#pragma unroll
    for (int k2 = 0; k2 < 2; ++k2) {
      const bf16x8 kop = *reinterpret_cast<const bf16x8*>(kt + koff[s] + k2 * 16 * G::RB);
#pragma unroll
      for (int qt = 0; qt < QT; ++qt)
        sacc[k2][qt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kop, qop[qt][s], sacc[k2][qt], 0, 0, 0);
    }
}

// keys of the chunk at or past `valid` (the sequence's last partial chunk) to -inf
template <int QT>
__device__ __forceinline__ void mask_tail16(f32x4 (&sacc)[2][QT], int valid, int lane) {
  const int g = lane >> 4;
#pragma unroll
  for (int k2 = 0; k2 < 2; ++k2)
#pragma unroll
    for (int r = 0; r < 4; ++r)
      if (k2 * 16 + 4 * g + r >= valid) {
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) sacc[k2][qt][r] = -INFINITY;
      }
}

// max / sum over the four lanes that hold one query (l, l^16, l^32, l^48);
// every one of the four gets the same bits
__device__ __forceinline__ float quad_max(float x) {
  x = fmaxf(x, __shfl_xor(x, 16));
  return swap_halves_max(x);
}
__device__ __forceinline__ float quad_sum(float x) {
  x = x + __shfl_xor(x, 16);
  return swap_halves_sum(x);
}

// the reference maximum (log2 units) of each query tile from a chunk that
// holds a valid key
template <int QT>
__device__ __forceinline__ void chunk_reference16(const f32x4 (&sacc)[2][QT], float sl2, float (&m_ref)[QT]) {
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    float mx = sacc[0][qt][0];
#pragma unroll
    for (int k2 = 0; k2 < 2; ++k2)
#pragma unroll
      for (int r = 0; r < 4; ++r) mx = fmaxf(mx, sacc[k2][qt][r]);
    m_ref[qt] = quad_max(mx) * sl2;
  }
}

template <int QT>
__device__ __forceinline__ void softmax16(const f32x4 (&sacc)[2][QT], bf16x8 (&pop)[QT], float (&l_part)[QT],
                                          const float (&m_ref)[QT], float sl2) {
  const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    u32x4 wv;
    float lsum = l_part[qt];
#pragma unroll
    for (int k2 = 0; k2 < 2; ++k2)
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[k2][qt][2 * e], sl2, -m_ref[qt]));
        const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[k2][qt][2 * e + 1], sl2, -m_ref[qt]));
        const bf16x2 pb = cvt2(p0, p1);
        lsum = __builtin_amdgcn_fdot2_f32_bf16(pb, ones, lsum, false);
        wv[k2 * 2 + e] = __builtin_bit_cast(unsigned, pb);
      }
    pop[qt] = __builtin_bit_cast(bf16x8, wv);
    l_part[qt] = lsum;
  }
}

// V^T operand of d tile dt: the values at d = 16dt + i of keys 4g + 0..3, then
// 16 + 4g + 0..3 (voff from operand_offsets16)
template <int D>
__device__ __forceinline__ bf16x8 tr_operand16(const unsigned char* tile, int voff) {
  using G = Geo<D>;
  const unsigned char* p = tile + voff;
  const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p));
  const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p + 16 * G::RB));
  const u32x2 lw = __builtin_bit_cast(u32x2, lo);
  const u32x2 hw = __builtin_bit_cast(u32x2, hi);
  const u32x4 vw = {lw[0], lw[1], hw[0], hw[1]};
  return __builtin_bit_cast(bf16x8, vw);
}

template <int D, int QT>
__device__ __forceinline__ void pv16(const bf16x8 (&pop)[QT], const unsigned char* vt, const int (&voff)[Geo16<D>::DT],
                                     f32x4 (&oacc)[Geo16<D>::DT][QT]) {
#pragma unroll
  for (int dt = 0; dt < Geo16<D>::DT; ++dt) {
    const bf16x8 vop = tr_operand16<D>(vt, voff[dt]);
#pragma unroll
    for (int qt = 0; qt < QT; ++qt)
      oacc[dt][qt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vop, pop[qt], oacc[dt][qt], 0, 0, 0);
  }
}

// After every kept block: a query whose row sum has grown past 2^64 moves its
// reference up by the sum's binary exponent and scales its O and l by the same
// power of two (exact).  Rows never come near 2^64 in practice, so this is one
// compare and a branch per block; a row that still overflows inside one block
// is caught by overflowed16 at the end.
template <int D, int QT>
__device__ __forceinline__ void rescale_if_large16(float (&l_part)[QT], float (&m_ref)[QT],
                                                   f32x4 (&oacc)[Geo16<D>::DT][QT]) {
  bool big = false;
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) big |= l_part[qt] > 0x1p64f;
  if (__builtin_amdgcn_ballot_w64(big) != 0) {
    asm volatile("");
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
      const float l_tot = quad_sum(l_part[qt]);
      const int e = l_tot > 0x1p64f ? __builtin_amdgcn_frexp_expf(l_tot) : 0;
      const float f = __builtin_amdgcn_ldexpf(1.0f, -e);
      l_part[qt] *= f;
#pragma unroll
      for (int dt = 0; dt < Geo16<D>::DT; ++dt)
#pragma unroll
        for (int r = 0; r < 4; ++r) oacc[dt][qt][r] *= f;
      m_ref[qt] += (float)e;
    }
  }
}

// a query that would need the per-iteration rescaling: sum past 2^100 or a
// non-finite accumulator
template <int D, int QT>
__device__ __forceinline__ bool overflowed16(const float (&l_tot)[QT], const f32x4 (&oacc)[Geo16<D>::DT][QT]) {
  bool bad = false;
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) bad |= !(l_tot[qt] < 0x1p100f);
#pragma unroll
  for (int dt = 0; dt < Geo16<D>::DT; ++dt)
#pragma unroll
    for (int qt = 0; qt < QT; ++qt)
#pragma unroll
      for (int r = 0; r < 4; ++r) bad |= !__builtin_isfinite(oacc[dt][qt][r]);
  return bad;
}

// O = O^T / l of the lane's two queries (qbase + qt*16 + i, those below N) at
// d = 16dt + 4g .. +4, and their LSE; zeros and -inf for a query that attended
// to nothing (has[qt] false)
template <int D, bool OUT_F32, int QT>
__device__ __forceinline__ void store_query16(void* out, float* lse, size_t head, size_t lse_head, int qbase, int N,
                                              const f32x4 (&oacc)[Geo16<D>::DT][QT], const float (&l_tot)[QT],
                                              const float (&m_ref)[QT], const bool (&has)[QT], int lane) {
  const int g = lane >> 4, i = lane & 15;
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    const int q = qbase + qt * 16 + i;
    if (q >= N) continue;
    const float inv = has[qt] ? 1.0f / l_tot[qt] : 0.0f;
    const size_t ob = head + (size_t)q * D;
#pragma unroll
    for (int dt = 0; dt < Geo16<D>::DT; ++dt) {
      const int d = dt * 16 + 4 * g;
      const float o0 = oacc[dt][qt][0] * inv, o1 = oacc[dt][qt][1] * inv;
      const float o2 = oacc[dt][qt][2] * inv, o3 = oacc[dt][qt][3] * inv;
      if constexpr (OUT_F32) {
        *reinterpret_cast<float4*>(static_cast<float*>(out) + ob + d) = make_float4(o0, o1, o2, o3);
      } else {
        const bf16x2 x = cvt2(o0, o1), y = cvt2(o2, o3);
        const bf16x4 o = {x[0], x[1], y[0], y[1]};
        *reinterpret_cast<bf16x4*>(static_cast<uint16_t*>(out) + ob + d) = o;
      }
    }
    if (lse && g == 0)
      lse[lse_head + q] = has[qt] ? (m_ref[qt] + __log2f(l_tot[qt])) * 0.69314718055994530942f : -INFINITY;
  }
}

}  // namespace attn
}  // namespace sva
