// Block-sparse (and dense) flash attention for gfx950 (Section 4.2.2: the kept
// blocks are computed exactly; Appendix A.2.2: FlashAttention dense fallback).
//
// Workgroup = one query block of S tokens (the selection granularity), S/32
// waves, each wave owning 32 query rows.  The key/value loop walks the block's
// kv_idx list (or every block, dense); each kept block is an S x D tile of K
// and of V, staged through LDS and shared by the waves.
//
// Per kept block and wave:
//   S^T = K Q^T   mfma_f32_32x32x16_bf16 with A = K rows read from LDS
//                 (ds_read_b128) and B = Q^T held in registers for the whole
//                 kernel.  Computing the transpose puts one query per lane
//                 (lane % 32) and 16 keys per 32-key subtile in its registers,
//                 so row max/sum need one cross-half exchange (lane ^ 32).
//   online softmax in float32, exp2 with the scale folded into log2(e)*c.
//   O^T += V^T P^T  mfma_f32_32x32x16_bf16 with B = P^T taken straight from
//                 the S^T accumulators (rounded to bf16) and A = V^T fetched
//                 from the row-major V tile with ds_read_b64_tr_b16, which
//                 transposes 16-bit elements across each group of 16 lanes.
//                 The key order inside a 16-key MFMA step is the order the S^T
//                 accumulator holds (keys h*4+0..3 and 8+h*4+0..3 for lane half
//                 h), and the transposed V fetch addresses exactly those keys.
// The next kept block's K/V tiles are fetched from global memory into
// registers while the current block computes.
#include "sva_internal.h"

namespace sva {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) __bf16 bf16x4;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;
typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((ext_vector_type(4))) short i16x4;
typedef __attribute__((ext_vector_type(2))) float f32x2;

typedef __attribute__((address_space(3))) i16x4 lds_i16x4;


// ds_read_b64_tr_b16 on an LDS address (the pointer must point into __shared__).
__device__ __forceinline__ i16x4 lds_read_tr16(const uint16_t* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p));
}

__device__ __forceinline__ bf16x2 cvt2(float a, float b) {
  f32x2 f = {a, b};
  return __builtin_convertvector(f, bf16x2);
}

// One query block (row = (b*H + h)*nB + i), computed by the whole workgroup.
template <int D, int S, bool SPARSE, bool OUT_F32>
__device__ __forceinline__ void attn_row(const AttnArgs& a, const int row) {
  constexpr int NW = S / 32;             // waves per workgroup
  constexpr int NT = NW * 64;            // threads
  constexpr int DP = (D + 31) / 32 * 32; // head dim padded to the 32-wide PV tiles
  constexpr int KS = D + 8;              // K row stride in LDS (elements)
  constexpr int VS = DP + 16;            // V row stride in LDS (elements)
  constexpr int KT = S / 32;             // 32-key subtiles per block
  constexpr int DQ = D / 16;             // 16-wide d steps of the QK^T contraction
  constexpr int DT = DP / 32;            // 32-wide d tiles of the PV product
  constexpr int CPR = D / 8;             // 16-byte chunks per token row
  constexpr int CH = S * CPR;            // chunks per tile
  constexpr int CPT = (CH + NT - 1) / NT;// chunks per thread per tile

  __shared__ __attribute__((aligned(16))) uint16_t Ks[S * KS];
  __shared__ __attribute__((aligned(16))) uint16_t Vs[S * VS];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = tid >> 6;
  const int hf = lane >> 5;              // lane half
  const int l32 = lane & 31;
  const int N = a.N, nB = a.nB;

  const int bh = row / nB;
  const int i = row - bh * nB;
  const size_t head = (size_t)bh * N * D;
  const uint16_t* Qh = a.q + head;
  const uint16_t* Kh = a.k + head;
  const uint16_t* Vh = a.v + head;

  if constexpr (DP > D) {
    // padding columns of the V tile are never loaded: zero them once
    for (int t = tid; t < S * (DP - D); t += NT) {
      const int r = t / (DP - D);
      Vs[r * VS + D + (t - r * (DP - D))] = 0;
    }
  }

  // Q^T operand: query (w*32 + l32), d = s*16 + hf*8 + 0..7
  const int qrow = i * S + w * 32 + l32;
  bf16x8 qop[DQ];
#pragma unroll
  for (int s = 0; s < DQ; ++s) {
    if (qrow < N) qop[s] = *reinterpret_cast<const bf16x8*>(Qh + (size_t)qrow * D + s * 16 + hf * 8);
    else qop[s] = bf16x8{};
  }

  int count;
  const int32_t* idxrow = nullptr;
  if constexpr (SPARSE) {
    count = min(max(a.kv_count[row], 0), a.kmax);
    idxrow = a.kv_idx + (size_t)row * a.kmax;
  } else {
    count = nB;
  }
  auto block_at = [&](int it) -> int { return SPARSE ? idxrow[it] : it; };
  auto next_valid = [&](int it) -> int {
    while (it < count) {
      const int j = block_at(it);
      if (j >= 0 && j < nB) break;
      ++it;
    }
    return it;
  };

  uint4 kreg[CPT], vreg[CPT];
  auto fetch = [&](int j) {
    const int valid = min(S, N - j * S);
    const uint16_t* kb = Kh + (size_t)j * S * D;
    const uint16_t* vb = Vh + (size_t)j * S * D;
#pragma unroll
    for (int u = 0; u < CPT; ++u) {
      const int c = tid + u * NT;
      const int r = c / CPR;
      const int col = (c - r * CPR) * 8;
      if (c < CH && r < valid) {
        kreg[u] = *reinterpret_cast<const uint4*>(kb + (size_t)r * D + col);
        vreg[u] = *reinterpret_cast<const uint4*>(vb + (size_t)r * D + col);
      } else {
        kreg[u] = make_uint4(0, 0, 0, 0);
        vreg[u] = make_uint4(0, 0, 0, 0);
      }
    }
  };
  auto stage = [&]() {
#pragma unroll
    for (int u = 0; u < CPT; ++u) {
      const int c = tid + u * NT;
      if (c < CH) {
        const int r = c / CPR;
        const int col = (c - r * CPR) * 8;
        *reinterpret_cast<uint4*>(Ks + r * KS + col) = kreg[u];
        *reinterpret_cast<uint4*>(Vs + r * VS + col) = vreg[u];
      }
    }
  };

  float m_run = -INFINITY;   // running max of the scaled logits (log2 domain)
  float l_run = 0.0f;        // this lane's partial row sum (its half of the keys)
  f32x16 oacc[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) oacc[dt] = f32x16{};

  const float sl2 = a.scale_log2;
  int it = next_valid(0);
  if (it < count) fetch(block_at(it));

  while (it < count) {
    const int j = block_at(it);
    __syncthreads();                     // previous tile fully consumed
    stage();
    __syncthreads();                     // tile visible to every wave
    const int nit = next_valid(it + 1);
    if (nit < count) fetch(block_at(nit));

    // ---- S^T = K Q^T ----
    f32x16 sacc[KT];
#pragma unroll
    for (int kt = 0; kt < KT; ++kt) {
      sacc[kt] = f32x16{};
#pragma unroll
      for (int s = 0; s < DQ; ++s) {
        const bf16x8 kop = *reinterpret_cast<const bf16x8*>(Ks + (kt * 32 + l32) * KS + s * 16 + hf * 8);
        sacc[kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kop, qop[s], sacc[kt], 0, 0, 0);
      }
    }
    // keys past the end of the sequence (last block only)
    const int valid = N - j * S;
    if (valid < S) {
#pragma unroll
      for (int kt = 0; kt < KT; ++kt)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = kt * 32 + (r >> 2) * 8 + hf * 4 + (r & 3);
          if (key >= valid) sacc[kt][r] = -INFINITY;
        }
    }
    // ---- online softmax ----
    float mx = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < KT; ++kt)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sacc[kt][r]);
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    const float m_new = fmaxf(m_run, mx * sl2);
    const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
    m_run = m_new;
    float rs = 0.0f;
    bf16x8 pop[KT][2];
#pragma unroll
    for (int kt = 0; kt < KT; ++kt) {
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
        bf16x8 pv;
#pragma unroll
        for (int e = 0; e < 8; e += 2) {
          const float p0 = __builtin_amdgcn_exp2f(fmaf(sacc[kt][kk * 8 + e], sl2, -m_new));
          const float p1 = __builtin_amdgcn_exp2f(fmaf(sacc[kt][kk * 8 + e + 1], sl2, -m_new));
          const bf16x2 pb = cvt2(p0, p1);
          pv[e] = pb[0];
          pv[e + 1] = pb[1];
          rs += (float)pb[0] + (float)pb[1];   // sum what the MFMA will see
        }
        pop[kt][kk] = pv;
      }
    }
    l_run = l_run * alpha + rs;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int r = 0; r < 16; ++r) oacc[dt][r] *= alpha;

    // ---- O^T += V^T P^T ----
    const int g = lane >> 4;             // 16-lane group
    const int n16 = lane & 15;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
      const int col = dt * 32 + (g & 1) * 16 + 4 * (n16 & 3);
#pragma unroll
      for (int kt = 0; kt < KT; ++kt)
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
          const int r0 = kt * 32 + kk * 16 + hf * 4 + (n16 >> 2);
          const i16x4 lo = lds_read_tr16(Vs + r0 * VS + col);
          const i16x4 hi = lds_read_tr16(Vs + (r0 + 8) * VS + col);
          const bf16x4 lob = __builtin_bit_cast(bf16x4, lo);
          const bf16x4 hib = __builtin_bit_cast(bf16x4, hi);
          const bf16x8 vop = {lob[0], lob[1], lob[2], lob[3], hib[0], hib[1], hib[2], hib[3]};
          oacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vop, pop[kt][kk], oacc[dt], 0, 0, 0);
        }
    }
    it = nit;
  }

  // ---- epilogue: O = O^T / l, LSE ----
  const float l_tot = l_run + __shfl_xor(l_run, 32, 64);
  const float inv = l_tot > 0.0f ? 1.0f / l_tot : 0.0f;
  if (qrow < N) {
    const size_t obase = head + (size_t)qrow * D;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
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
      a.lse[(size_t)bh * N + qrow] =
          l_tot > 0.0f ? (m_run + __log2f(l_tot)) * 0.69314718055994530942f : -INFINITY;
    }
  }
}

// Recomputes the query blocks the fixed-reference kernel marked (NaN first
// output element).  A small grid scans the marks 64 rows at a time (one row
// per lane, one ballot) and runs the per-block body only for marked rows, so
// the common case (nothing marked) costs a few microseconds.
template <int D, int S, bool SPARSE, bool OUT_F32>
__global__ __launch_bounds__(S * 2) void attn_marked_kernel(AttnArgs a) {
  const int lane = threadIdx.x & 63;
  for (int base = blockIdx.x * 64; base < a.n_rows; base += gridDim.x * 64) {
    const int r = base + lane;
    bool marked = false;
    if (r < a.n_rows) {
      const int bh = r / a.nB;
      const size_t first = (size_t)bh * a.N * D + (size_t)(r - bh * a.nB) * S * D;
      marked = OUT_F32 ? __builtin_isnan(static_cast<const float*>(a.out)[first])
                       : ((static_cast<const uint16_t*>(a.out)[first] & 0x7FFF) > 0x7F80);
    }
    uint64_t mask = __builtin_amdgcn_ballot_w64(marked);
    // every wave holds the same mask before any marked row is rewritten, so
    // all waves run the same rows (and barriers) below
    __syncthreads();
    while (mask != 0) {
      const int b = __builtin_ctzll(mask);
      mask &= mask - 1;
      attn_row<D, S, SPARSE, OUT_F32>(a, base + b);
      __syncthreads();                   // LDS tiles are reused by the next row
    }
  }
}

template <int D, int S>
hipError_t launch_ds(const Dims& d, bool sparse, const AttnArgs& a, hipStream_t stream) {
  const int groups = (a.n_rows + 63) / 64;
  dim3 grid(groups < 2048 ? groups : 2048), block(S * 2);
  if (sparse) {
    if (d.out_f32) hipLaunchKernelGGL((attn_marked_kernel<D, S, true, true>), grid, block, 0, stream, a);
    else hipLaunchKernelGGL((attn_marked_kernel<D, S, true, false>), grid, block, 0, stream, a);
  } else {
    if (d.out_f32) hipLaunchKernelGGL((attn_marked_kernel<D, S, false, true>), grid, block, 0, stream, a);
    else hipLaunchKernelGGL((attn_marked_kernel<D, S, false, false>), grid, block, 0, stream, a);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attention_rescaling(const Dims& d, bool sparse, const AttnArgs& a, hipStream_t stream) {
  switch (d.D * 1000 + d.S) {
    case 64064: return launch_ds<64, 64>(d, sparse, a, stream);
    case 64128: return launch_ds<64, 128>(d, sparse, a, stream);
    case 112064: return launch_ds<112, 64>(d, sparse, a, stream);
    case 112128: return launch_ds<112, 128>(d, sparse, a, stream);
    case 128064: return launch_ds<128, 64>(d, sparse, a, stream);
    case 128128: return launch_ds<128, 128>(d, sparse, a, stream);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_attention(const Dims& d, bool sparse, const uint16_t* q, const uint16_t* k,
                            const uint16_t* v, const int32_t* kv_idx, const int32_t* kv_count,
                            int kmax, void* out, float* lse, hipStream_t stream) {
  // Dense attention does not depend on the block size: at S = 64 it runs as
  // 128-token query tiles (four waves share every staged key chunk instead of
  // two; the same keys, in the same 32-key chunks and order).
  Dims dd = d;
  if (!sparse && d.S == 64) {
    dd.S = 128;
    dd.nB = (d.N + 127) / 128;
  }
  AttnArgs a;
  a.q = q;
  a.k = k;
  a.v = v;
  a.kv_idx = kv_idx;
  a.kv_count = kv_count;
  a.out = out;
  a.lse = lse;
  a.N = dd.N;
  a.nB = dd.nB;
  a.kmax = kmax;
  a.n_rows = dd.B * dd.H * dd.nB;
  a.scale_log2 = (float)(dd.scale * 1.4426950408889634);
  const int64_t fb = ((int64_t)dd.frame_tokens + dd.S / 2) / dd.S;
  a.frame_blocks = fb < 1 ? 1 : (fb > dd.nB ? dd.nB : (int)fb);
  // fixed-reference-max kernel (block pairs for sparse 64-token blocks), then
  // the rescaling kernel for any block it marked
  hipError_t e = (sparse && pair_attention_fits(dd, kmax)) ? launch_attention_pair(dd, a, stream)
                                                     : launch_attention_q16(dd, sparse, a, stream);
  if (e != hipSuccess) return e;
  return launch_attention_rescaling(dd, sparse, a, stream);
}

}  // namespace sva
