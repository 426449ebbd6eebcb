// First-order remainder of the key blocks a query block does not keep
// (Section 4.2.2: the non-critical blocks are compensated to first order
// instead of dropped).
//
// For query q of query block i and a dropped key block j (n_j valid tokens,
// means kbar_j and vbar_j, moment M_j[e][d] = sum_t v_t[e] (k_t - kbar_j)[d]),
// the block's exponentials are expanded to first order about the block's mean
// key, with the weight of the first-order term taken at the block-mean query
// (so that the term is one matrix per query block):
//   row sum    += n_j exp(c q.kbar_j)
//   numerator  += n_j exp(c q.kbar_j) vbar_j + exp(c qbar_i.kbar_j) c M_j q
// on top of the exact sums over the kept keys.  Four kernels:
//   rem_moments_kernel  one workgroup per key block: kbar, vbar (bf16) and M
//                       (bf16, [e][d]) as V^T (K - kbar) on MFMA, both
//                       operands by transpose reads of LDS tiles
//   rem_weights_kernel  per query block i: r_i = max_j c qbar_i.kbar_j and
//                       E[i][j] = exp(c qbar_i.kbar_j - r_i) for the dropped j,
//                       0 for kept and padding columns (bf16, chunk-blocked)
//   rem_gemm_kernel     T_i = sum_j E[i][j] M_j: per head one GEMM of E
//                       [nB x nB] with the flattened moments [nB x D*D] (MFMA,
//                       M and E tiles staged in LDS by direct loads)
//   rem_attn_kernel     per 128 queries: the kept-block result (float32 O and
//                       LSE) and exp(r_i) c T_i q as the starting numerator,
//                       then an online softmax over the nB pooled keys kbar_j
//                       with weight n_j (kept and padding blocks masked),
//                       values vbar_j
#include "attn_w16.h"

namespace sva {
namespace {

using namespace attn;

constexpr float kLog2e = 1.4426950408889634f;

__device__ __forceinline__ uint16_t bf16_bits(float x) { return __builtin_bit_cast(uint16_t, (__bf16)x); }

// ---------------------------------------------------------------------------
// Block means and moments.  One workgroup (4 waves) per (b, h, key block j);
// rows j >= nB (padding up to `rows`) are written as zeros.  The block's K and
// V rows are staged by direct loads as 32-row V-swizzled tiles (rows past the
// block's end zeroed), then, on MFMA with both operands from the LDS
// transpose read:
//   P = V^T K             tile (et, dt): A = the V tile at et, B = the K tile at dt
//   sv = V^T 1, sk = 1^T K   the same reads against an all-ones operand: sv
//                            lands in P's row layout, sk in its column layout
//   M = P - sv sk^T / n,  kbar = sk / n,  vbar = sv / n
// so the means and the moment come from one pass over exact bf16 products with
// float32 sums.  Wave w takes the (et, dt) tiles with (et*DT + dt) % 4 == w;
// at DT = 4 its column tile dt = w is fixed.
// ---------------------------------------------------------------------------
template <int D, int S>
__global__ __launch_bounds__(256) void rem_moments_kernel(RemMomentArgs a) {
  using G = Geo<D>;
  constexpr int NT = 256;
  constexpr int NCHK = S / 32;               // 32-row tiles per block
  constexpr int CT = 32 * G::RB;
  constexpr int NUW = CT / 1024 / 4;         // direct-load pieces per wave per tile
  constexpr int TILES = G::DT * G::DT;
  constexpr int TPW = (TILES + 3) / 4;       // output tiles per wave
  static_assert(NUW >= 1, "tile split");
  // K and V tiles in one array: after the products it holds M for the store
  __shared__ __attribute__((aligned(1024))) unsigned char KVt[2][NCHK][CT];
  static_assert(2 * NCHK * CT >= D * D * 2, "M staging");
  unsigned char (*Kt)[CT] = KVt[0];
  unsigned char (*Vt)[CT] = KVt[1];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int hf = lane >> 5, l32 = lane & 31;
  const int item = blockIdx.x;               // bh * rows + j
  const int bh = item / a.rows;
  const int j = item - bh * a.rows;
  const size_t dd = (size_t)D * D;
  uint16_t* kbar = a.kbar + (size_t)item * D;
  uint16_t* vbar = a.vbar + (size_t)item * D;
  uint16_t* mom = a.mom + (size_t)item * dd;
  if (j >= a.nB) {
    for (int t = tid; t < D; t += NT) {
      kbar[t] = 0;
      vbar[t] = 0;
    }
    for (int t = tid; t < (int)(dd / 8); t += NT) reinterpret_cast<uint4*>(mom)[t] = make_uint4(0, 0, 0, 0);
    return;
  }
  const int t0 = j * S;
  const int n = min(S, a.N - t0);
  const uint16_t* Kb = a.k + ((size_t)bh * a.N + t0) * D;
  const uint16_t* Vb = a.v + ((size_t)bh * a.N + t0) * D;

  // Both tensors with the V swizzle (the loader's second tensor path): rows
  // of a partial block past its end read an earlier row, zeroed below.
  ChunkLoader<D, NUW, CT> lk, lv;
  loader_init(lk, Kb, Kb, n, &Kt[0][0], &Kt[0][0], w, lane);
  loader_init(lv, Vb, Vb, n, &Vt[0][0], &Vt[0][0], w, lane);
#pragma unroll
  for (int ch = 0; ch < NCHK; ++ch) {
    load_tile<false>(lk, ch, ch * 32);
    load_tile<false>(lv, ch, ch * 32);
  }
  wait_vmcnt<0>();
  __syncthreads();
  if (n < S) {
    for (int p = tid; p < (S - n) * G::NCH; p += NT) {
      const int t = n + p / G::NCH, c = p % G::NCH;
      const int off = (t >> 5) * CT + (t & 31) * G::RB + c * 16;
      *reinterpret_cast<uint4*>(&Kt[0][0] + off) = make_uint4(0, 0, 0, 0);
      *reinterpret_cast<uint4*>(&Vt[0][0] + off) = make_uint4(0, 0, 0, 0);
    }
    __syncthreads();
  }

  const u32x4 one_bits = {0x3F803F80u, 0x3F803F80u, 0x3F803F80u, 0x3F803F80u};   // bf16 1.0 x 8
  const bf16x8 ones = __builtin_bit_cast(bf16x8, one_bits);
  static_assert(4 % G::DT == 0, "a wave's column tile is fixed");
  const int dtw = w % G::DT;                 // this wave's column tile
  const int db = tr_offset<D>(lane, dtw);
  f32x16 acc[TPW], sk = f32x16{};
#pragma unroll
  for (int x = 0; x < TPW; ++x) acc[x] = f32x16{};
#pragma unroll
  for (int ch = 0; ch < NCHK; ++ch)
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      const bf16x8 kb = tr_operand<D>(&Kt[ch][0], db, kk);
      sk = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ones, kb, sk, 0, 0, 0);
#pragma unroll
      for (int x = 0; x < TPW; ++x) {
        const int tile = w + 4 * x;
        if (tile < TILES) {
          const int et = tile / G::DT;
          acc[x] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(tr_operand<D>(&Vt[ch][0], tr_offset<D>(lane, et), kk), kb,
                                                           acc[x], 0, 0, 0);
        }
      }
    }
  const float inv_n = 1.0f / (float)n;
  // means: the K sums of columns dtw*32 .. (written by the wave with et = 0),
  // and per tile the V sums of its rows (written by the tile with dt = 0);
  // the moment is P - sv sk^T / n
#pragma unroll
  for (int x = 0; x < TPW; ++x) {
    const int tile = w + 4 * x;
    if (tile < TILES) {
      const int et = tile / G::DT;
      const int ea = tr_offset<D>(lane, et);
      f32x16 sv = f32x16{};
#pragma unroll
      for (int ch = 0; ch < NCHK; ++ch)
#pragma unroll
        for (int kk = 0; kk < 2; ++kk)
          sv = __builtin_amdgcn_mfma_f32_32x32x16_bf16(tr_operand<D>(&Vt[ch][0], ea, kk), ones, sv, 0, 0, 0);
      if (dtw == 0 && l32 == 0) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int e = et * 32 + (r >> 2) * 8 + hf * 4 + (r & 3);
          if (e < D) vbar[e] = bf16_bits(sv[r] * inv_n);
        }
      }
      if (et == 0 && hf == 0 && dtw * 32 + l32 < D) kbar[dtw * 32 + l32] = bf16_bits(sk[0] * inv_n);
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[x][r] = __builtin_fmaf(-sv[r] * inv_n, sk[r], acc[x][r]);
    }
  }

  // M through LDS (row e, D bf16 per row) so that the global stores are
  // whole 16-byte pieces of consecutive rows
  __syncthreads();                           // every wave is done with the tiles
  uint16_t* Ms = reinterpret_cast<uint16_t*>(&KVt[0][0][0]);
#pragma unroll
  for (int x = 0; x < TPW; ++x) {
    const int tile = w + 4 * x;
    if (tile < TILES) {
      const int et = tile / G::DT;
      const int d = dtw * 32 + l32;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int e = et * 32 + (r >> 2) * 8 + hf * 4 + (r & 3);
        if (e < D && d < D) Ms[e * D + d] = bf16_bits(acc[x][r]);
      }
    }
  }
  __syncthreads();
  for (int p = tid; p < D * D / 8; p += NT)
    reinterpret_cast<uint4*>(mom)[p] = reinterpret_cast<const uint4*>(Ms)[p];
}

// ---------------------------------------------------------------------------
// First-order weights.  A workgroup of four waves takes 128 query blocks of
// one head, a lane one query block i (32 per wave).  The scores c qbar_i.kbar_j
// are a small dense product per head, done on MFMA as S^T = Kbar Qbar^T over
// 32-key chunks; each float32 mean is split into bf16 high and low parts and
// the three products hi.hi + hi.lo + lo.hi are summed in float32 (relative
// error about 2^-16, against the 2^-9 of E's bf16 storage).  Pass one takes
// the row maxima r_i (a lane's registers and the lane pair), pass two writes
// E = exp(s - r_i) chunk-blocked, one 16-byte piece per lane and key half;
// then the kept entries of each row's list are set to zero.
// ---------------------------------------------------------------------------
constexpr int kRemRows = 128;              // query blocks per workgroup

// Position of key jj (0..31) of a chunk in a row of E: the eight keys one MFMA
// lane takes for (kk, hf) -- kk*16 + hf*4 + 0..3, then kk*16 + 8 + hf*4 + 0..3,
// the key order of a 32x32x16 S^T register group -- are the 16-byte piece
// kk*2 + hf.
__host__ __device__ __forceinline__ int e_position(int jj) {
  const int kk = jj >> 4, r = jj & 15;
  return kk * 16 + ((r >> 2) & 1) * 8 + (r >> 3) * 4 + (r & 3);
}

template <int D>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2)))
void rem_weights_kernel(RemWeightArgs a) {
  using G = Geo<D>;
  constexpr int NT = 256;
  constexpr int CT = 32 * G::RB;
  __shared__ __attribute__((aligned(1024))) unsigned char Kh[CT], Kl[CT];
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int hf = lane >> 5, l32 = lane & 31;
  const int nB = a.nB, nBp = a.nBp, nBr = a.nBr, nch = nBp / 32;
  const int groups = (nB + kRemRows - 1) / kRemRows;
  const int bh = blockIdx.x / groups;
  const int i0 = (blockIdx.x - bh * groups) * kRemRows;
  const int i = i0 + w * 32 + l32;           // this lane's query block
  const bool live = i < nB;
  const float c = a.scale;
  const float* kp = a.k_pool + (size_t)bh * nB * D;

  // Qbar^T operand of row i, high and low bf16 parts: d = s*16 + hf*8 + 0..7
  auto split8 = [](const float* x, bf16x8& hi, bf16x8& lo) {
    u32x4 h, l;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const bf16x2 ph = cvt2(x[2 * e], x[2 * e + 1]);
      const bf16x2 pl = cvt2(x[2 * e] - (float)ph[0], x[2 * e + 1] - (float)ph[1]);
      h[e] = __builtin_bit_cast(unsigned, ph);
      l[e] = __builtin_bit_cast(unsigned, pl);
    }
    hi = __builtin_bit_cast(bf16x8, h);
    lo = __builtin_bit_cast(bf16x8, l);
  };
  bf16x8 qh[G::DQ], ql[G::DQ];
  {
    const float* qr = a.q_pool + ((size_t)bh * nB + (live ? i : 0)) * D;
#pragma unroll
    for (int s = 0; s < G::DQ; ++s) {
      float x[8];
      const float4 x0 = *reinterpret_cast<const float4*>(qr + s * 16 + hf * 8);
      const float4 x1 = *reinterpret_cast<const float4*>(qr + s * 16 + hf * 8 + 4);
      x[0] = x0.x; x[1] = x0.y; x[2] = x0.z; x[3] = x0.w;
      x[4] = x1.x; x[5] = x1.y; x[6] = x1.z; x[7] = x1.w;
      if (!live) {
#pragma unroll
        for (int e = 0; e < 8; ++e) x[e] = 0.0f;
      }
      split8(x, qh[s], ql[s]);
    }
  }
  int koff[G::DQ], voff[G::DT];
  operand_offsets<D>(lane, koff, voff);

  // scores of chunk ch (natural-log units; -inf past nB), lane = row i
  auto chunk_scores = [&](int ch, f32x16& sc) {
    __syncthreads();                         // the previous chunk's tiles are read
    for (int p = tid; p < 32 * G::DCH; p += NT) {
      const int r = p / G::DCH, cp = p - (p / G::DCH) * G::DCH;
      const int j = ch * 32 + r;
      float x[8];
      if (j < nB) {
        const float4 x0 = *reinterpret_cast<const float4*>(kp + (size_t)j * D + cp * 8);
        const float4 x1 = *reinterpret_cast<const float4*>(kp + (size_t)j * D + cp * 8 + 4);
        x[0] = x0.x; x[1] = x0.y; x[2] = x0.z; x[3] = x0.w;
        x[4] = x1.x; x[5] = x1.y; x[6] = x1.z; x[7] = x1.w;
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) x[e] = 0.0f;
      }
      bf16x8 hi, lo;
      split8(x, hi, lo);
      const int off = r * G::RB + (swz_k<G::NCH>(r, cp) << 4);
      *reinterpret_cast<bf16x8*>(Kh + off) = hi;
      *reinterpret_cast<bf16x8*>(Kl + off) = lo;
    }
    __syncthreads();
    f32x16 acc = f32x16{};
#pragma unroll
    for (int s = 0; s < G::DQ; ++s) {
      const bf16x8 kh = *reinterpret_cast<const bf16x8*>(Kh + koff[s]);
      const bf16x8 kl = *reinterpret_cast<const bf16x8*>(Kl + koff[s]);
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kh, qh[s], acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kh, ql[s], acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kl, qh[s], acc, 0, 0, 0);
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int j = ch * 32 + (r >> 2) * 8 + hf * 4 + (r & 3);
      sc[r] = j < nB ? acc[r] * c : -INFINITY;
    }
  };

  float mx = -INFINITY;
  for (int ch = 0; ch < nch; ++ch) {
    f32x16 sc;
    chunk_scores(ch, sc);
#pragma unroll
    for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sc[r]);
  }
  const float rmax = swap_halves_max(mx);
  if (live && hf == 0) a.r[(size_t)bh * nBp + i] = rmax;

  for (int ch = 0; ch < nch; ++ch) {
    f32x16 sc;
    chunk_scores(ch, sc);
    if (live) {
      uint16_t* Ec = a.E + (((size_t)bh * nch + ch) * nBr + i) * 32;
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
        u32x4 pk;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float e0 = exp2f((sc[kk * 8 + 2 * e] - rmax) * kLog2e);
          const float e1 = exp2f((sc[kk * 8 + 2 * e + 1] - rmax) * kLog2e);
          pk[e] = __builtin_bit_cast(unsigned, cvt2(e0, e1));
        }
        *reinterpret_cast<u32x4*>(Ec + kk * 16 + hf * 8) = pk;
      }
    }
  }

  // the blocks a row keeps carry no first-order weight
  __syncthreads();
  for (int rr = 0; rr < kRemRows && i0 + rr < nB; ++rr) {
    const int row = bh * nB + i0 + rr;
    const int cnt = min(max(a.kv_count[row], 0), a.kmax);
    const int32_t* idx = a.kv_idx + (size_t)row * a.kmax;
    for (int t = tid; t < cnt; t += NT) {
      const int j = idx[t];
      if (j >= 0 && j < nB) a.E[(((size_t)bh * nch + (j >> 5)) * nBr + i0 + rr) * 32 + e_position(j & 31)] = 0;
    }
  }
}

// ---------------------------------------------------------------------------
// T_i = sum_j E[i][j] M_j, per head: C [nB x D*D] = E [nB x nBp] . M [nBp x D*D].
// A workgroup takes 128 columns (one LDS tile row of 256 bytes) and 256 rows
// i (64 per wave, two 32-row halves); each transpose read of M feeds both
// halves' MFMAs.  Per 32-key chunk, the M tile (32 x 128, V-swizzled) and the
// E tile (256 rows x 64 bytes, contiguous in the chunk-blocked layout; the
// 16-byte pieces of row r XOR-swizzled by (r/4)%4 so that 16 lanes reading 16
// consecutive rows hit all 64 banks) are staged by direct loads in three LDS
// stages, two chunks ahead.  Each chunk issues one load group (chunk 0 again
// past the end), so the wait counts are constants.  The waves run the PV step
// with E in place of P.  Workgroups of one column tile are consecutive in XCD
// order, so the M tile they share comes from one L2.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2)))
void rem_gemm_kernel(RemGemmArgs a) {
  using G = Geo<128>;
  constexpr int CT = 32 * G::RB;             // M tile: 32 rows x 128 columns of bf16
  constexpr int ET = kRemGemmRows * 64;      // E tile: 256 rows x 32 keys of bf16
  constexpr int NUW = CT / 1024 / 4;         // M direct loads per wave per chunk
  constexpr int NUE = ET / 1024 / 4;         // E direct loads per wave per chunk
  constexpr int NST = 3, PD = 2;             // LDS stages, load distance (chunks)
  __shared__ __attribute__((aligned(1024))) unsigned char Ms[NST][CT];
  __shared__ __attribute__((aligned(1024))) unsigned char Es[NST][ET];

  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int hf = lane >> 5, l32 = lane & 31;
  const int DD = a.DD, nB = a.nB, nBp = a.nBp, nBr = a.nBr;
  const int nct = DD / 128, nrg = (nB + kRemGemmRows - 1) / kRemGemmRows;
  const int id = __builtin_amdgcn_readfirstlane(xcd_remap(blockIdx.x, a.n_wg));
  const int rg = id % nrg;
  const int tt = id / nrg;
  const int ct = tt % nct;
  const int bh = tt / nct;
  const int c0 = ct * 128;
  const int nch = nBp / 32;

  const __amdgpu_buffer_rsrc_t mrs = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(a.mom + (size_t)bh * nBp * DD), (short)0, nBp * DD * 2, 0x00020000);
  const __amdgpu_buffer_rsrc_t ers = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(a.E + (size_t)bh * nch * nBr * 32), (short)0, nch * nBr * 64, 0x00020000);
  int mv[NUW], ev[NUE];
#pragma unroll
  for (int v = 0; v < NUW; ++v) {
    const int r = (w * NUW + v) * G::RPI + lane / G::NCH;
    mv[v] = (r * DD + c0 + swz_v<G::NCH>(r, lane % G::NCH) * 8) * 2;
  }
#pragma unroll
  for (int v = 0; v < NUE; ++v) {
    const int r = (w * NUE + v) * 16 + (lane >> 2);   // row of the E tile
    ev[v] = r * 64 + (((lane & 3) ^ ((r >> 2) & 3)) << 4);
  }
  const unsigned ms_base = __builtin_amdgcn_readfirstlane((unsigned)(size_t)(const lds_u8*)&Ms[0][0]);
  const unsigned es_base = __builtin_amdgcn_readfirstlane((unsigned)(size_t)(const lds_u8*)&Es[0][0]);
  auto fetch = [&](int st, int ch) {
    const int c = ch < nch ? ch : 0;         // past the end: chunk 0 again (in bounds, unused)
#pragma unroll
    for (int v = 0; v < NUW; ++v) buffer_to_lds(mrs, ms_base + st * CT + (w * NUW + v) * 1024, mv[v], c * 32 * DD * 2);
#pragma unroll
    for (int v = 0; v < NUE; ++v)
      buffer_to_lds(ers, es_base + st * ET + (w * NUE + v) * 1024, ev[v], (c * nBr + rg * kRemGemmRows) * 64);
  };
  // E operand offsets in a stage: row w*64 + h2*32 + l32, piece kk*2 + hf
  int eoff[2][2];
#pragma unroll
  for (int h2 = 0; h2 < 2; ++h2)
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      const int r = w * 64 + h2 * 32 + l32;
      eoff[h2][kk] = r * 64 + (((kk * 2 + hf) ^ ((r >> 2) & 3)) << 4);
    }

  int koff[G::DQ], voff[G::DT];
  operand_offsets<128>(lane, koff, voff);
  f32x16 acc[2][G::DT];
#pragma unroll
  for (int h2 = 0; h2 < 2; ++h2)
#pragma unroll
    for (int dt = 0; dt < G::DT; ++dt) acc[h2][dt] = f32x16{};
  fetch(0, 0);
  fetch(1, 1);
  for (int ch0 = 0; ch0 < nch; ch0 += NST) {
#pragma unroll
    for (int c = 0; c < NST; ++c) {
      const int ch = ch0 + c;
      if (ch >= nch) break;
      wait_vmcnt_lds_idle<NUW + NUE>();      // chunk ch landed (chunk ch+1 may be in flight)
      wg_barrier();                          // every wave's; chunk ch-1's stage is free
      fetch((c + PD) % NST, ch + PD);
      bf16x8 eop[2][2];
#pragma unroll
      for (int h2 = 0; h2 < 2; ++h2)
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) eop[h2][kk] = *reinterpret_cast<const bf16x8*>(&Es[c][0] + eoff[h2][kk]);
#pragma unroll
      for (int dt = 0; dt < G::DT; ++dt)
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
          const bf16x8 mop = tr_operand<128>(&Ms[c][0], voff[dt], kk);
#pragma unroll
          for (int h2 = 0; h2 < 2; ++h2)
            acc[h2][dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(mop, eop[h2][kk], acc[h2][dt], 0, 0, 0);
        }
    }
  }
  wait_vmcnt<0>();
#pragma unroll
  for (int h2 = 0; h2 < 2; ++h2) {
    const int i = rg * kRemGemmRows + w * 64 + h2 * 32 + l32;
    if (i >= nB) continue;
    uint16_t* Tr = a.T + ((size_t)bh * nBp + i) * DD + c0;
#pragma unroll
    for (int dt = 0; dt < G::DT; ++dt)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        const int col = dt * 32 + r4 * 8 + hf * 4;
        const bf16x2 x = cvt2(acc[h2][dt][r4 * 4 + 0], acc[h2][dt][r4 * 4 + 1]);
        const bf16x2 y = cvt2(acc[h2][dt][r4 * 4 + 2], acc[h2][dt][r4 * 4 + 3]);
        const bf16x4 o = {x[0], x[1], y[0], y[1]};
        *reinterpret_cast<bf16x4*>(Tr + col) = o;
      }
  }
}

// ---------------------------------------------------------------------------
// Remainder attention and merge, on mfma_f32_16x16x32_bf16 with the per-chunk
// arithmetic of the kept-block kernels (attn_w16.h).  One workgroup of four
// waves (32 queries each, two 16-query tiles) per 128 queries: one query block
// at S = 128, two at S = 64 (the pooled keys are the same for every query
// block of a head; only the masks differ).  The pooled keys kbar_j of the head
// are walked in 32-row chunks (four LDS stages, loads three chunks ahead):
//   x   = c*log2e * (q.kbar_j) + log2 n_j - m        (log2 units)
//   p   = exp2(x), rounded to bf16, then ANDed with the chunk's 16-bit masks
//         (zero for kept and padding blocks), l summed from the masked p
//   O^T += Vbar^T P^T
// The masks are tabulated once per workgroup in LDS, four 32-bit words per
// lane group and chunk (two keys each), so a chunk costs one LDS read of them
// and one AND per two keys.  A kept block's x is at most about 0 (the pooled
// logit plus log2 n_j is at most the block's log-sum-exp, which the reference
// m >= LSE of the kept part bounds), so only dropped blocks can move the
// reference: m starts at max(LSE of the kept part, r_i) and moves up only
// when a chunk's x passes 8, which is rare.  The last chunk (the last block's
// n_j, padding blocks) takes the general form.  The first-order term
// exp(r_i) c T_i q (the rows of T_i staged as the first chunks of the
// pipeline: the S step with T's rows as keys puts (T_i q)[e] where O^T keeps
// d = e) and the kept-block result (O and LSE in float32, weight exp(LSE))
// are the starting numerator and row sum, so the end is one division.
// ---------------------------------------------------------------------------
template <int D, int S, bool OUT_F32>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2)))
void rem_attn_kernel(RemAttnArgs a) {
  using G = Geo<D>;
  using G16 = Geo16<D>;
  constexpr int NW = 4;                      // waves: 128 queries
  constexpr int NQB = 128 / S;               // query blocks per workgroup
  constexpr int CT = 32 * G::RB;
  constexpr int NUW = CT / 1024 / NW;
  constexpr int NTT = G::DT;                 // 32-row tiles of T_i
  constexpr int NTC = NQB * NTT;             // T chunks ahead of the pooled chunks
  constexpr int kChunks = kRemMaxBlocks / 32;
  constexpr int NST = 4, PD = 3;
  static_assert(NUW >= 1, "tile split");
  __shared__ __attribute__((aligned(1024))) unsigned char Ks[NST][CT];
  __shared__ __attribute__((aligned(1024))) unsigned char Vs[NST][CT];
  // pm[b][ch][4g + 2k2 + e]: the masks of keys 16k2 + 4g + 2e (low half) and
  // + 1 (high half) of chunk ch for query block b: 0xffff where the key's
  // block is dropped (it takes part), 0 where kept or padding
  __shared__ __attribute__((aligned(16))) uint32_t pm[NQB][kChunks][16];

  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int g = lane >> 4;
  const int N = a.N, nB = a.nB, nBp = a.nBp;
  const int nch = nBp / 32;
  const int groups = (nB + NQB - 1) / NQB;
  const int item = __builtin_amdgcn_readfirstlane(xcd_remap(blockIdx.x, a.n_rows));
  const int bh = item / groups;
  const int ib0 = (item - bh * groups) * NQB;
  const int qb = w * 32 / S;                 // this wave's query block within the workgroup
  const int i_raw = ib0 + qb;                // may be nB (no such block: the wave only helps load)
  const int i = min(i_raw, nB - 1);

  for (int t = threadIdx.x; t < NQB * nch * 16; t += 256) {
    const int b2 = t / (nch * 16), rest = t - b2 * (nch * 16);
    const int ch = rest >> 4, slot = rest & 15;
    const int j0 = ch * 32 + ((slot >> 1) & 1) * 16 + (slot >> 2) * 4 + (slot & 1) * 2;
    pm[b2][ch][slot] = (j0 < nB ? 0x0000ffffu : 0u) | (j0 + 1 < nB ? 0xffff0000u : 0u);
  }
  __syncthreads();
#pragma unroll
  for (int b2 = 0; b2 < NQB; ++b2) {
    if (ib0 + b2 >= nB) break;
    const int row = bh * nB + ib0 + b2;
    const int cnt = min(max(a.kv_count[row], 0), a.kmax);
    const int32_t* idx = a.kv_idx + (size_t)row * a.kmax;
    for (int t = threadIdx.x; t < cnt; t += 256) {
      const int j = idx[t];
      if (j >= 0 && j < nB) {
        const int jj = j & 31;
        const int slot = ((jj >> 2) & 3) * 4 + (jj >> 4) * 2 + ((jj >> 1) & 1);
        atomicAnd(&pm[b2][j >> 5][slot], (jj & 1) ? 0x0000ffffu : 0xffff0000u);
      }
    }
  }
  __syncthreads();

  const int qbase = i_raw * S + (w * 32) % S;
  bf16x8 qop[2][G16::KS];
  load_q16<D>(qop, a.q + (size_t)bh * N * D, qbase, N, lane);

  ChunkLoader<D, NUW, CT, true> ld;
  loader_init(ld, a.kbar + (size_t)bh * nBp * D, a.vbar + (size_t)bh * nBp * D, nBp, &Ks[0][0], &Vs[0][0], w,
              lane);
  int koff[G16::KS], voff[G16::DT];
  operand_offsets16<D>(lane, koff, voff);

  const float sl2 = a.scale_log2;
  const float r2 = a.r[(size_t)bh * nBp + i] * kLog2e;   // block-score maximum, log2 units
  float m_ref[2], l_part[2], f1[2], l_a[2];
  f32x4 oacc[G16::DT][2];
#pragma unroll
  for (int qt = 0; qt < 2; ++qt) {
    const int q = qbase + qt * 16 + (lane & 15);
    const float lse_a = q < N ? a.lse_a[(size_t)bh * N + q] : -INFINITY;
    m_ref[qt] = fmaxf(lse_a * kLog2e, r2);
    l_a[qt] = __builtin_amdgcn_exp2f(lse_a * kLog2e - m_ref[qt]);   // 0 without a kept part
    f1[qt] = a.scale * __builtin_amdgcn_exp2f(r2 - m_ref[qt]);
    l_part[qt] = g == 0 ? l_a[qt] : 0.0f;
    const size_t ob = ((size_t)bh * N + (q < N ? q : 0)) * D;
#pragma unroll
    for (int dt = 0; dt < G16::DT; ++dt) {
      const float4 o = q < N ? *reinterpret_cast<const float4*>(a.o_a + ob + dt * 16 + 4 * g)
                             : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
      oacc[dt][qt] = f32x4{l_a[qt] * o.x, l_a[qt] * o.y, l_a[qt] * o.z, l_a[qt] * o.w};
    }
  }
  const float log2_s = S == 128 ? 7.0f : 6.0f;
  const float log2_last = __log2f((float)(N - (nB - 1) * S));

  // T tiles (with a dummy V tile), then the pooled chunks; chunk 0 again past
  // the end, so each chunk issues one load group and the wait counts are
  // constants.
  ChunkLoader<D, NUW, CT, true> tl[NQB];     // T_i of each block: D rows of D, like a K tile
#pragma unroll
  for (int b2 = 0; b2 < NQB; ++b2) {
    const uint16_t* Tb = a.T + ((size_t)bh * nBp + min(ib0 + b2, nB - 1)) * D * D;
    loader_init(tl[b2], Tb, Tb, D, &Ks[0][0], &Vs[0][0], w, lane);
  }
  auto fetch_pooled = [&](int st, int gc) {
    const int ch = gc - NTC;
    load_chunk(ld, st, ch < nch ? ch * 32 : 0);
  };
  auto fetch_const = [&](int st, int gc) {
    if (gc < NTC) {
      load_tile<true>(tl[gc / NTT], st, (gc % NTT) * 32);
      load_tile<false>(ld, st, 0);
    } else {
      fetch_pooled(st, gc);
    }
  };
#pragma unroll
  for (int gc = 0; gc < PD; ++gc) fetch_const(gc, gc);
#pragma unroll
  for (int gc = 0; gc < NTC; ++gc) {         // chunk gc: T rows 32*(gc % NTT) .. of block gc / NTT
    wait_vmcnt_lds_idle<2 * NUW * (PD - 1)>();       // chunk gc landed
    wg_barrier();                                   // every wave's; the stage of chunk gc-1 is free
    fetch_const((gc + PD) % NST, gc + PD);
    if (gc / NTT == qb) {
      f32x4 tacc[2][2];
      qk16<D>(tacc, &Ks[gc % NST][0], koff, qop);
#pragma unroll
      for (int k2 = 0; k2 < 2; ++k2) {
        const int dt = 2 * (gc % NTT) + k2;          // rows 16*dt + 4g + r of T_i: d = e
        if (dt < G16::DT) {
#pragma unroll
          for (int qt = 0; qt < 2; ++qt)
#pragma unroll
            for (int r = 0; r < 4; ++r) oacc[dt][qt][r] = __builtin_fmaf(f1[qt], tacc[k2][qt][r], oacc[dt][qt][r]);
        }
      }
    }
  }

  const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
  const int last_ch = (nB - 1) / 32;
  // x in place of s (log2 units, relative to m_ref); returns this lane's max
  auto logits = [&](f32x4 (&x)[2][2], int ch) {
    float mx = -INFINITY;
    if (ch != last_ch) {
#pragma unroll
      for (int qt = 0; qt < 2; ++qt) {
        const float bias = log2_s - m_ref[qt];
#pragma unroll
        for (int k2 = 0; k2 < 2; ++k2)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            x[k2][qt][r] = __builtin_fmaf(x[k2][qt][r], sl2, bias);
            mx = fmaxf(mx, x[k2][qt][r]);
          }
      }
    } else {
#pragma unroll
      for (int k2 = 0; k2 < 2; ++k2)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int j = ch * 32 + k2 * 16 + 4 * g + r;
          const float lj = j >= nB ? -INFINITY : (j == nB - 1 ? log2_last : log2_s);
#pragma unroll
          for (int qt = 0; qt < 2; ++qt) {
            x[k2][qt][r] = __builtin_fmaf(x[k2][qt][r], sl2, lj - m_ref[qt]);
            mx = fmaxf(mx, x[k2][qt][r]);
          }
        }
    }
    return mx;
  };
  auto softmax_masked = [&](const f32x4 (&x)[2][2], const u32x4& mk, bf16x8 (&pop)[2]) {
#pragma unroll
    for (int qt = 0; qt < 2; ++qt) {
      u32x4 wv;
      float lsum = l_part[qt];
#pragma unroll
      for (int k2 = 0; k2 < 2; ++k2)
#pragma unroll
        for (int e = 0; e < 2; ++e) {
          const float p0 = __builtin_amdgcn_exp2f(x[k2][qt][2 * e]);
          const float p1 = __builtin_amdgcn_exp2f(x[k2][qt][2 * e + 1]);
          const unsigned u = __builtin_bit_cast(unsigned, cvt2(p0, p1)) & mk[k2 * 2 + e];
          lsum = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, u), ones, lsum, false);
          wv[k2 * 2 + e] = u;
        }
      pop[qt] = __builtin_bit_cast(bf16x8, wv);
      l_part[qt] = lsum;
    }
  };

  wait_vmcnt_lds_idle<2 * NUW * (PD - 1)>();         // pooled chunk 0 landed
  wg_barrier();
  f32x4 sacc[2][2];
  qk16<D>(sacc, &Ks[NTC % NST][0], koff, qop);
  const uint32_t* pmw = &pm[qb][0][4 * g];
  for (int ch0 = 0; ch0 < nch; ch0 += NST) {
#pragma unroll
    for (int c = 0; c < NST; ++c) {
      const int ch = ch0 + c;
      if (ch >= nch) break;
      wait_vmcnt_lds_idle<2 * NUW * (PD - 2)>();     // chunk ch+1 landed
      wg_barrier();
      fetch_pooled((NTC + c + PD) % NST, NTC + ch + PD);
      f32x4 snext[2][2];
      qk16<D>(snext, &Ks[(NTC + c + 1) % NST][0], koff, qop);
      const u32x4 mk = *reinterpret_cast<const u32x4*>(pmw + ch * 16);
      const float mxl = logits(sacc, ch);
      if (__builtin_amdgcn_ballot_w64(mxl > 8.0f) != 0) {
        // a dropped block's logit passed the reference by more than 8: move it
#pragma unroll
        for (int qt = 0; qt < 2; ++qt) {
          float mx = -INFINITY;
#pragma unroll
          for (int k2 = 0; k2 < 2; ++k2)
#pragma unroll
            for (int r = 0; r < 4; ++r) mx = fmaxf(mx, sacc[k2][qt][r]);
          mx = quad_max(mx);
          if (mx > 8.0f) {
            const float f = __builtin_amdgcn_exp2f(-mx);
            l_part[qt] *= f;
#pragma unroll
            for (int dt = 0; dt < G16::DT; ++dt)
#pragma unroll
              for (int r = 0; r < 4; ++r) oacc[dt][qt][r] *= f;
#pragma unroll
            for (int k2 = 0; k2 < 2; ++k2)
#pragma unroll
              for (int r = 0; r < 4; ++r) sacc[k2][qt][r] -= mx;
            m_ref[qt] += mx;
          }
        }
      }
      bf16x8 pop[2];
      softmax_masked(sacc, mk, pop);
      pv16<D>(pop, &Vs[(NTC + c) % NST][0], voff, oacc);
#pragma unroll
      for (int x = 0; x < 2; ++x) {
        sacc[x][0] = snext[x][0];
        sacc[x][1] = snext[x][1];
      }
    }
  }
  wait_vmcnt<0>();

  float l_tot[2];
  l_tot[0] = quad_sum(l_part[0]);
  l_tot[1] = quad_sum(l_part[1]);
  const bool has[2] = {l_tot[0] > 0.0f, l_tot[1] > 0.0f};
  store_query16<D, OUT_F32>(a.out, a.lse, (size_t)bh * N * D, (size_t)bh * N, qbase, N, oacc, l_tot, m_ref, has,
                            lane);
}

template <int D, int S>
hipError_t launch_moments_ds(const Dims& d, const RemMomentArgs& a, hipStream_t stream) {
  const int n = d.B * d.H * a.rows;
  hipLaunchKernelGGL((rem_moments_kernel<D, S>), dim3(n), dim3(256), 0, stream, a);
  return hipGetLastError();
}

template <int D, int S>
hipError_t launch_rem_attn_ds(const Dims& d, const RemAttnArgs& a, hipStream_t stream) {
  constexpr int NQB = 128 / S;
  RemAttnArgs g = a;
  g.n_rows = d.B * d.H * ((d.nB + NQB - 1) / NQB);   // workgroups
  dim3 grid(g.n_rows), block(256);
  if (d.out_f32) hipLaunchKernelGGL((rem_attn_kernel<D, S, true>), grid, block, 0, stream, g);
  else hipLaunchKernelGGL((rem_attn_kernel<D, S, false>), grid, block, 0, stream, g);
  return hipGetLastError();
}

template <int D>
hipError_t launch_weights_d(const Dims& d, const RemWeightArgs& a, hipStream_t stream) {
  const int n = d.B * d.H * ((d.nB + kRemRows - 1) / kRemRows);
  hipLaunchKernelGGL((rem_weights_kernel<D>), dim3(n), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace

int rem_padded_blocks(int nB) { return (nB + 31) / 32 * 32; }
int rem_weight_rows(int nB) { return (nB + kRemGemmRows - 1) / kRemGemmRows * kRemGemmRows; }

hipError_t launch_block_moments(const Dims& d, const RemMomentArgs& a, hipStream_t stream) {
  switch (d.D * 1000 + d.S) {
    case 64128: return launch_moments_ds<64, 128>(d, a, stream);
    case 112128: return launch_moments_ds<112, 128>(d, a, stream);
    case 128128: return launch_moments_ds<128, 128>(d, a, stream);
    case 64064: return launch_moments_ds<64, 64>(d, a, stream);
    case 112064: return launch_moments_ds<112, 64>(d, a, stream);
    case 128064: return launch_moments_ds<128, 64>(d, a, stream);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_remainder(const Dims& d, const RemWeightArgs& wa, const RemGemmArgs& ga, const RemAttnArgs& aa,
                            hipStream_t stream) {
  hipError_t e;
  switch (d.D) {
    case 64: e = launch_weights_d<64>(d, wa, stream); break;
    case 112: e = launch_weights_d<112>(d, wa, stream); break;
    case 128: e = launch_weights_d<128>(d, wa, stream); break;
    default: return hipErrorInvalidValue;
  }
  if (e != hipSuccess) return e;
  RemGemmArgs g = ga;
  g.n_wg = d.B * d.H * (g.DD / 128) * ((d.nB + kRemGemmRows - 1) / kRemGemmRows);
  hipLaunchKernelGGL(rem_gemm_kernel, dim3(g.n_wg), dim3(256), 0, stream, g);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  switch (d.D * 1000 + d.S) {
    case 64128: return launch_rem_attn_ds<64, 128>(d, aa, stream);
    case 112128: return launch_rem_attn_ds<112, 128>(d, aa, stream);
    case 128128: return launch_rem_attn_ds<128, 128>(d, aa, stream);
    case 64064: return launch_rem_attn_ds<64, 64>(d, aa, stream);
    case 112064: return launch_rem_attn_ds<112, 64>(d, aa, stream);
    case 128064: return launch_rem_attn_ds<128, 64>(d, aa, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace sva
