// Block scores and block selection ("score-based routing", Appendix A.2.2;
// the block-wise similarity of Section 4.2.2).
#include <type_traits>

#include "sva_internal.h"

namespace sva {
namespace {

__device__ __forceinline__ uint64_t order_key(double s) {
  if (s == 0.0) s = 0.0;          // -0 and +0 compare equal: give them one key
  const uint64_t b = (uint64_t)__double_as_longlong(s);
  return (b >> 63) ? ~b : (b | 0x8000000000000000ull);
}

struct SelectArgs {
  const float* q_pool;
  const float* k_pool;
  int32_t* kv_idx;
  int32_t* kv_count;
  uint8_t* mask;
  int nB, D, kmax, n_groups, n_work;
  double scale;
  int mode, k, cap, n_forced;
  double tau;
};

// ---------------------------------------------------------------------------
// Selection with the scores in registers.  A workgroup of NW waves takes
// R = NW*RW = 16 query-block rows of one (b, h) (eight waves of two rows, or
// sixteen of one; launch_select picks by block count and rule); each wave
// owns RW of them, and lane l holds
// the float64 scores of blocks j = t*64 + l (t < NT) for each of its rows.
// kbar is staged through LDS 64 blocks at a time (the next chunk is loaded
// into registers while this one is used), so every kbar row is read once per
// R query rows.  The scores of a chunk are float64 matrix products (16 rows x
// 64 keys, one 16-key tile per wave), passed through LDS to the lane-per-key
// layout of the rows' owners.
//
// Both rules end in a threshold key T and a quota: keys above T are kept, and
// of the keys equal to T the `quota` lowest block indices.
// top-k : T is the k-th largest order key, found bit by bit from the top (a
//         candidate bit stays set when at least k keys are >= the candidate,
//         counted with one ballot per register); the search stops early once
//         exactly k keys are >= the candidate.
// mass  : the forced (first-frame) blocks are kept and their softmax mass
//         counted; over the other blocks T is the largest key whose upper set
//         (keys >= T) brings the mass to tau, found bit by bit with the mass
//         of each candidate's upper set as a wave sum.  The search stops once
//         the bracket [T, T_hi) holds a single key (the block whose addition
//         crosses tau); equal keys at T are added in index order until the
//         mass reaches tau.  If that needs more blocks than the cap allows,
//         the kept blocks are the top (cap - forced) by the top-k search.
// The kept indices are written in ascending order from ballots.
__device__ __forceinline__ uint32_t lanes_below(uint64_t m) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

// Wave reductions of doubles on DPP lane moves (each half of the double moved
// by the same pattern): within rows of 16 lanes by quad and mirror
// permutations, then across the four rows by the row broadcasts; lane 63 ends
// with the result, which every lane then reads (so all lanes hold the same
// bits and control flow on it stays uniform).
template <int CTRL, int ROWS>
__device__ __forceinline__ double dpp_d(double x, double ident) {
  const long long xi = __double_as_longlong(x), ii = __double_as_longlong(ident);
  const int lo = __builtin_amdgcn_update_dpp((int)ii, (int)xi, CTRL, ROWS, 0xf, false);
  const int hi = __builtin_amdgcn_update_dpp((int)(ii >> 32), (int)(xi >> 32), CTRL, ROWS, 0xf, false);
  return __longlong_as_double((long long)(((unsigned long long)(unsigned)hi << 32) | (unsigned)lo));
}

__device__ __forceinline__ double lane63_d(double x) {
  const long long xi = __double_as_longlong(x);
  const int lo = __builtin_amdgcn_readlane((int)xi, 63);
  const int hi = __builtin_amdgcn_readlane((int)(xi >> 32), 63);
  return __longlong_as_double((long long)(((unsigned long long)(unsigned)hi << 32) | (unsigned)lo));
}

__device__ __forceinline__ double wave_sum_d(double v) {
  v += dpp_d<0xB1, 0xf>(v, 0.0);     // quad_perm 1,0,3,2
  v += dpp_d<0x4E, 0xf>(v, 0.0);     // quad_perm 2,3,0,1
  v += dpp_d<0x141, 0xf>(v, 0.0);    // row_half_mirror
  v += dpp_d<0x140, 0xf>(v, 0.0);    // row_mirror
  v += dpp_d<0x142, 0xa>(v, 0.0);    // row_bcast:15
  v += dpp_d<0x143, 0xc>(v, 0.0);    // row_bcast:31
  return lane63_d(v);
}

__device__ __forceinline__ double wave_max_d(double v) {
  v = fmax(v, dpp_d<0xB1, 0xf>(v, -INFINITY));
  v = fmax(v, dpp_d<0x4E, 0xf>(v, -INFINITY));
  v = fmax(v, dpp_d<0x141, 0xf>(v, -INFINITY));
  v = fmax(v, dpp_d<0x140, 0xf>(v, -INFINITY));
  v = fmax(v, dpp_d<0x142, 0xa>(v, -INFINITY));
  v = fmax(v, dpp_d<0x143, 0xc>(v, -INFINITY));
  return lane63_d(v);
}

// k-th largest key (k >= 1, at least k keys > 0); returns T and the number of
// keys equal to T to keep.
template <int NT>
__device__ __forceinline__ void kth_key(const uint64_t (&key)[NT], uint32_t k, uint64_t& T_out,
                                        uint32_t& quota) {
  uint64_t T = 0;
  for (int b = 63; b >= 0; --b) {
    const uint64_t cand = T | (1ull << b);
    uint32_t cnt = 0;
#pragma unroll
    for (int t = 0; t < NT; ++t) cnt += __builtin_popcountll(__builtin_amdgcn_ballot_w64(key[t] >= cand));
    if (cnt >= k) T = cand;
    if (cnt == k) break;
  }
  uint32_t above = 0;
#pragma unroll
  for (int t = 0; t < NT; ++t) above += __builtin_popcountll(__builtin_amdgcn_ballot_w64(key[t] > T));
  T_out = T;
  quota = k - above;
}

// OCC: waves per SIMD the register allocation must allow (4: two workgroups
// of eight waves per CU, which overlaps one workgroup's scores with the
// other's searches)
template <int NT, int RW, int NW, bool MASS, int OCC>
__global__ __launch_bounds__(NW * 64, OCC) void select_reg_kernel(SelectArgs a) {
  constexpr int NTH = NW * 64;       // threads
  constexpr int R = NW * RW;         // rows of the workgroup (16)
  static_assert(R == 16, "the score tiles hold 16 rows");
  constexpr int KP = 132;            // kbar row pitch in LDS (floats): conflict-free b128 reads
  constexpr int QP = 130;            // qbar row pitch in LDS (doubles): the 16 rows of a read group on distinct banks
  constexpr int SP = 66;             // score staging row pitch (doubles)
  typedef double f64x4 __attribute__((ext_vector_type(4)));
  __shared__ __attribute__((aligned(16))) double qs[16 * QP];
  __shared__ __attribute__((aligned(16))) float ks[64 * KP];
  __shared__ __attribute__((aligned(16))) double ss[16 * SP];

  const int nB = a.nB, D = a.D;
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int work = xcd_remap(blockIdx.x, a.n_work);
  const int bh = work / a.n_groups;
  const int i0 = (work - bh * a.n_groups) * R;
  const float* qsrc = a.q_pool + (size_t)bh * nB * D;
  const float* ksrc = a.k_pool + (size_t)bh * nB * D;

  // qbar of the 16 rows in float64
  for (int t = threadIdx.x; t < 16 * D; t += NTH) {
    const int g = t / D, d = t - g * D;
    qs[g * QP + d] = (i0 + g < nB) ? (double)qsrc[(size_t)(i0 + g) * D + d] : 0.0;
  }

  // kbar chunk: 64 rows x D floats = 16*D float4, at most NPRE per thread (D <= 128)
  constexpr int NPRE = 2048 / NTH;
  const int nf4 = 16 * D;
  const int d4 = D / 4;
  float4 pre[NPRE];
  auto load_chunk = [&](int c) {
#pragma unroll
    for (int u = 0; u < NPRE; ++u) {
      const int e = threadIdx.x + u * NTH;
      const int r = e / d4, c4 = e - r * d4;
      const int j = c * 64 + r;
      pre[u] = (e < nf4 && j < nB) ? *reinterpret_cast<const float4*>(ksrc + (size_t)j * D + c4 * 4)
                                   : make_float4(0.f, 0.f, 0.f, 0.f);
    }
  };
  auto store_chunk = [&]() {
#pragma unroll
    for (int u = 0; u < NPRE; ++u) {
      const int e = threadIdx.x + u * NTH;
      const int r = e / d4, c4 = e - r * d4;
      if (e < nf4) *reinterpret_cast<float4*>(ks + r * KP + c4 * 4) = pre[u];
    }
  };

  // Scores on mfma_f64_16x16x4f64: wave w < 4 forms the 16 x 16 tile of keys
  // c*64 + 16w + 0..15 against the 16 rows, S^T = Kbar Qbar^T (with eight
  // waves the other four share the SIMDs and wait).    Lane
  // l = 16g + j feeds key j (A) and row j (B) at d = g*DG + s for step s, so
  // the four lane groups split d into four runs of DG; the result puts key
  // g + 4r of row j in its register r.  The fp32 products are exact in
  // float64, so only the sums round (in an order free of consequence: the
  // oracle's scores are a library matrix product).
  const int DG = D >> 2;             // 16, 28 or 32: a multiple of 4
  const int j16 = lane & 15, g4 = lane >> 4;
  const float* ka = ks + ((w & 3) * 16 + j16) * KP + g4 * DG;
  const double* qb = qs + j16 * QP + g4 * DG;

  double sc[RW][NT];
  load_chunk(0);
#pragma unroll
  for (int c = 0; c < NT; ++c) {
    __syncthreads();                   // the previous chunk and its scores are consumed (q rows written)
    store_chunk();
    __syncthreads();
    if (c + 1 < NT && (c + 1) * 64 < nB) load_chunk(c + 1);
    if (c * 64 < nB && w < 4) {
      f64x4 acc0 = {0.0, 0.0, 0.0, 0.0}, acc1 = {0.0, 0.0, 0.0, 0.0};
      for (int s = 0; s < DG; s += 4) {
        const float4 kv = *reinterpret_cast<const float4*>(ka + s);
        const double2 q01 = *reinterpret_cast<const double2*>(qb + s);
        const double2 q23 = *reinterpret_cast<const double2*>(qb + s + 2);
        acc0 = __builtin_amdgcn_mfma_f64_16x16x4f64((double)kv.x, q01.x, acc0, 0, 0, 0);
        acc1 = __builtin_amdgcn_mfma_f64_16x16x4f64((double)kv.y, q01.y, acc1, 0, 0, 0);
        acc0 = __builtin_amdgcn_mfma_f64_16x16x4f64((double)kv.z, q23.x, acc0, 0, 0, 0);
        acc1 = __builtin_amdgcn_mfma_f64_16x16x4f64((double)kv.w, q23.y, acc1, 0, 0, 0);
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) ss[j16 * SP + w * 16 + g4 + 4 * r] = acc0[r] + acc1[r];
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < RW; ++r) sc[r][c] = (c * 64 < nB) ? a.scale * ss[(w * RW + r) * SP + lane] : 0.0;
  }

  // one row at a time: the row index must be a compile-time constant so the
  // score registers stay registers
  auto select_row = [&](auto rc) {
    constexpr int r = decltype(rc)::value;
    const int i = i0 + w * RW + r;
    if (i >= nB) return;               // uniform: rows past the head's last block
    const size_t row = (size_t)bh * nB + i;
    const int nF = MASS ? a.n_forced : 0;
    uint64_t key[NT];
    // every valid key is > 0 (order_key maps -inf to 0x000F...); forced and
    // padding blocks get key 0 and never pass a candidate
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const int j = t * 64 + lane;
      key[t] = (j < nB && j >= nF) ? order_key(sc[r][t]) : 0ull;
    }
    uint64_t T = 0;
    uint32_t quota = 0;
    if constexpr (!MASS) {
      kth_key<NT>(key, (uint32_t)a.k, T, quota);
    } else {
      // softmax weights over all blocks, as the definition: exp(s - max) / sum
      double mx = -INFINITY;
#pragma unroll
      for (int t = 0; t < NT; ++t)
        if (t * 64 + lane < nB) mx = fmax(mx, sc[r][t]);
      mx = wave_max_d(mx);
      double p[NT];
      double z = 0.0;
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        p[t] = (t * 64 + lane < nB) ? exp(sc[r][t] - mx) : 0.0;
        z += p[t];
      }
      z = wave_sum_d(z);
      double mf = 0.0, mo = 0.0;
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        p[t] = p[t] / z;
        if (t * 64 + lane < nF) mf += p[t];
        else mo += p[t];
      }
      mf = wave_sum_d(mf);
      mo = wave_sum_d(mo);
      const int M = nB - nF;             // blocks that may be added
      const int budget = a.cap - nF;
      int n_add;                         // blocks the mass rule adds (before the cap)
      if (mf >= a.tau || budget <= 0 || M <= 0) {
        n_add = 0;
      } else if (mf + mo < a.tau) {
        n_add = M;                       // tau is out of reach: everything, up to the cap
        T = 0;
        quota = 0;
      } else {
        // bracket: mass(upper set of T) >= tau > mass(upper set of T_hi)
        uint64_t T_lo = 0;
        uint32_t cnt_lo = (uint32_t)M, cnt_hi = 0;
        double mass_hi = mf;
        bool single = false;
        for (int b = 63; b >= 0; --b) {
          const uint64_t cand = T_lo | (1ull << b);
          uint32_t cnt = 0;
          double part = 0.0;
#pragma unroll
          for (int t = 0; t < NT; ++t) {
            const bool ge = key[t] >= cand;
            cnt += __builtin_popcountll(__builtin_amdgcn_ballot_w64(ge));
            part += ge ? p[t] : 0.0;
          }
          const double m = mf + wave_sum_d(part);
          if (m >= a.tau) { T_lo = cand; cnt_lo = cnt; }
          else { cnt_hi = cnt; mass_hi = m; }
          if (cnt_lo - cnt_hi == 1) { single = true; break; }
        }
        if (single) {
          // the one key in [T_lo, T_hi) is the block whose addition crosses
          // tau; the (non-zero) keys >= T_lo are it and the cnt_hi keys above
          // it, so it is their minimum
          uint64_t mn = ~0ull;
#pragma unroll
          for (int t = 0; t < NT; ++t)
            if (key[t] != 0 && key[t] >= T_lo && key[t] < mn) mn = key[t];
#pragma unroll
          for (int off = 32; off > 0; off >>= 1) {
            const uint64_t o = __shfl_xor(mn, off, 64);
            mn = o < mn ? o : mn;
          }
          T = mn;
          quota = 1;
          n_add = (int)cnt_hi + 1;
        } else {
          // T_lo is an exact key held by several blocks: add them in index
          // order until the mass reaches tau
          T = T_lo;
          double run = mass_hi;
          uint32_t taken = 0;
          bool done = false;
#pragma unroll
          for (int t = 0; t < NT; ++t) {
            const bool eq = key[t] == T;
            const uint64_t em = __builtin_amdgcn_ballot_w64(eq);
            if (!done && em != 0) {       // uniform
              double v = eq ? p[t] : 0.0;
              for (int off = 1; off < 64; off <<= 1) {
                const double o = __shfl_up(v, off, 64);
                if (lane >= off) v += o;
              }
              // first tie lane whose running mass reaches tau
              const uint64_t hit = __builtin_amdgcn_ballot_w64(eq && run + v >= a.tau);
              if (hit != 0) {
                const int l0 = __builtin_ctzll(hit);
                taken += __builtin_popcountll(em & ((2ull << l0) - 1));
                done = true;
              } else {
                taken += __builtin_popcountll(em);
                run += __shfl(v, 63, 64);
              }
            }
          }
          quota = taken;
          n_add = (int)cnt_hi + (int)taken;
        }
      }
      if (n_add > budget) {
        // the cap binds: the best (cap - forced) blocks
        kth_key<NT>(key, (uint32_t)budget, T, quota);
      } else if (n_add == 0) {
        T = ~0ull;                       // nothing but the forced blocks
        quota = 0;
      }
    }
    int32_t* out = a.kv_idx + row * (size_t)a.kmax;
    uint8_t* mrow = a.mask ? a.mask + row * (size_t)nB : nullptr;
    uint32_t base = 0, ties = 0;
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const int j = t * 64 + lane;
      const bool eq = key[t] != 0 && key[t] == T;
      const uint64_t em = __builtin_amdgcn_ballot_w64(eq);
      const uint32_t my_tie = ties + lanes_below(em);
      const bool forced = j < nF && j < nB;
      const bool kp = forced || (key[t] != 0 && key[t] > T) || (eq && my_tie < quota);
      const uint64_t km = __builtin_amdgcn_ballot_w64(kp);
      const uint32_t pos = base + lanes_below(km);
      if (kp && pos < (uint32_t)a.kmax) out[pos] = j;
      if (mrow && j < nB) mrow[j] = kp ? 1 : 0;
      base += __builtin_popcountll(km);
      ties += __builtin_popcountll(em);
    }
    for (int p = (int)base + lane; p < a.kmax; p += 64) out[p] = -1;
    if (lane == 0) a.kv_count[row] = (int32_t)min(base, (uint32_t)a.kmax);
  };
  select_row(std::integral_constant<int, 0>{});
  if constexpr (RW > 1) select_row(std::integral_constant<int, 1>{});
  if constexpr (RW > 2) select_row(std::integral_constant<int, 2>{});
  if constexpr (RW > 3) select_row(std::integral_constant<int, 3>{});
}

template <int NT, int RW, int NW, bool MASS, int OCC = 1>
hipError_t launch_reg(SelectArgs a, int B, int H, hipStream_t stream) {
  a.n_groups = (a.nB + NW * RW - 1) / (NW * RW);
  a.n_work = B * H * a.n_groups;
  hipLaunchKernelGGL((select_reg_kernel<NT, RW, NW, MASS, OCC>), dim3(a.n_work), dim3(NW * 64), 0, stream, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_select(const Dims& d, const SelectRule& r, const float* q_pool,
                         const float* k_pool, int kmax, int32_t* kv_idx, int32_t* kv_count,
                         uint8_t* mask, hipStream_t stream) {
  SelectArgs a;
  a.q_pool = q_pool;
  a.k_pool = k_pool;
  a.kv_idx = kv_idx;
  a.kv_count = kv_count;
  a.mask = mask;
  a.nB = d.nB;
  a.D = d.D;
  a.kmax = kmax;
  a.scale = (double)d.scale;
  a.mode = r.mode;
  a.k = r.k;
  a.cap = r.cap;
  a.n_forced = r.n_forced;
  a.tau = r.tau;
  // nB <= SVA_SELECT_MAX_BLOCKS (2048) and D <= 128 are checked by the caller
  const int nt = (d.nB + 63) / 64;
  // Shapes by block count (chunks of 64 blocks, nt) and rule, each measured
  // against its neighbours:
  // - eight waves of two rows: 7-37% faster than four of four rows at every
  //   block count (more waves for the latency-bound threshold search);
  // - a chunk count fitted to nt: 0.339 -> 0.326 ms at the 64B-class layer
  //   (14 chunks instead of 16);
  // - the mass rule's search (a wave sum per candidate bit) gains from one
  //   row per wave: 0.597 -> 0.533 ms at the 22B-class layer; the top-k
  //   search loses (0.339 -> 0.395 ms at the 64B-class layer);
  // - at 17-20 chunks, top-k holds two workgroups per CU only with the
  //   registers capped at 128 (a few values spill): 0.83 -> 0.555 ms on the
  //   CFG-sweep layer (19 chunks), against 0.646 ms for sixteen waves of one
  //   row and one workgroup per CU.
  const bool mass = a.mode != 0;
  if (nt <= 1) return mass ? launch_reg<1, 2, 8, true>(a, d.B, d.H, stream) : launch_reg<1, 2, 8, false>(a, d.B, d.H, stream);
  if (nt <= 2) return mass ? launch_reg<2, 2, 8, true>(a, d.B, d.H, stream) : launch_reg<2, 2, 8, false>(a, d.B, d.H, stream);
  if (nt <= 4) return mass ? launch_reg<4, 2, 8, true>(a, d.B, d.H, stream) : launch_reg<4, 2, 8, false>(a, d.B, d.H, stream);
  if (nt <= 8) return mass ? launch_reg<8, 2, 8, true>(a, d.B, d.H, stream) : launch_reg<8, 2, 8, false>(a, d.B, d.H, stream);
  if (mass) {
    if (nt <= 16) return launch_reg<16, 1, 16, true>(a, d.B, d.H, stream);
    if (nt <= 20) return launch_reg<20, 1, 16, true>(a, d.B, d.H, stream);
    if (nt <= 24) return launch_reg<24, 2, 8, true>(a, d.B, d.H, stream);
    if (nt <= 32) return launch_reg<32, 2, 8, true>(a, d.B, d.H, stream);
  } else {
    if (nt <= 12) return launch_reg<12, 2, 8, false>(a, d.B, d.H, stream);
    if (nt <= 14) return launch_reg<14, 2, 8, false>(a, d.B, d.H, stream);
    if (nt <= 16) return launch_reg<16, 2, 8, false>(a, d.B, d.H, stream);
    if (nt <= 20) return launch_reg<20, 2, 8, false, 4>(a, d.B, d.H, stream);
    if (nt <= 24) return launch_reg<24, 1, 16, false>(a, d.B, d.H, stream);
    if (nt <= 32) return launch_reg<32, 2, 8, false>(a, d.B, d.H, stream);
  }
  return hipErrorInvalidValue;
}

}  // namespace sva
