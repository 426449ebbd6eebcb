// Block scores and block selection ("score-based routing", Appendix A.2.2;
// the block-wise similarity of Section 4.2.2).
//
// One workgroup of 4 waves handles 4 consecutive query-block rows of one
// (b, h).  Phase 1 computes the 4 x nB score tile s[i, j] = c * <qbar_i, kbar_j>
// in float64 into LDS: kbar is streamed through LDS in chunks of 64 blocks with
// coalesced loads, so each kbar row is read once per 4 query rows.  The fp32
// products are exact in float64, so only the float64 sum rounds.
//
// Phase 2 gives each wave one row:
//   top-k: a radix select over order-preserving 64-bit keys of the float64
//          scores (8 passes of 8-bit digits, histogram in LDS) finds the k-th
//          largest key T and how many elements equal to T are still needed;
//          those ties are taken in ascending block order.
//   mass : softmax weights in float64; the non-forced blocks are sorted by
//          (score desc, index asc) with a bitonic network in LDS; a prefix sum
//          over that order finds the first point where the forced mass plus the
//          added mass reaches tau, bounded by the cap.
// Both finish with an ordered compaction (wave prefix sums) that writes the
// kept indices in ascending order, pads with -1, and writes the optional mask.
#include "sva_internal.h"

namespace sva {
namespace {

constexpr int kRows = 4;          // query-block rows per workgroup (one per wave)
constexpr int kThreads = 256;
constexpr int kChunkJ = 64;       // kbar rows staged per phase-1 chunk

__device__ __forceinline__ uint64_t order_key(double s) {
  if (s == 0.0) s = 0.0;          // -0 and +0 compare equal: give them one key
  const uint64_t b = (uint64_t)__double_as_longlong(s);
  return (b >> 63) ? ~b : (b | 0x8000000000000000ull);
}

__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t v) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const uint32_t o = __shfl_up(v, off, 64);
    if (lane >= off) v += o;
  }
  return v;
}

__device__ __forceinline__ double wave_incl_scan_f64(double v) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const double o = __shfl_up(v, off, 64);
    if (lane >= off) v += o;
  }
  return v;
}

__device__ __forceinline__ double wave_max_f64(double v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v = fmax(v, __shfl_xor(v, off, 64));
  return v;
}

__device__ __forceinline__ double wave_sum_f64(double v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

__device__ __forceinline__ int wave_min_i32(int v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v = min(v, __shfl_xor(v, off, 64));
  return v;
}

// Orders this wave's LDS writes before its later LDS reads of other lanes'
// data (LDS requests of one wave are served in issue order; this keeps the
// compiler from moving the reads up).
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

struct SelectArgs {
  const float* q_pool;
  const float* k_pool;
  int32_t* kv_idx;
  int32_t* kv_count;
  uint8_t* mask;
  int nB, D, kmax, n_groups, n_work;
  double scale;
  int mode, k, cap, n_forced, sort_n;  // sort_n: power of two >= nB - n_forced
  double tau;
};

// Writes one row's kept flags (given by keep(j)) in ascending order.
template <typename KeepFn>
__device__ void compact_row(const SelectArgs& a, size_t row, int lane, KeepFn keep) {
  const int nB = a.nB;
  const int per = (nB + 63) / 64;
  const int j0 = min(nB, lane * per);
  const int j1 = min(nB, j0 + per);
  uint32_t n = 0;
  for (int j = j0; j < j1; ++j) n += keep(j) ? 1u : 0u;
  const uint32_t incl = wave_incl_scan(n);
  uint32_t pos = incl - n;
  const uint32_t total = __shfl(incl, 63, 64);
  int32_t* out = a.kv_idx + row * (size_t)a.kmax;
  uint8_t* mrow = a.mask ? a.mask + row * (size_t)nB : nullptr;
  for (int j = j0; j < j1; ++j) {
    const bool kp = keep(j);
    if (kp) {
      if (pos < (uint32_t)a.kmax) out[pos] = j;   // never past the row, whatever the flags say
      ++pos;
    }
    if (mrow) mrow[j] = kp ? 1 : 0;
  }
  for (int p = (int)total + lane; p < a.kmax; p += 64) out[p] = -1;
  if (lane == 0) a.kv_count[row] = (int32_t)min(total, (uint32_t)a.kmax);
}

__global__ __launch_bounds__(kThreads) void select_kernel(SelectArgs a) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  const int nB = a.nB, D = a.D;
  double* scores = reinterpret_cast<double*>(smem);                 // [kRows][nB]
  unsigned char* area = smem + (size_t)kRows * nB * sizeof(double);  // phase scratch

  const int work = xcd_remap(blockIdx.x, a.n_work);
  const int bh = work / a.n_groups;
  const int i0 = (work - bh * a.n_groups) * kRows;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = tid >> 6;

  // ---------------- phase 1: score tile ----------------
  {
    float* qt = reinterpret_cast<float*>(area);                      // [kRows][D]
    float* kt = qt + kRows * D;                                      // [kChunkJ][D+1]
    const float* qsrc = a.q_pool + ((size_t)bh * nB) * D;
    const float* ksrc = a.k_pool + ((size_t)bh * nB) * D;
    for (int t = tid; t < kRows * D; t += kThreads) {
      const int g = t / D, d = t - g * D;
      qt[t] = (i0 + g < nB) ? qsrc[(size_t)(i0 + g) * D + d] : 0.0f;
    }
    const int g = tid / kChunkJ;
    const int jj = tid - g * kChunkJ;
    for (int j0 = 0; j0 < nB; j0 += kChunkJ) {
      __syncthreads();
      const int rows = min(kChunkJ, nB - j0);
      for (int t = tid; t < rows * D; t += kThreads) {
        const int r = t / D, d = t - r * D;
        kt[r * (D + 1) + d] = ksrc[(size_t)(j0 + r) * D + d];
      }
      __syncthreads();
      if (jj < rows) {
        const float* qa = qt + g * D;
        const float* ka = kt + jj * (D + 1);
        double acc = 0.0;
        for (int d = 0; d < D; ++d) acc = fma((double)qa[d], (double)ka[d], acc);
        scores[g * nB + j0 + jj] = a.scale * acc;
      }
    }
    __syncthreads();
  }

  const int i = i0 + w;
  const bool row_ok = i < nB;
  const size_t row = (size_t)bh * nB + (row_ok ? i : 0);
  const double* sc = scores + w * nB;

  if (a.mode == 0) {
    // ---------------- top-k: radix select ----------------
    uint32_t* hist = reinterpret_cast<uint32_t*>(area) + w * 256;
    uint64_t prefix = 0;
    uint32_t need = (uint32_t)a.k;   // rank (1-based) of the wanted key among the rest
    for (int pass = 0; pass < 8; ++pass) {
      const int shift = 56 - 8 * pass;
      for (int b = lane; b < 256; b += 64) hist[b] = 0;
      __syncthreads();
      if (row_ok) {
        for (int j = lane; j < nB; j += 64) {
          const uint64_t key = order_key(sc[j]);
          if (pass == 0 || (key >> (shift + 8)) == prefix)
            atomicAdd(&hist[(key >> shift) & 255u], 1u);
        }
      }
      __syncthreads();
      // lane l owns bins 255-4l .. 252-4l (descending); scan counts from the top
      uint32_t c[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) c[e] = hist[255 - 4 * lane - e];
      const uint32_t tot = c[0] + c[1] + c[2] + c[3];
      const uint32_t incl = wave_incl_scan(tot);
      const uint32_t excl = incl - tot;
      const bool mine = excl < need && need <= incl;
      int digit = 0;
      uint32_t above = excl;
      if (mine) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          if (above + c[e] >= need) { digit = 255 - 4 * lane - e; break; }
          above += c[e];
        }
      }
      const uint64_t bal = __ballot(mine);
      const int src = bal ? (__ffsll((unsigned long long)bal) - 1) : 0;
      digit = __shfl(digit, src, 64);
      above = __shfl(above, src, 64);
      prefix = (prefix << 8) | (uint64_t)digit;
      need -= above;
    }
    const uint64_t T = prefix;
    unsigned char* flags = reinterpret_cast<unsigned char*>(area) + kRows * 256 * sizeof(uint32_t) +
                           (size_t)w * nB;
    if (row_ok) {
      // keys above T are kept; of the keys equal to T, the `need` lowest indices
      const int per = (nB + 63) / 64;
      const int j0 = min(nB, lane * per), j1 = min(nB, j0 + per);
      uint32_t neq = 0;
      for (int j = j0; j < j1; ++j) neq += (order_key(sc[j]) == T) ? 1u : 0u;
      uint32_t tie_rank = wave_incl_scan(neq) - neq;   // ties in lower lanes' ranges
      for (int j = j0; j < j1; ++j) {
        const uint64_t key = order_key(sc[j]);
        bool kp = key > T;
        if (key == T) kp = (tie_rank++ < need);
        flags[j] = kp ? 1 : 0;
      }
      wave_lds_sync();
      compact_row(a, row, lane, [&](int j) -> bool { return flags[j] != 0; });
    }
  } else {
    // ---------------- cumulative mass ----------------
    const int nF = a.n_forced;
    const int M = nB - nF;
    const int P = a.sort_n;
    uint64_t* skey = reinterpret_cast<uint64_t*>(area) + (size_t)w * P;
    uint16_t* sidx = reinterpret_cast<uint16_t*>(reinterpret_cast<uint64_t*>(area) + (size_t)kRows * P) +
                     (size_t)w * P;
    unsigned char* flags = reinterpret_cast<unsigned char*>(
                               reinterpret_cast<uint16_t*>(reinterpret_cast<uint64_t*>(area) +
                                                           (size_t)kRows * P) + (size_t)kRows * P) +
                           (size_t)w * nB;

    double mx = -INFINITY;
    for (int j = lane; j < nB; j += 64) mx = fmax(mx, sc[j]);
    mx = wave_max_f64(mx);
    double z = 0.0;
    for (int j = lane; j < nB; j += 64) z += exp(sc[j] - mx);
    z = wave_sum_f64(z);
    const double inv_z = 1.0 / z;
    double mf = 0.0;
    for (int j = lane; j < nF; j += 64) mf += exp(sc[j] - mx) * inv_z;
    mf = wave_sum_f64(mf);

    for (int t = lane; t < P; t += 64) {
      if (t < M) { skey[t] = order_key(sc[nF + t]); sidx[t] = (uint16_t)(nF + t); }
      else { skey[t] = 0; sidx[t] = 0xFFFF; }
    }
    for (int j = lane; j < nB; j += 64) flags[j] = (j < nF) ? 1 : 0;
    __syncthreads();
    // bitonic sort, final order: key descending, index ascending
    for (int size = 2; size <= P; size <<= 1) {
      for (int stride = size >> 1; stride > 0; stride >>= 1) {
        for (int t = lane; t < P / 2; t += 64) {
          const int lo = 2 * t - (t & (stride - 1));
          const int hi = lo + stride;
          const bool desc = (lo & size) == 0;   // this run ends up "before" order
          const uint64_t ka = skey[lo], kb = skey[hi];
          const uint16_t ia = sidx[lo], ib = sidx[hi];
          // "a before b" in the final order
          const bool a_first = (ka > kb) || (ka == kb && ia < ib);
          if (a_first != desc) {
            skey[lo] = kb; skey[hi] = ka;
            sidx[lo] = ib; sidx[hi] = ia;
          }
        }
        __syncthreads();
      }
    }
    if (row_ok) {
      int n_add = 0;
      const int budget = a.cap - nF;
      if (mf < a.tau && budget > 0) {
        const int L = min(M, budget);
        const int per = (L + 63) / 64;
        const int t0 = min(L, lane * per), t1 = min(L, t0 + per);
        double part = 0.0;
        for (int t = t0; t < t1; ++t) part += exp(sc[sidx[t]] - mx) * inv_z;
        double m = mf + (wave_incl_scan_f64(part) - part);
        int first = L;   // position of the first block whose addition reaches tau
        for (int t = t0; t < t1; ++t) {
          m += exp(sc[sidx[t]] - mx) * inv_z;
          if (m >= a.tau) { first = t; break; }
        }
        first = wave_min_i32(first);
        n_add = (first < L) ? first + 1 : L;
      }
      for (int t = lane; t < n_add; t += 64) flags[sidx[t]] = 1;
      wave_lds_sync();
      compact_row(a, row, lane, [&](int j) -> bool { return flags[j] != 0; });
    }
  }
}

// ---------------------------------------------------------------------------
// Top-k with the scores in registers.  A workgroup (4 waves) takes R = 4*RW
// query-block rows of one (b, h); each wave owns RW of them, and lane l holds
// the float64 scores of blocks j = t*64 + l (t < NT) for each of its rows.
// kbar is staged through LDS 64 blocks at a time (the next chunk is loaded
// into registers while this one is used), so every kbar row is read once per
// R query rows; each score is the same sequential float64 fma chain over d as
// in select_kernel, so both give identical bits.
// The threshold T is found bit by bit from the top: a candidate bit stays set
// when at least k keys are >= the candidate (counted with one ballot per
// register); the search ends at the k-th largest key, or earlier once exactly
// k keys are >= the candidate.  Keys above T are kept, and of the keys equal to
// T the k - #above lowest block indices; the kept indices are written in
// ascending order from ballots.
template <int NT, int RW>
__global__ __launch_bounds__(kThreads) void topk_kernel(SelectArgs a) {
  constexpr int R = 4 * RW;
  constexpr int KP = 132;            // kbar row pitch in LDS (floats): conflict-free b128 reads
  constexpr int QP = 128;            // qbar row pitch in LDS (doubles)
  __shared__ __attribute__((aligned(16))) double qs[R * QP];
  __shared__ __attribute__((aligned(16))) float ks[64 * KP];

  const int nB = a.nB, D = a.D;
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int work = xcd_remap(blockIdx.x, a.n_work);
  const int bh = work / a.n_groups;
  const int i0 = (work - bh * a.n_groups) * R;
  const float* qsrc = a.q_pool + (size_t)bh * nB * D;
  const float* ksrc = a.k_pool + (size_t)bh * nB * D;

  for (int t = threadIdx.x; t < R * D; t += kThreads) {
    const int g = t / D, d = t - g * D;
    qs[g * QP + d] = (i0 + g < nB) ? (double)qsrc[(size_t)(i0 + g) * D + d] : 0.0;
  }

  // kbar chunk: 64 rows x D floats = 16*D float4, at most 8 per thread (D <= 128)
  const int nf4 = 16 * D;
  const int d4 = D / 4;
  float4 pre[8];
  auto load_chunk = [&](int c) {
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int e = threadIdx.x + u * kThreads;
      const int r = e / d4, c4 = e - r * d4;
      const int j = c * 64 + r;
      pre[u] = (e < nf4 && j < nB) ? *reinterpret_cast<const float4*>(ksrc + (size_t)j * D + c4 * 4)
                                   : make_float4(0.f, 0.f, 0.f, 0.f);
    }
  };
  auto store_chunk = [&]() {
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int e = threadIdx.x + u * kThreads;
      const int r = e / d4, c4 = e - r * d4;
      if (e < nf4) *reinterpret_cast<float4*>(ks + r * KP + c4 * 4) = pre[u];
    }
  };

  double sc[RW][NT];
  load_chunk(0);
#pragma unroll
  for (int c = 0; c < NT; ++c) {
    __syncthreads();                   // the previous chunk is consumed (q rows written)
    store_chunk();
    __syncthreads();
    if (c + 1 < NT && (c + 1) * 64 < nB) load_chunk(c + 1);
    double acc[RW];
#pragma unroll
    for (int r = 0; r < RW; ++r) acc[r] = 0.0;
    if (c * 64 < nB) {
      const float* krow = ks + lane * KP;
      const double* qrow = qs + (w * RW) * QP;
      for (int d = 0; d < D; d += 4) {
        const float4 kv = *reinterpret_cast<const float4*>(krow + d);
        const double k0 = kv.x, k1 = kv.y, k2 = kv.z, k3 = kv.w;
#pragma unroll
        for (int r = 0; r < RW; ++r) {
          const double2 qa = *reinterpret_cast<const double2*>(qrow + r * QP + d);
          const double2 qb = *reinterpret_cast<const double2*>(qrow + r * QP + d + 2);
          double x = fma(qa.x, k0, acc[r]);
          x = fma(qa.y, k1, x);
          x = fma(qb.x, k2, x);
          acc[r] = fma(qb.y, k3, x);
        }
      }
    }
#pragma unroll
    for (int r = 0; r < RW; ++r) sc[r][c] = a.scale * acc[r];
  }

  const uint32_t k = (uint32_t)a.k;
#pragma unroll
  for (int r = 0; r < RW; ++r) {
    const int i = i0 + w * RW + r;
    if (i >= nB) break;                // uniform: rows past the head's last block
    const size_t row = (size_t)bh * nB + i;
    uint64_t key[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) key[t] = (t * 64 + lane < nB) ? order_key(sc[r][t]) : 0ull;
    // every valid key is > 0 (order_key maps -inf to 0x000F...), so T > 0.
    // Once exactly k keys are >= the candidate they are the top k (equal keys
    // cannot straddle it) and the search stops with T = candidate.
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
    const uint32_t need = k - above;   // keys equal to T still to take, lowest indices first
    int32_t* out = a.kv_idx + row * (size_t)a.kmax;
    uint8_t* mrow = a.mask ? a.mask + row * (size_t)nB : nullptr;
    uint32_t base = 0, ties = 0;
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const int j = t * 64 + lane;
      const bool eq = key[t] == T;
      const uint64_t em = __builtin_amdgcn_ballot_w64(eq);
      const uint32_t my_tie = ties + __builtin_amdgcn_mbcnt_hi((uint32_t)(em >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)em, 0u));
      const bool kp = key[t] > T || (eq && my_tie < need);
      const uint64_t km = __builtin_amdgcn_ballot_w64(kp);
      const uint32_t pos = base + __builtin_amdgcn_mbcnt_hi((uint32_t)(km >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)km, 0u));
      if (kp && pos < (uint32_t)a.kmax) out[pos] = j;
      if (mrow && j < nB) mrow[j] = kp ? 1 : 0;
      base += __builtin_popcountll(km);
      ties += __builtin_popcountll(em);
    }
    for (int p = (int)base + lane; p < a.kmax; p += 64) out[p] = -1;
    if (lane == 0) a.kv_count[row] = (int32_t)min(base, (uint32_t)a.kmax);
  }
}

template <int NT, int RW>
hipError_t launch_topk(SelectArgs a, int B, int H, hipStream_t stream) {
  a.n_groups = (a.nB + 4 * RW - 1) / (4 * RW);
  a.n_work = B * H * a.n_groups;
  hipLaunchKernelGGL((topk_kernel<NT, RW>), dim3(a.n_work), dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace

size_t select_smem_bytes(int nB, int D, int mode, int sort_n) {
  const size_t scores = (size_t)kRows * nB * sizeof(double);
  const size_t p1 = (size_t)kRows * D * sizeof(float) + (size_t)kChunkJ * (D + 1) * sizeof(float);
  size_t p2;
  if (mode == 0) {
    p2 = (size_t)kRows * 256 * sizeof(uint32_t) + (size_t)kRows * nB;
  } else {
    p2 = (size_t)kRows * sort_n * (sizeof(uint64_t) + sizeof(uint16_t)) + (size_t)kRows * nB;
  }
  return scores + (p1 > p2 ? p1 : p2);
}

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
  a.n_groups = (d.nB + kRows - 1) / kRows;
  a.n_work = d.B * d.H * a.n_groups;
  a.scale = (double)d.scale;
  a.mode = r.mode;
  a.k = r.k;
  a.cap = r.cap;
  a.n_forced = r.n_forced;
  a.tau = r.tau;
  int m = d.nB - r.n_forced;
  int p = 1;
  while (p < m) p <<= 1;
  a.sort_n = (r.mode == 1) ? p : 0;
  if (r.mode == 0 && d.D <= 128) {
    const int nt = (d.nB + 63) / 64;
    if (nt <= 1) return launch_topk<1, 4>(a, d.B, d.H, stream);
    if (nt <= 2) return launch_topk<2, 4>(a, d.B, d.H, stream);
    if (nt <= 4) return launch_topk<4, 4>(a, d.B, d.H, stream);
    if (nt <= 8) return launch_topk<8, 4>(a, d.B, d.H, stream);
    if (nt <= 16) return launch_topk<16, 4>(a, d.B, d.H, stream);
    if (nt <= 24) return launch_topk<24, 2>(a, d.B, d.H, stream);
    if (nt <= 32) return launch_topk<32, 2>(a, d.B, d.H, stream);
  }
  const size_t smem = select_smem_bytes(d.nB, d.D, r.mode, a.sort_n);
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(select_kernel),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(select_kernel, dim3(a.n_work), dim3(kThreads), smem, stream, a);
  return hipGetLastError();
}

}  // namespace sva
