// feat_norm token pruning (Section 4.2.3 token pruning; Appendix A.2.2 keeps
// 50% of the video tokens by the feat_norm saliency score): token scores, the
// kept-token selection, and the gather / scatter around the pruned span.
//
//   score  s[b, n] = sum_c x[b, n, c]^2 in float64 (the products of bf16 values
//          are exact there); one wave per token, 16-byte loads.
//   select the k largest scores of each batch entry (ties to the lower token
//          index), listed in ascending order: a grid-wide radix select over
//          the scores' order keys finds the k-th largest key, then a counting
//          pass and a write pass over token segments emit kept_idx (ascending)
//          and kept_pos (the position of each kept token, -1 for the others).
//   gather x_kept[b, j] = x[b, kept_idx[b, j]]; scatter out[b, n] = y_kept[b,
//          kept_pos[b, n]] for kept tokens and base[b, n] for the others.  One
//          wave per row, 16-byte loads and stores.
#include <mutex>

#include "sva_internal.h"

namespace sva {
namespace {

__device__ __forceinline__ float lo16(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float hi16(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

__device__ __forceinline__ uint64_t order_key(double s) {
  if (s == 0.0) s = 0.0;           // -0 and +0 compare equal: give them one key
  const uint64_t b = (uint64_t)__double_as_longlong(s);
  return (b >> 63) ? ~b : (b | 0x8000000000000000ull);
}

__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

// ---- selection: a radix select over the 64-bit order keys, grid-wide ----
//
// Digits of 12 bits from the top (bits 63..52, 51..40, ..., 3..0): each pass
// histograms the digit of every key that matches the prefix resolved so far
// (an LDS histogram per workgroup, flushed to the batch entry's global one);
// the last workgroup to finish the pass (a ticket counter, no waiting) picks
// the digit holding the k-th largest key and clears the histogram for the next
// pass.  The search ends when every key with the resolved prefix is needed
// (then the prefix with zero low bits is the threshold) or all 64 bits are
// resolved; later passes return at once.  Then a counting pass finds, per
// token segment, the keys above the threshold and equal to it, the last
// workgroup turns those counts into output offsets and tie quotas, and the
// write pass emits kept_idx and kept_pos in token order.

constexpr int kDigitBits = 12;
constexpr int kBins = 1 << kDigitBits;
constexpr int kPasses = 6;                       // ceil(64 / 12)
constexpr int kSegThreads = 512;
constexpr int kMaxSegs = 1024;
// tokens per segment (one workgroup each): fewer, larger segments cut the
// per-workgroup cost of the cross-workgroup hand-off (a release fence and a
// ticket atomic); 2048 measured fastest at 111600 tokens
constexpr int kSegTokens = 2048;

struct SelState {            // per batch entry, at the head of its workspace slice
  unsigned long long prefix; // the resolved high bits of the k-th largest key
  int need;                  // keys still to take among those matching the prefix
  int done;                  // the threshold is resolved
  unsigned int ticket;       // workgroups finished in the current pass
  int need_eq;               // keys equal to the threshold that are kept
  int pad[2];
};

static_assert(sizeof(SelState) + sizeof(uint32_t) * kBins + 4 * sizeof(int) * kMaxSegs <=
                  kTokenSelectWsStride, "workspace slice per batch entry");

struct SelWs {
  SelState* st;
  uint32_t* hist;            // [kBins]
  int* gt;                   // [kMaxSegs] per segment: keys above the threshold
  int* eq;                   // [kMaxSegs] per segment: keys equal to it
  int* kept_before;          // [kMaxSegs] exclusive offsets into kept_idx
  int* eq_before;            // [kMaxSegs] equal keys in earlier segments
};

__device__ __forceinline__ SelWs sel_ws(unsigned char* ws, int b) {
  unsigned char* p = ws + (size_t)b * kTokenSelectWsStride;
  SelWs w;
  w.st = reinterpret_cast<SelState*>(p);
  w.hist = reinterpret_cast<uint32_t*>(p + sizeof(SelState));
  w.gt = reinterpret_cast<int*>(w.hist + kBins);
  w.eq = w.gt + kMaxSegs;
  w.kept_before = w.eq + kMaxSegs;
  w.eq_before = w.kept_before + kMaxSegs;
  return w;
}

// workgroup-wide exclusive prefix sum (and the total) of one value per thread;
// every thread calls it
__device__ int block_scan(int v, int* red, int& total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int incl = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int o = __shfl_up(incl, off, 64);
    if (lane >= off) incl += o;
  }
  if (lane == 63) red[w] = incl;
  __syncthreads();
  int before = 0, tot = 0;
#pragma unroll
  for (int i = 0; i < kSegThreads / 64; ++i) {
    const int r = red[i];
    before += i < w ? r : 0;
    tot += r;
  }
  __syncthreads();
  total = tot;
  return before + incl - v;
}

// scores: one wave per token; blocks below B also initialise the selection state
__global__ __launch_bounds__(256) void token_score_kernel(const uint16_t* __restrict__ x,
                                                          double* __restrict__ scores,
                                                          unsigned char* __restrict__ ws, int B,
                                                          int rows, int C, int k) {
  if (blockIdx.x < (unsigned)B) {
    const SelWs w = sel_ws(ws, blockIdx.x);
    for (int i = threadIdx.x; i < kBins; i += 256) w.hist[i] = 0;
    if (threadIdx.x == 0) {
      w.st->prefix = 0;
      w.st->need = k;
      w.st->done = 0;
      w.st->ticket = 0;
      w.st->need_eq = 0;
    }
  }
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const uint16_t* p = x + (size_t)row * C;
  double acc = 0.0;
  for (int c = lane * 8; c < C; c += 512) {
    const uint4 q = *reinterpret_cast<const uint4*>(p + c);
    const float v[8] = {lo16(q.x), hi16(q.x), lo16(q.y), hi16(q.y), lo16(q.z), hi16(q.z), lo16(q.w), hi16(q.w)};
#pragma unroll
    for (int e = 0; e < 8; ++e) acc = fma((double)v[e], (double)v[e], acc);
  }
  acc = wave_sum(acc);
  if (lane == 0) scores[row] = acc;
}

// true in the one workgroup that finishes the pass last (all threads call it)
__device__ bool last_to_finish(unsigned int* ticket, int* flag) {
  __threadfence();
  __syncthreads();
  if (threadIdx.x == 0) *flag = atomicAdd(ticket, 1u) == gridDim.x - 1;
  __syncthreads();
  const bool last = *flag;
  if (last) __threadfence();
  return last;
}

// one digit of the radix select; grid (segments, B)
__global__ __launch_bounds__(kSegThreads) void token_pass_kernel(const double* __restrict__ scores,
                                                                 unsigned char* __restrict__ ws,
                                                                 int N, int seg_len, int pass) {
  __shared__ uint32_t h[kBins];
  __shared__ int red[kSegThreads / 64];
  __shared__ int flag;
  __shared__ int pick[3];
  const int b = blockIdx.y;
  const SelWs w = sel_ws(ws, b);
  if (w.st->done) return;                                   // uniform
  const int hi = 63 - kDigitBits * pass;
  const int lo = hi - kDigitBits + 1 > 0 ? hi - kDigitBits + 1 : 0;
  const uint64_t mask = (1ull << (hi - lo + 1)) - 1;
  const uint64_t prefix = w.st->prefix;
  for (int i = threadIdx.x; i < kBins; i += kSegThreads) h[i] = 0;
  __syncthreads();
  const double* s = scores + (size_t)b * N;
  const int n0 = blockIdx.x * seg_len, n1 = min(N, n0 + seg_len);
  for (int n = n0 + threadIdx.x; n < n1; n += kSegThreads) {
    const uint64_t key = order_key(s[n]);
    if (hi == 63 || (key >> (hi + 1)) == (prefix >> (hi + 1)))
      atomicAdd(&h[(key >> lo) & mask], 1u);
  }
  __syncthreads();
  for (int i = threadIdx.x; i < kBins; i += kSegThreads)
    if (h[i]) atomicAdd(&w.hist[i], h[i]);
  if (!last_to_finish(&w.st->ticket, &flag)) return;

  // the last workgroup: bins from the top until the k-th largest key is reached
  constexpr int BPT = kBins / kSegThreads;                  // bins per thread
  const int t0 = threadIdx.x * BPT;
  uint32_t mine[BPT];
  int sum = 0;
#pragma unroll
  for (int e = 0; e < BPT; ++e) {
    mine[e] = __hip_atomic_load(&w.hist[t0 + e], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    sum += (int)mine[e];
  }
  int total;
  const int excl = block_scan(sum, red, total);
  int above = total - excl - sum;                           // keys in higher bins
  const int need = w.st->need;
#pragma unroll
  for (int e = BPT - 1; e >= 0; --e) {
    const int c = (int)mine[e];
    if (above < need && need <= above + c) {
      pick[0] = t0 + e;
      pick[1] = above;
      pick[2] = c;
    }
    above += c;
  }
  __syncthreads();
  for (int i = threadIdx.x; i < kBins; i += kSegThreads) w.hist[i] = 0;
  if (threadIdx.x == 0) {
    const int left = need - pick[1];
    w.st->prefix = prefix | ((uint64_t)pick[0] << lo);
    w.st->need = left;
    w.st->done = (left == pick[2] || lo == 0) ? 1 : 0;
    w.st->ticket = 0;
  }
}

// keys above and equal to the threshold per segment; the last workgroup turns
// them into output offsets and tie quotas.  grid (segments, B)
__global__ __launch_bounds__(kSegThreads) void token_count_kernel(const double* __restrict__ scores,
                                                                  unsigned char* __restrict__ ws,
                                                                  int N, int seg_len, int k) {
  __shared__ int red[kSegThreads / 64];
  __shared__ int flag;
  const int b = blockIdx.y;
  const SelWs w = sel_ws(ws, b);
  const uint64_t T = w.st->prefix;
  const double* s = scores + (size_t)b * N;
  const int n0 = blockIdx.x * seg_len, n1 = min(N, n0 + seg_len);
  int gt = 0, eq = 0;
  for (int n = n0 + threadIdx.x; n < n1; n += kSegThreads) {
    const uint64_t key = order_key(s[n]);
    gt += key > T ? 1 : 0;
    eq += key == T ? 1 : 0;
  }
  int tg, te;
  block_scan(gt, red, tg);
  block_scan(eq, red, te);
  if (threadIdx.x == 0) {
    w.gt[blockIdx.x] = tg;
    w.eq[blockIdx.x] = te;
  }
  if (!last_to_finish(&w.st->ticket, &flag)) return;

  const int nseg = gridDim.x;
  constexpr int SPT = kMaxSegs / kSegThreads;               // segments per thread
  int g[SPT], e[SPT], sg = 0, se = 0;
#pragma unroll
  for (int i = 0; i < SPT; ++i) {
    const int sgi = threadIdx.x * SPT + i;
    g[i] = sgi < nseg ? __hip_atomic_load(&w.gt[sgi], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : 0;
    e[i] = sgi < nseg ? __hip_atomic_load(&w.eq[sgi], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : 0;
    sg += g[i];
    se += e[i];
  }
  int all_gt, all_eq;
  block_scan(sg, red, all_gt);
  int eb = block_scan(se, red, all_eq);
  const int need_eq = k - all_gt;                           // equal keys kept, lowest index first
  int take[SPT], st = 0;
#pragma unroll
  for (int i = 0; i < SPT; ++i) {
    take[i] = max(0, min(e[i], need_eq - eb));
    eb += e[i];
    st += g[i] + take[i];
  }
  int unused;
  int kb = block_scan(st, red, unused);
  eb -= se;
#pragma unroll
  for (int i = 0; i < SPT; ++i) {
    const int sgi = threadIdx.x * SPT + i;
    if (sgi < nseg) {
      w.kept_before[sgi] = kb;
      w.eq_before[sgi] = eb;
    }
    kb += g[i] + take[i];
    eb += e[i];
  }
  if (threadIdx.x == 0) {
    w.st->need_eq = need_eq;
    w.st->ticket = 0;
  }
}

// kept_idx (ascending) and kept_pos, segment by segment in token order.  grid (segments, B)
__global__ __launch_bounds__(kSegThreads) void token_write_kernel(const double* __restrict__ scores,
                                                                  const unsigned char* __restrict__ ws,
                                                                  int32_t* __restrict__ kept_idx,
                                                                  int32_t* __restrict__ kept_pos,
                                                                  int N, int seg_len, int k) {
  __shared__ int red[kSegThreads / 64];
  const int b = blockIdx.y;
  const SelWs w = sel_ws(const_cast<unsigned char*>(ws), b);
  const uint64_t T = w.st->prefix;
  const int need_eq = w.st->need_eq;
  int pos = w.kept_before[blockIdx.x], ties = w.eq_before[blockIdx.x];
  const double* s = scores + (size_t)b * N;
  const int n0 = blockIdx.x * seg_len, n1 = min(N, n0 + seg_len);
  for (int base = n0; base < n1; base += kSegThreads) {      // uniform trip count
    const int n = base + threadIdx.x;
    uint64_t key = 0;
    if (n < n1) key = order_key(s[n]);
    const bool in = n < n1;
    const int is_eq = (in && key == T) ? 1 : 0;
    int n_eq;
    const int eq_rank = ties + block_scan(is_eq, red, n_eq);
    const int kp = (in && (key > T || (is_eq && eq_rank < need_eq))) ? 1 : 0;
    int n_kp;
    const int p = pos + block_scan(kp, red, n_kp);
    if (in) {
      if (kp && p < k) kept_idx[(size_t)b * k + p] = n;
      kept_pos[(size_t)b * N + n] = (kp && p < k) ? p : -1;
    }
    ties += n_eq;
    pos += n_kp;
  }
}

// x_kept[b, j] = x[b, kept_idx[b, j]]; one wave per kept row
__global__ __launch_bounds__(256) void token_gather_kernel(const uint16_t* __restrict__ x,
                                                           const int32_t* __restrict__ kept_idx,
                                                           uint16_t* __restrict__ x_kept, int B,
                                                           int N, int C, int k) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);   // b * k + j
  if (row >= B * k) return;
  const int b = row / k;
  const int n = kept_idx[row];
  uint16_t* dst = x_kept + (size_t)row * C;
  if (n < 0 || n >= N) {                     // not a token of this entry: zeros
    for (int c = lane * 8; c < C; c += 512) *reinterpret_cast<uint4*>(dst + c) = make_uint4(0, 0, 0, 0);
    return;
  }
  const uint16_t* src = x + ((size_t)b * N + n) * C;
  for (int c = lane * 8; c < C; c += 512)
    *reinterpret_cast<uint4*>(dst + c) = *reinterpret_cast<const uint4*>(src + c);
}

// out[b, n] = y_kept[b, kept_pos[b, n]] if kept, else base[b, n]; one wave per row
__global__ __launch_bounds__(256) void token_scatter_kernel(const uint16_t* __restrict__ y_kept,
                                                            const int32_t* __restrict__ kept_pos,
                                                            const uint16_t* __restrict__ base,
                                                            uint16_t* __restrict__ out, int B,
                                                            int N, int C, int k) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);   // b * N + n
  if (row >= B * N) return;
  const int b = row / N;
  const int pos = kept_pos[row];
  const uint16_t* src = (pos >= 0 && pos < k) ? y_kept + ((size_t)b * k + pos) * C : base + (size_t)row * C;
  uint16_t* dst = out + (size_t)row * C;
  for (int c = lane * 8; c < C; c += 512)
    *reinterpret_cast<uint4*>(dst + c) = *reinterpret_cast<const uint4*>(src + c);
}

}  // namespace

int token_select_segments(int N) {
  const int nseg = (N + kSegTokens - 1) / kSegTokens;
  return nseg < kMaxSegs ? nseg : kMaxSegs;
}

hipError_t launch_token_select(int B, int N, int C, int k, const uint16_t* x, double* scores,
                               int32_t* kept_idx, int32_t* kept_pos, void* workspace,
                               hipStream_t stream) {
  unsigned char* ws = static_cast<unsigned char*>(workspace);
  const int rows = B * N;
  const int grid = max((rows + 3) / 4, B);
  hipLaunchKernelGGL(token_score_kernel, dim3(grid), dim3(256), 0, stream, x, scores, ws, B, rows, C, k);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int nseg = token_select_segments(N);
  const int seg_len = (N + nseg - 1) / nseg;
  for (int pass = 0; pass < kPasses; ++pass) {
    hipLaunchKernelGGL(token_pass_kernel, dim3(nseg, B), dim3(kSegThreads), 0, stream, scores, ws, N,
                       seg_len, pass);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  hipLaunchKernelGGL(token_count_kernel, dim3(nseg, B), dim3(kSegThreads), 0, stream, scores, ws, N,
                     seg_len, k);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(token_write_kernel, dim3(nseg, B), dim3(kSegThreads), 0, stream, scores, ws,
                     kept_idx, kept_pos, N, seg_len, k);
  return hipGetLastError();
}

// Workspace of the allocation-free token selection (sva_token_select_noalloc):
// kTokenSelectStaticBatch slices.  Each GPU the library runs on holds its own
// copy until the process ends; host code never passes the array's name to a
// kernel (in host code it is a stand-in, not a device address), only the
// per-device address hipGetSymbolAddress returns.
static __device__ __align__(256) unsigned char scratch[kTokenSelectStaticBatch * kTokenSelectWsStride];

hipError_t token_select_scratch(hipStream_t stream, void** ptr) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static void* addr[kMaxDevices] = {};
  int dev = 0;
  hipError_t e = stream ? hipStreamGetDevice(stream, &dev) : hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    // once per device, with that device current
    int cur = 0;
    if ((e = hipGetDevice(&cur)) != hipSuccess) return e;
    if (cur != dev && (e = hipSetDevice(dev)) != hipSuccess) return e;
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    const hipError_t back = cur != dev ? hipSetDevice(cur) : hipSuccess;
    if (e != hipSuccess) return e;
    if (back != hipSuccess) return back;
    if (!p) return hipErrorInvalidSymbol;
    addr[dev] = p;
  }
  *ptr = addr[dev];
  return hipSuccess;
}

hipError_t launch_token_gather(int B, int N, int C, int k, const uint16_t* x, const int32_t* kept_idx,
                               uint16_t* x_kept, hipStream_t stream) {
  const int rows = B * k;
  hipLaunchKernelGGL(token_gather_kernel, dim3((rows + 3) / 4), dim3(256), 0, stream, x, kept_idx,
                     x_kept, B, N, C, k);
  return hipGetLastError();
}

hipError_t launch_token_scatter(int B, int N, int C, int k, const uint16_t* y_kept,
                                const int32_t* kept_pos, const uint16_t* base, uint16_t* out,
                                hipStream_t stream) {
  const int rows = B * N;
  hipLaunchKernelGGL(token_scatter_kernel, dim3((rows + 3) / 4), dim3(256), 0, stream, y_kept,
                     kept_pos, base, out, B, N, C, k);
  return hipGetLastError();
}

}  // namespace sva
