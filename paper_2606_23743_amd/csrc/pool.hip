// Block mean-pooling of Q and K (the block summaries the routing score compares;
// Section 4.2.2 "block-wise similarity", Appendix A.2.2 "score-based routing").
//
// One workgroup per (tensor, b, h, block).  The block's S x D bf16 tile is read
// once with 16-byte loads (coalesced: consecutive threads read consecutive
// 16-byte chunks of a row); each thread accumulates 8 columns over a strided
// set of rows in float64, partial sums meet in LDS, and D threads finish the
// mean over the block's valid tokens and round once to float32.  The kernel
// is bound by HBM reads: 2*S*D bytes in, 4*D bytes out per block.
#include "sva_internal.h"

namespace sva {
namespace {

constexpr int kPoolThreads = 256;

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

template <int D>
__global__ __launch_bounds__(kPoolThreads) void pool_kernel(const uint16_t* __restrict__ q,
                                                            const uint16_t* __restrict__ k,
                                                            float* __restrict__ q_pool,
                                                            float* __restrict__ k_pool, int N,
                                                            int S, int nB, int n_rows) {
  constexpr int kChunks = D / 8;                    // 16-byte chunks per token row
  constexpr int kRowsPerPass = kPoolThreads / kChunks;
  __shared__ double part[kRowsPerPass][D];

  const int row = xcd_remap(blockIdx.x, n_rows);    // (b*H + h)*nB + i
  const uint16_t* src = blockIdx.y ? k : q;
  float* dst = blockIdx.y ? k_pool : q_pool;
  const int bh = row / nB;
  const int i = row - bh * nB;
  const int start = i * S;
  const int valid = min(S, N - start);
  const uint16_t* base = src + ((size_t)bh * N + start) * D;

  const int t = threadIdx.x;
  const int r0 = t / kChunks;
  const int c = t - r0 * kChunks;
  if (r0 < kRowsPerPass) {
    double acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll 4
    for (int r = r0; r < valid; r += kRowsPerPass) {
      const uint4 w = *reinterpret_cast<const uint4*>(base + (size_t)r * D + c * 8);
      acc[0] += bf16_lo(w.x); acc[1] += bf16_hi(w.x);
      acc[2] += bf16_lo(w.y); acc[3] += bf16_hi(w.y);
      acc[4] += bf16_lo(w.z); acc[5] += bf16_hi(w.z);
      acc[6] += bf16_lo(w.w); acc[7] += bf16_hi(w.w);
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) part[r0][c * 8 + e] = acc[e];
  }
  __syncthreads();
  if (t < D) {
    double s = 0.0;
#pragma unroll 4
    for (int r = 0; r < kRowsPerPass; ++r) s += part[r][t];
    dst[(size_t)row * D + t] = (float)(s / (double)valid);
  }
}

}  // namespace

hipError_t launch_pool(const Dims& d, const uint16_t* q, const uint16_t* k, float* q_pool,
                       float* k_pool, hipStream_t stream) {
  const int n_rows = d.B * d.H * d.nB;
  dim3 grid(n_rows, 2);
  switch (d.D) {
    case 64:
      hipLaunchKernelGGL(pool_kernel<64>, grid, dim3(kPoolThreads), 0, stream, q, k, q_pool,
                         k_pool, d.N, d.S, d.nB, n_rows);
      break;
    case 112:
      hipLaunchKernelGGL(pool_kernel<112>, grid, dim3(kPoolThreads), 0, stream, q, k, q_pool,
                         k_pool, d.N, d.S, d.nB, n_rows);
      break;
    case 128:
      hipLaunchKernelGGL(pool_kernel<128>, grid, dim3(kPoolThreads), 0, stream, q, k, q_pool,
                         k_pool, d.N, d.S, d.nB, n_rows);
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace sva
