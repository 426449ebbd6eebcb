// fp8 (e4m3) quantisation of Q, K, V for 8-bit attention (Section 4.2.4
// points to 8-bit attention with outlier smoothing, the SageAttention series).
//
// Scales are powers of two 2^e (the MX e8m0 scales the gfx950 matrix
// instructions apply themselves): for a group with largest magnitude a, e is
// the smallest exponent with a <= 448 * 2^e, so x * 2^-e is exact in float32
// and the hardware conversion (round to nearest even) gives the code.
//   stats  the float64 channel sums of K over all N tokens (mean rounded once
//          to bf16: the smoothing vector) and the channel maxima of |V| (V's
//          per-channel exponents): segment partials, then a fixed-order sum.
//   Q, K   one workgroup per (tensor, b, h, block): Q is first multiplied by
//          the softmax scale in base 2 (float32), so the code product is the
//          logit in base-2 units; K subtracts the smoothing vector in float32;
//          the block's largest magnitude sets its exponent; codes are written
//          [B, H, Np, DP] (Np = nB * S, rows past N zero).
//   V      one workgroup per (b, h, block): codes with the channel exponents,
//          transposed through LDS into 64-key tiles [B, H, Np/64, DP, 64], the
//          layout the attention kernel stages directly.
// DP is D rounded up to a multiple of 64 (the fp8 matrix instructions take 64
// channels per step): at D = 112 the codes of channels 112..127 are zero and
// their V exponent is 0.
#include "sva_internal.h"

namespace sva {
namespace {

constexpr int kThreads = 256;
constexpr int kStatThreads = 1024;

__device__ __forceinline__ float lo16(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float hi16(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// smallest e in [-127, 127] with amax <= 448 * 2^e; 0 for amax = 0.
// 448 = 0.875 * 2^9 and amax = f * 2^x with f in [0.5, 1).
__device__ __forceinline__ int scale_exp(float amax) {
  if (!(amax > 0.0f)) return 0;
  int x;
  const float f = frexpf(amax, &x);
  const int e = f <= 0.875f ? x - 9 : x - 8;
  return e < -127 ? -127 : (e > 127 ? 127 : e);
}

// four float32 values -> four e4m3 codes (round to nearest even), packed
__device__ __forceinline__ uint32_t pack4_e4m3(float a, float b, float c, float d) {
  int w = 0;
  w = __builtin_amdgcn_cvt_pk_fp8_f32(a, b, w, false);
  w = __builtin_amdgcn_cvt_pk_fp8_f32(c, d, w, true);
  return (uint32_t)w;
}

// a float64 value rounded once to bf16 (nearest, ties to even), as bf16 bits
__device__ __forceinline__ uint16_t round_bf16_bits(double x) {
  if (x == 0.0) return (uint16_t)(__double_as_longlong(x) >> 48);
  int e;
  (void)frexp(x, &e);
  const int sh = e - 8 > -133 ? e - 8 : -133;          // spacing of bf16 values near x
  const double r = ldexp(rint(ldexp(x, -sh)), sh);     // exact: a bf16 value
  return (uint16_t)(__float_as_uint((float)r) >> 16);
}

// Channel statistics in two steps, so that every CU takes part: segment
// workgroups of kStatRows tokens write float64 partial sums of K and float32
// partial maxima of |V| per channel, then one small workgroup per (b, h) adds
// them in segment order (deterministic).  The partials are staged in the
// head's K-code region, which the Q/K quantiser overwrites right after (it is
// at least 12 * nseg * DP bytes: Np >= 64 tokens of DP bytes each).
constexpr int kStatRows = 1024;

template <int D>
__global__ __launch_bounds__(kStatThreads) void fp8_stats_partial_kernel(Fp8QuantArgs a) {
  constexpr int DP = (D + 63) / 64 * 64;
  constexpr int TPR = DP / 8;                 // lanes per token row
  constexpr int RPP = kStatThreads / TPR;     // rows per pass
  __shared__ double part_s[RPP][DP];
  __shared__ float part_m[RPP][DP];
  const int seg = blockIdx.x, bh = blockIdx.y;
  const int nseg = gridDim.x;
  const int N = a.N;
  const int r0 = threadIdx.x / TPR, c = threadIdx.x % TPR;
  const bool live = c < D / 8;                // D = 112: lanes 14, 15 hold no channel
  const uint16_t* K = a.k + (size_t)bh * N * D;
  const uint16_t* V = a.v + (size_t)bh * N * D;
  const int n0 = seg * kStatRows, n1 = min(N, n0 + kStatRows);
  double s[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  float m[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  for (int r = n0 + r0; live && r < n1; r += RPP) {
    const uint4 kw = *reinterpret_cast<const uint4*>(K + (size_t)r * D + c * 8);
    const uint4 vw = *reinterpret_cast<const uint4*>(V + (size_t)r * D + c * 8);
    const float kx[8] = {lo16(kw.x), hi16(kw.x), lo16(kw.y), hi16(kw.y), lo16(kw.z), hi16(kw.z), lo16(kw.w), hi16(kw.w)};
    const float vx[8] = {lo16(vw.x), hi16(vw.x), lo16(vw.y), hi16(vw.y), lo16(vw.z), hi16(vw.z), lo16(vw.w), hi16(vw.w)};
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      s[e] += (double)kx[e];
      m[e] = fmaxf(m[e], fabsf(vx[e]));
    }
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    part_s[r0][c * 8 + e] = s[e];
    part_m[r0][c * 8 + e] = m[e];
  }
  __syncthreads();
  if (threadIdx.x < DP) {
    const int d = threadIdx.x;
    double t = 0.0;
    float mx = 0.0f;
    for (int r = 0; r < RPP; ++r) {          // fixed order: deterministic
      t += part_s[r][d];
      mx = fmaxf(mx, part_m[r][d]);
    }
    unsigned char* scratch = a.k8 + (size_t)bh * a.Np * DP;
    reinterpret_cast<double*>(scratch)[(size_t)seg * DP + d] = t;
    reinterpret_cast<float*>(scratch + (size_t)nseg * DP * sizeof(double))[(size_t)seg * DP + d] = mx;
  }
}

template <int D>
__global__ __launch_bounds__(128) void fp8_stats_final_kernel(Fp8QuantArgs a, int nseg) {
  constexpr int DP = (D + 63) / 64 * 64;
  const int bh = blockIdx.x, d = threadIdx.x;
  if (d >= DP) return;
  const unsigned char* scratch = a.k8 + (size_t)bh * a.Np * DP;
  const double* ps = reinterpret_cast<const double*>(scratch);
  const float* pm = reinterpret_cast<const float*>(scratch + (size_t)nseg * DP * sizeof(double));
  double t = 0.0;
  float mx = 0.0f;
  for (int g = 0; g < nseg; ++g) {           // segment order: deterministic
    t += ps[(size_t)g * DP + d];
    mx = fmaxf(mx, pm[(size_t)g * DP + d]);
  }
  if (d < D) a.k_mean[(size_t)bh * D + d] = round_bf16_bits(t / (double)a.N);
  a.v_exp[(size_t)bh * DP + d] = scale_exp(mx);     // padding channels: 0
}

// Q (blockIdx.y == 0) or smoothed K (blockIdx.y == 1) of one block
template <int D, int S>
__global__ __launch_bounds__(kThreads) void fp8_quant_qk_kernel(Fp8QuantArgs a) {
  constexpr int DP = (D + 63) / 64 * 64;
  constexpr int TPR = DP / 8;
  constexpr int RPP = kThreads / TPR;
  constexpr int NP = S / RPP;
  __shared__ float red[kThreads / 64];
  const int row = xcd_remap(blockIdx.x, a.n_rows);      // (b*H + h)*nB + i
  const bool is_k = blockIdx.y != 0;
  const int nB = a.nB, N = a.N, Np = a.Np;
  const int bh = row / nB;
  const int i = row - bh * nB;
  const int valid = min(S, N - i * S);
  const uint16_t* src = (is_k ? a.k : a.q) + ((size_t)bh * N + (size_t)i * S) * D;
  uint8_t* dst = (is_k ? a.k8 : a.q8) + ((size_t)bh * Np + (size_t)i * S) * DP;
  const int r0 = threadIdx.x / TPR, c = threadIdx.x % TPR;
  const bool live = c < D / 8;                // padding lanes write zero codes
  float sub[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  const float mul = is_k ? 1.0f : a.q_mul;
  if (is_k && live) {
    const uint4 mw = *reinterpret_cast<const uint4*>(a.k_mean + (size_t)bh * D + c * 8);
    const float mv[8] = {lo16(mw.x), hi16(mw.x), lo16(mw.y), hi16(mw.y), lo16(mw.z), hi16(mw.z), lo16(mw.w), hi16(mw.w)};
#pragma unroll
    for (int e = 0; e < 8; ++e) sub[e] = mv[e];
  }
  float x[NP][8];
  float amax = 0.0f;
#pragma unroll
  for (int p = 0; p < NP; ++p) {
    const int r = r0 + p * RPP;
    uint4 w = make_uint4(0, 0, 0, 0);
    if (live && r < valid) w = *reinterpret_cast<const uint4*>(src + (size_t)r * D + c * 8);
    const float v[8] = {lo16(w.x), hi16(w.x), lo16(w.y), hi16(w.y), lo16(w.z), hi16(w.z), lo16(w.w), hi16(w.w)};
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      // K: float32 difference (sub is zero for Q); Q: float32 product (mul is 1 for K)
      x[p][e] = (live && r < valid) ? __builtin_fmaf(v[e], mul, -sub[e]) : 0.0f;
      amax = fmaxf(amax, fabsf(x[p][e]));
    }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) amax = fmaxf(amax, __shfl_xor(amax, off, 64));
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = amax;
  __syncthreads();
  float bmax = red[0];
#pragma unroll
  for (int w = 1; w < kThreads / 64; ++w) bmax = fmaxf(bmax, red[w]);
  const int e = scale_exp(bmax);
  if (threadIdx.x == 0) (is_k ? a.k_exp : a.q_exp)[row] = e;
#pragma unroll
  for (int p = 0; p < NP; ++p) {
    const int r = r0 + p * RPP;
    uint2 o;
    o.x = pack4_e4m3(ldexpf(x[p][0], -e), ldexpf(x[p][1], -e), ldexpf(x[p][2], -e), ldexpf(x[p][3], -e));
    o.y = pack4_e4m3(ldexpf(x[p][4], -e), ldexpf(x[p][5], -e), ldexpf(x[p][6], -e), ldexpf(x[p][7], -e));
    *reinterpret_cast<uint2*>(dst + (size_t)r * DP + c * 8) = o;   // rows past N, padding: zeros
  }
}

// V of one block, transposed into 64-key tiles
template <int D, int S>
__global__ __launch_bounds__(kThreads) void fp8_quant_v_kernel(Fp8QuantArgs a) {
  constexpr int DP = (D + 63) / 64 * 64;
  __shared__ __attribute__((aligned(16))) uint16_t tile[S][D];
  const int row = xcd_remap(blockIdx.x, a.n_rows);
  const int nB = a.nB, N = a.N, Np = a.Np;
  const int bh = row / nB;
  const int i = row - bh * nB;
  const int valid = min(S, N - i * S);
  const uint16_t* src = a.v + ((size_t)bh * N + (size_t)i * S) * D;
  for (int u = threadIdx.x; u < S * D / 8; u += kThreads) {
    const int r = u / (D / 8), c = u % (D / 8);
    uint4 w = make_uint4(0, 0, 0, 0);
    if (r < valid) w = *reinterpret_cast<const uint4*>(src + (size_t)r * D + c * 8);
    *reinterpret_cast<uint4*>(&tile[r][c * 8]) = w;
  }
  __syncthreads();
  const int nC = Np / 64;
  // item (d, 8-token group): consecutive threads take consecutive channels
  for (int u = threadIdx.x; u < DP * (S / 8); u += kThreads) {
    const int d = u % DP, t8 = u / DP;
    uint2 o = make_uint2(0, 0);                          // padding channels: zero codes
    if (d < D) {
      const int e = a.v_exp[(size_t)bh * DP + d];
      float v[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) v[k] = ldexpf(__uint_as_float((uint32_t)tile[t8 * 8 + k][d] << 16), -e);
      o.x = pack4_e4m3(v[0], v[1], v[2], v[3]);
      o.y = pack4_e4m3(v[4], v[5], v[6], v[7]);
    }
    const int tok = i * S + t8 * 8;                      // first token of the group
    const size_t off = (((size_t)bh * nC + tok / 64) * DP + d) * 64 + (tok % 64);
    *reinterpret_cast<uint2*>(a.v8 + off) = o;
  }
}

template <int D, int S>
void launch_quant_ds(const Fp8QuantArgs& a, int BH, hipStream_t stream) {
  const int nseg = (a.N + kStatRows - 1) / kStatRows;
  hipLaunchKernelGGL((fp8_stats_partial_kernel<D>), dim3(nseg, BH), dim3(kStatThreads), 0, stream, a);
  hipLaunchKernelGGL((fp8_stats_final_kernel<D>), dim3(BH), dim3(128), 0, stream, a, nseg);
  hipLaunchKernelGGL((fp8_quant_qk_kernel<D, S>), dim3(a.n_rows, 2), dim3(kThreads), 0, stream, a);
  hipLaunchKernelGGL((fp8_quant_v_kernel<D, S>), dim3(a.n_rows), dim3(kThreads), 0, stream, a);
}

}  // namespace

hipError_t launch_quantize_fp8(const Dims& d, const Fp8QuantArgs& args, hipStream_t stream) {
  Fp8QuantArgs a = args;
  a.N = d.N;
  a.nB = d.nB;
  a.Np = d.nB * d.S;
  a.n_rows = d.B * d.H * d.nB;
  const int BH = d.B * d.H;
  switch (d.D * 1000 + d.S) {
    case 64064: launch_quant_ds<64, 64>(a, BH, stream); break;
    case 64128: launch_quant_ds<64, 128>(a, BH, stream); break;
    case 112064: launch_quant_ds<112, 64>(a, BH, stream); break;
    case 112128: launch_quant_ds<112, 128>(a, BH, stream); break;
    case 128064: launch_quant_ds<128, 64>(a, BH, stream); break;
    case 128128: launch_quant_ds<128, 128>(a, BH, stream); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace sva
