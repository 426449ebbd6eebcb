// Fused QK RMSNorm + 3-D RoPE + block pooling: the producer of the Q and K the
// sparse path consumes, with the block summaries of Section 4.2.2 taken in the
// same pass (Section 4.2.5 names "fused RoPE + norm"; Appendix A.2.2 lists
// fused QKNorm+RoPE in the LTX-2.3 stack).
//
// Per token (head dimension D):
//   y = x / sqrt(mean(x^2) + eps) * gamma
//   pair p = (y[2p], y[2p+1]) turns by pos_a * base^(-i/n_a), where the D/2
//   pairs form contiguous groups for the t, y, x axes (n_y = n_x = D/6 rounded
//   down, n_t the rest), i is the pair's index in its group and pos_a the
//   token's coordinate on that axis (t-major raster order)
//   the result is rounded once to bf16 and written; the block summary is the
//   mean of the rounded outputs over the block's valid tokens.
//
// One workgroup per (tensor, b, h, block).  A token row is owned by TPR lanes
// (16, or 8 when D = 64), each holding 8 consecutive elements (4 pairs): one
// 16-byte load, the sum of squares reduced over the row's lanes, the pair
// rotations, one 16-byte store.  A rotation angle is formed and reduced
// modulo one turn in float64 (integer position times a float64 frequency),
// then the hardware sine and cosine (which take turns) give it in float32
// within 3e-7.  A pair's angle depends on one coordinate
// only, so the workgroup first tabulates (cos, sin) in LDS for the t, y and x
// values its block covers (about 1.8k entries for a 45 x 80 frame), and the
// token loop reads them; a block whose ranges would overflow the table takes
// its angles directly.  Block sums of the rounded outputs are
// kept in float64 (exact for bf16 values), so the summaries equal those the
// pooling kernel would compute from the written tensors.  The kernel is bound
// by HBM: 2*S*D bytes read and written per block.
#include "sva_internal.h"

namespace sva {
namespace {

constexpr int kThreads = 256;

__device__ __forceinline__ float lo16(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float hi16(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

typedef __attribute__((ext_vector_type(2))) float float2v;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;

template <int D, int S>
__global__ __launch_bounds__(kThreads) void qknorm_rope_pool_kernel(RopeArgs a) {
  constexpr int TPR = (D == 64) ? 8 : 16;     // lanes per token row
  constexpr int NCH = D / 8;                  // chunks of 8 elements holding data
  constexpr int RPP = kThreads / TPR;         // token rows per pass
  constexpr int NP = S / RPP;                 // passes: rows each lane handles
  constexpr int NYX = D / 6;                  // rotation pairs of the y and of the x axis
  constexpr int NT = D / 2 - 2 * NYX;         // rotation pairs of the t axis
  constexpr int kTab = 3072;                  // (cos, sin) entries of the per-block table
  static_assert(RPP * D * sizeof(double) <= kTab * sizeof(float2), "partial sums fit the table");
  // the (cos, sin) table during the token loop, the partial block sums after it
  __shared__ __attribute__((aligned(16))) unsigned char shared_buf[kTab * sizeof(float2)];
  float2* tab = reinterpret_cast<float2*>(shared_buf);
  double (*part)[D] = reinterpret_cast<double (*)[D]>(shared_buf);
  __shared__ double freq_s[D / 2];
  __shared__ int3 tok_pos[S];                  // per token: (t, y, x)

  const int row = xcd_remap(blockIdx.x, a.n_rows);   // (b*H + h)*nB + i
  const bool is_k = blockIdx.y != 0;
  const uint16_t* src = is_k ? a.k_in : a.q_in;
  uint16_t* dst = is_k ? a.k_out : a.q_out;
  const float* gamma = is_k ? a.gamma_k : a.gamma_q;
  float* pool = is_k ? a.k_pool : a.q_pool;
  const int N = a.N, nB = a.nB;
  const int bh = row / nB;
  const int i = row - bh * nB;
  const int start = i * S;
  const int valid = min(S, N - start);
  const size_t base = ((size_t)bh * N + start) * D;
  const int W = a.grid_w, H = a.grid_h, HW = H * W;

  const int r0 = threadIdx.x / TPR;
  const int c = threadIdx.x - r0 * TPR;
  const bool live = c < NCH;                  // D = 112: chunks 14, 15 hold nothing

  // every row this lane handles is loaded first; the table below is built
  // while the loads are in flight
  uint4 w[NP];
#pragma unroll
  for (int k = 0; k < NP; ++k) {
    const int r = r0 + k * RPP;
    w[k] = make_uint4(0, 0, 0, 0);
    if (live && r < valid) w[k] = *reinterpret_cast<const uint4*>(src + base + (size_t)r * D + c * 8);
  }

  // coordinates of the block's tokens, once per token
  if (threadIdx.x < valid) {
    const int n = start + threadIdx.x;
    const int t = n / HW;
    const int rem = n - t * HW;
    const int yy = rem / W;
    tok_pos[threadIdx.x] = make_int3(t, yy, rem - yy * W);
  }
  constexpr double kTwoPi = 6.283185307179586476925286766559;
  // pair frequencies base^(-i/n) in float64, once per workgroup
  if (threadIdx.x < D / 2) {
    const int p = threadIdx.x;
    int idx, n;
    if (p < NT) { idx = p; n = NT; }
    else if (p < NT + NYX) { idx = p - NT; n = NYX; }
    else { idx = p - NT - NYX; n = NYX; }
    freq_s[p] = pow(a.base, -(double)idx / (double)n) * (1.0 / kTwoPi);   // turns per unit
  }
  // the coordinate ranges the block covers: t0..t1, y over one frame or all
  // rows, x over one row or the whole width
  const int t0 = start / HW, t1 = (start + valid - 1) / HW;
  const int y0 = (start - t0 * HW) / W, y1 = (start + valid - 1 - t1 * HW) / W;
  const int x0 = start - t0 * HW - y0 * W, x1 = start + valid - 1 - t1 * HW - y1 * W;
  const int ylo = (t0 == t1) ? y0 : 0, yhi = (t0 == t1) ? y1 : H - 1;
  const int xlo = (t0 == t1 && y0 == y1) ? x0 : 0, xhi = (t0 == t1 && y0 == y1) ? x1 : W - 1;
  const int ct = t1 - t0 + 1, cy = yhi - ylo + 1, cx = xhi - xlo + 1;
  const int off_y = ct * NT, off_x = off_y + cy * NYX;
  const int n_tab = off_x + cx * NYX;
  const bool use_tab = n_tab <= kTab;          // uniform
  __syncthreads();                             // freq_s and tok_pos ready
  // the angle pos * f in turns (f / 2pi held in float64), reduced to
  // [-1/2, 1/2] in float64; the hardware sin and cos take turns
  auto turn = [&](int pos, double f_turns, float& sn, float& cs) {
    double rev = (double)pos * f_turns;
    rev -= rint(rev);
    sn = __builtin_amdgcn_sinf((float)rev);
    cs = __builtin_amdgcn_cosf((float)rev);
  };
  if (use_tab) {
    for (int e = threadIdx.x; e < n_tab; e += kThreads) {
      int pos, p;
      if (e < off_y) { pos = t0 + e / NT; p = e % NT; }
      else if (e < off_x) { const int u = e - off_y; pos = ylo + u / NYX; p = NT + u % NYX; }
      else { const int u = e - off_x; pos = xlo + u / NYX; p = NT + NYX + u % NYX; }
      float sn, cs;
      turn(pos, freq_s[p], sn, cs);
      tab[e] = make_float2(cs, sn);
    }
    __syncthreads();
  }

  // this lane's 8 weights; its 4 pairs' axes, indices in their groups and frequencies
  float g[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) g[e] = live ? gamma[c * 8 + e] : 0.0f;
  int axis[4], gidx[4];
  double freq[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int p = min(c * 4 + e, D / 2 - 1);
    axis[e] = p < NT ? 0 : (p < NT + NYX ? 1 : 2);
    gidx[e] = axis[e] == 0 ? p : (axis[e] == 1 ? p - NT : p - NT - NYX);
    freq[e] = freq_s[p];
  }

  double acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
  for (int k = 0; k < NP; ++k) {
    const int r = r0 + k * RPP;
    if (r >= valid) break;                     // rows are shared by a row's lanes
    const uint4 wk = w[k];
    float x[8] = {lo16(wk.x), hi16(wk.x), lo16(wk.y), hi16(wk.y), lo16(wk.z), hi16(wk.z), lo16(wk.w), hi16(wk.w)};
    float ss = 0.0f;
#pragma unroll
    for (int e = 0; e < 8; ++e) ss = fmaf(x[e], x[e], ss);
#pragma unroll
    for (int off = TPR / 2; off > 0; off >>= 1) ss += __shfl_xor(ss, off, TPR);
    const float inv = 1.0f / sqrtf(ss / (float)D + a.eps);

    const int3 tp = tok_pos[r];
    const int t = tp.x, yy = tp.y, xx = tp.z;
    uint32_t o[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float sn, cs;
      if (use_tab) {
        const int ti = axis[e] == 0 ? (t - t0) * NT + gidx[e]
                                    : (axis[e] == 1 ? off_y + (yy - ylo) * NYX + gidx[e]
                                                    : off_x + (xx - xlo) * NYX + gidx[e]);
        const float2 v = tab[ti];
        cs = v.x;
        sn = v.y;
      } else {
        turn(axis[e] == 0 ? t : (axis[e] == 1 ? yy : xx), freq[e], sn, cs);
      }
      const float u = x[2 * e] * inv * g[2 * e];
      const float v = x[2 * e + 1] * inv * g[2 * e + 1];
      const float2v f2 = {u * cs - v * sn, u * sn + v * cs};
      const uint32_t b = __builtin_bit_cast(uint32_t, __builtin_convertvector(f2, bf16x2));  // RNE
      o[e] = b;
      acc[2 * e] += lo16(b);
      acc[2 * e + 1] += hi16(b);
    }
    if (live) *reinterpret_cast<uint4*>(dst + base + (size_t)r * D + c * 8) = make_uint4(o[0], o[1], o[2], o[3]);
  }
  __syncthreads();                             // every lane is done with the table
  if (live) {
#pragma unroll
    for (int e = 0; e < 8; ++e) part[r0][c * 8 + e] = acc[e];
  }
  __syncthreads();
  if (threadIdx.x < D) {
    double s = 0.0;
    for (int rr = 0; rr < RPP; ++rr) s += part[rr][threadIdx.x];
    pool[(size_t)row * D + threadIdx.x] = (float)(s / (double)valid);
  }
}

}  // namespace

template <int D, int S>
void launch_ds(const RopeArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL((qknorm_rope_pool_kernel<D, S>), dim3(a.n_rows, 2), dim3(kThreads), 0, stream, a);
}

hipError_t launch_qknorm_rope_pool(const Dims& d, const RopeArgs& args, hipStream_t stream) {
  RopeArgs a = args;
  a.n_rows = d.B * d.H * d.nB;
  a.N = d.N;
  a.nB = d.nB;
  a.S = d.S;
  switch (d.D * 1000 + d.S) {
    case 64064: launch_ds<64, 64>(a, stream); break;
    case 64128: launch_ds<64, 128>(a, stream); break;
    case 112064: launch_ds<112, 64>(a, stream); break;
    case 112128: launch_ds<112, 128>(a, stream); break;
    case 128064: launch_ds<128, 64>(a, stream); break;
    case 128128: launch_ds<128, 128>(a, stream); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace sva
