// Internal declarations shared by the HIP translation units of libsva.so.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "attn_args.h"
#include "xcd.h"

namespace sva {

// Problem sizes after host validation.
struct Dims {
  int B, H, N, D, S, nB;
  int frame_tokens;   // grid_h * grid_w
  double scale;       // softmax scale c (resolved, > 0)
  bool out_f32;
};

// Selection rule after host validation (counts already derived).
struct SelectRule {
  int mode;     // 0 top-k, 1 cumulative mass
  int k;        // top-k: blocks kept per row
  double tau;   // mass: threshold
  int cap;      // mass: most blocks kept per row
  int n_forced; // mass: forced first-frame blocks 0 .. n_forced-1
};

// The rescaling (per-iteration online softmax) kernel; attention.hip.
hipError_t launch_attention_rescaling(const Dims& d, bool sparse, const AttnArgs& a, hipStream_t stream);

// 32-queries-per-wave, two-waves-per-SIMD attention with a fixed reference max
// on 16x16x32 products; attention_q16.hip.
hipError_t launch_attention_q16(const Dims& d, bool sparse, const AttnArgs& a, hipStream_t stream);

// Sparse attention for 64-token blocks, two neighbouring query blocks per
// workgroup walking the union of their lists; attention_pair.hip.  Used when
// pair_attention_fits (S = 64, D = 128, at most 4096 key blocks, rows of at
// least 15% of the blocks).
bool pair_attention_fits(const Dims& d, int kmax);
hipError_t launch_attention_pair(const Dims& d, const AttnArgs& a, hipStream_t stream);

// fp8 (e4m3) quantisation and attention; fp8_quant.hip, attention_fp8.hip.
// Codes: q8, k8 [B, H, Np, D]; v8 [B, H, Np/64, D, 64] (Np = nB * S, padding
// rows zero).  Exponents: q_exp, k_exp [B, H, nB]; v_exp [B, H, D].
struct Fp8QuantArgs {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  uint8_t* q8;
  uint8_t* k8;
  uint8_t* v8;
  int32_t* q_exp;
  int32_t* k_exp;
  int32_t* v_exp;
  uint16_t* k_mean;   // bf16 [B, H, D]
  int N, nB, Np, n_rows;
  float q_mul;        // c * log2(e) in float32: Q is multiplied by it before quantising
};
hipError_t launch_quantize_fp8(const Dims& d, const Fp8QuantArgs& a, hipStream_t stream);

struct Fp8AttnArgs {
  const uint8_t* q8;
  const uint8_t* k8;
  const uint8_t* v8;
  const int32_t* q_exp;
  const int32_t* k_exp;
  const int32_t* v_exp;
  const int32_t* kv_idx;
  const int32_t* kv_count;
  void* out;
  float* lse;
  int N, nB, Np, kmax, n_rows;
  int frame_blocks;   // query blocks per frame of the latent grid, rounded (>= 1)
};
// Largest kept-block list (and nB for the dense form) the fp8 kernel holds.
constexpr int kFp8MaxList = 2047;
hipError_t launch_attention_fp8(const Dims& d, bool sparse, const Fp8AttnArgs& a, hipStream_t stream);

// First-order remainder of the dropped key blocks; remainder.hip.  Block
// arrays are padded to nBp = rem_padded_blocks(nB) rows (a multiple of 32;
// padding rows zero).  Layouts per (b, h): kbar, vbar [nBp, D] bf16; moments
// [nBp, D, D] bf16 with M[e][d] = sum_t V[t][e] (K[t][d] - kbar[d]); E bf16
// [nBp/32 chunks][nBr rows][32] (nBr = rem_weight_rows(nB); the 32 keys of a
// chunk permuted so that each MFMA lane's eight values are one 16-byte piece);
// r [nBp] float32; T [nBp, D, D] bf16.
constexpr int kRemMaxBlocks = 4096;
constexpr int kRemGemmRows = 256;   // rows i per workgroup of the T GEMM
int rem_padded_blocks(int nB);
// Rows of each 32-key chunk of E: nB rounded up to kRemGemmRows.
int rem_weight_rows(int nB);
struct RemMomentArgs {
  const uint16_t* k;
  const uint16_t* v;
  uint16_t* kbar;
  uint16_t* vbar;
  uint16_t* mom;
  int N, nB, rows;    // rows: blocks per head in the outputs (nB, or nBp when padded)
};
struct RemWeightArgs {
  const float* q_pool;
  const float* k_pool;
  const int32_t* kv_idx;
  const int32_t* kv_count;
  uint16_t* E;
  float* r;
  int nB, nBp, nBr, kmax;
  float scale;        // c
};
struct RemGemmArgs {
  const uint16_t* E;
  const uint16_t* mom;
  uint16_t* T;
  int nB, nBp, nBr, DD, n_wg;   // n_wg: set by the launcher
};
struct RemAttnArgs {
  const uint16_t* q;
  const uint16_t* kbar;
  const uint16_t* vbar;
  const int32_t* kv_idx;
  const int32_t* kv_count;
  const uint16_t* T;
  const float* r;
  const float* o_a;   // kept-block attention, float32 [B, H, N, D]
  const float* lse_a; // its LSE [B, H, N]
  void* out;
  float* lse;
  int N, nB, nBp, kmax, n_rows;   // n_rows: workgroups, set by the launcher
  float scale;        // c
  float scale_log2;   // c * log2(e)
};
hipError_t launch_block_moments(const Dims& d, const RemMomentArgs& a, hipStream_t stream);
hipError_t launch_remainder(const Dims& d, const RemWeightArgs& wa, const RemGemmArgs& ga,
                            const RemAttnArgs& aa, hipStream_t stream);

hipError_t launch_pool(const Dims& d, const uint16_t* q, const uint16_t* k, float* q_pool,
                       float* k_pool, hipStream_t stream);

// Arguments of the fused QKNorm + RoPE + pool producer; qknorm_rope.hip.
struct RopeArgs {
  const uint16_t* q_in;
  const uint16_t* k_in;
  const float* gamma_q;
  const float* gamma_k;
  uint16_t* q_out;
  uint16_t* k_out;
  float* q_pool;
  float* k_pool;
  int N, nB, S, n_rows, grid_h, grid_w;
  float eps;
  double base;
};
hipError_t launch_qknorm_rope_pool(const Dims& d, const RopeArgs& a, hipStream_t stream);

// feat_norm token pruning; token_prune.hip.
// Device workspace of the token selection: one slice of this many bytes per batch entry.
constexpr size_t kTokenSelectWsStride = 33024;
// Batch entries the allocation-free selection's static workspace holds.
constexpr int kTokenSelectStaticBatch = 16;
// Device address of that workspace on the device of `stream` (looked up once
// per device); token_prune.hip.
hipError_t token_select_scratch(hipStream_t stream, void** ptr);
hipError_t launch_token_select(int B, int N, int C, int k, const uint16_t* x, double* scores,
                               int32_t* kept_idx, int32_t* kept_pos, void* workspace,
                               hipStream_t stream);
hipError_t launch_token_gather(int B, int N, int C, int k, const uint16_t* x, const int32_t* kept_idx,
                               uint16_t* x_kept, hipStream_t stream);
hipError_t launch_token_scatter(int B, int N, int C, int k, const uint16_t* y_kept,
                                const int32_t* kept_pos, const uint16_t* base, uint16_t* out,
                                hipStream_t stream);

hipError_t launch_select(const Dims& d, const SelectRule& r, const float* q_pool,
                         const float* k_pool, int kmax, int32_t* kv_idx, int32_t* kv_count,
                         uint8_t* mask, hipStream_t stream);

hipError_t launch_attention(const Dims& d, bool sparse, const uint16_t* q, const uint16_t* k,
                            const uint16_t* v, const int32_t* kv_idx, const int32_t* kv_count,
                            int kmax, void* out, float* lse, hipStream_t stream);

}  // namespace sva
