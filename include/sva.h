/*
 * sva.h -- block-sparse spatiotemporal self-attention for video DiTs on
 * AMD Instinct MI355X (gfx950).  C ABI of libsva.so.
 *
 * The operation (paper Section 4.2.2 "Sparse Attention"; Appendix A.2.2, the
 * LTX-2.3 stage-2 setting: block size 64, density 0.1, score-based routing,
 * dense FlashAttention fallback): dense self-attention over the T x H x W
 * video-token grid is replaced by attention that visits, for each query block,
 * only the key/value blocks a block-importance score selects.  The paper
 * prints no formula for the score or the selection; this library implements
 * the reading below, step by step:
 *
 *   blocks   the grid is flattened t-major (n = (t*H + y)*W + x) and cut into
 *            nB = ceil(N/S) contiguous blocks of S tokens; the last block may
 *            be partial.
 *   pool     qbar_i = mean of Q over the valid tokens of block i; same for K.
 *   score    s[i,j] = c * <qbar_i, kbar_j>, c = softmax scale.
 *   select   top-k: the k blocks with the largest s[i,j] (ties: lower j wins),
 *            or cumulative mass: forced first-frame blocks, then blocks by
 *            descending score while the kept softmax mass over j is below tau
 *            and fewer than `cap` blocks are kept.
 *   attend   for each valid query n of block i: softmax(c * Q[n] . K[m]) V[m]
 *            over the valid keys m of the kept blocks only.
 *
 * Conventions for every entry point:
 *   - Tensors are row-major and contiguous: Q, K, V, O are [B, H, N, D]
 *     (D fastest), pooled summaries [B, H, nB, D] float32, kv_idx
 *     [B, H, nB, kmax] int32, kv_count [B, H, nB] int32, mask [B, H, nB, nB]
 *     uint8, lse [B, H, N] float32.
 *   - Q, K, V, O are bf16 (O may be float32, see sva_problem.out_dtype).  All
 *     device pointers are device memory owned by the caller; the library never
 *     allocates, frees or keeps them.  Q/K/V/O must be 16-byte aligned, the
 *     other arrays 4-byte aligned (mask: any alignment).
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).  Work
 *     is enqueued asynchronously; no call synchronizes the host.
 *   - Every call returns an sva_status.  Arguments are validated on the host
 *     before anything is launched; on any error nothing is launched and no
 *     output is touched.  SVA_ERR_HIP reports a launch error from the runtime.
 *   - The library keeps no state between calls and is safe to call from
 *     several host threads.
 */
#ifndef SVA_H
#define SVA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SVA_VERSION_MAJOR 0
#define SVA_VERSION_MINOR 1

typedef enum sva_status {
  SVA_OK = 0,
  SVA_ERR_INVALID_ARG = 1, /* null pointer, value out of range, bad enum          */
  SVA_ERR_SHAPE = 2,       /* N != T*H*W, kmax too small, sizes overflow          */
  SVA_ERR_ALIGNMENT = 3,   /* pointer not aligned as required                     */
  SVA_ERR_UNSUPPORTED = 4, /* valid but not implemented (head_dim, block, nB)     */
  SVA_ERR_HIP = 5          /* the HIP runtime reported an error at launch         */
} sva_status;

typedef enum sva_dtype { SVA_BF16 = 0, SVA_F32 = 1 } sva_dtype;

typedef enum sva_select_mode {
  SVA_SELECT_TOPK = 0,    /* keep k blocks per query block                         */
  SVA_SELECT_CUMMASS = 1  /* keep blocks until the softmax mass reaches tau        */
} sva_select_mode;

/* One video self-attention problem. */
typedef struct sva_problem {
  int32_t batch;         /* B >= 1                                                 */
  int32_t heads;         /* H >= 1                                                 */
  int32_t seq_len;       /* N >= 1 tokens; must equal grid_t*grid_h*grid_w         */
  int32_t head_dim;      /* D in {64, 112, 128}                                    */
  int32_t grid_t;        /* latent frames T >= 1                                   */
  int32_t grid_h;        /* latent height >= 1                                     */
  int32_t grid_w;        /* latent width  >= 1                                     */
  int32_t block_size;    /* S in {64, 128}: query block == key/value block         */
  double softmax_scale;  /* c; <= 0 selects 1/sqrt(D)                              */
  int32_t out_dtype;     /* sva_dtype of O: SVA_BF16 or SVA_F32                     */
} sva_problem;

/* Block-selection rule. */
typedef struct sva_select_params {
  int32_t mode;             /* sva_select_mode                                      */
  double keep_ratio;        /* top-k: r in (0, 1]; k = clamp(ceil(r*nB - 1e-6), 1, nB) */
  int32_t topk;             /* top-k: k > 0 overrides keep_ratio (clamped to nB)    */
  double mass_threshold;    /* mass: tau in (0, 1]                                  */
  double max_keep_ratio;    /* mass: rho in (0, 1]; cap = clamp(ceil(rho*nB - 1e-6), |F|, nB) */
  int32_t force_first_frame;/* mass: nonzero keeps every block holding a token of
                               frame t = 0 (blocks j with j*S < grid_h*grid_w)      */
} sva_select_params;

/* Largest nB that sva_select_blocks accepts (a row's scores are held in
 * registers, 32 per lane). */
#define SVA_SELECT_MAX_BLOCKS 2048

/* nB = ceil(N / S) for a validated problem.  Host only. */
int sva_num_blocks(const sva_problem* prob, int32_t* n_blocks);

/* Kept blocks per row that sva_select_blocks may write: k in top-k mode, cap in
 * mass mode.  kv_idx needs at least this many columns.  Host only. */
int sva_max_keep(const sva_problem* prob, const sva_select_params* sel, int32_t* kmax);

/* Step 1: block mean-pooling of Q and K (Section 4.2.2: a block-wise summary
 * is what the routing score compares).
 *   q, k    : bf16 [B, H, N, D] device
 *   q_pool  : float32 [B, H, nB, D] device, written
 *   k_pool  : float32 [B, H, nB, D] device, written
 * Each output is the mean over the block's valid tokens, accumulated in
 * float64 and rounded once to float32. */
int sva_pool_blocks(const sva_problem* prob, const void* q, const void* k,
                    float* q_pool, float* k_pool, void* stream);

/* RMSNorm and rotary-embedding parameters of sva_qknorm_rope_pool. */
typedef struct sva_rope_params {
  double eps;        /* RMSNorm epsilon, finite and >= 0 (e.g. 1e-6)              */
  double rope_base;  /* rotary base, finite and > 1 (e.g. 10000)                   */
} sva_rope_params;

/* Step 1 fused with the producer of Q and K (Section 4.2.5 names fused
 * RoPE + norm; Appendix A.2.2 lists fused QKNorm+RoPE in the LTX-2.3 stack;
 * the paper prints no formula, so this is the reading implemented).  For every
 * token of Q and of K:
 *   y = x / sqrt(mean_d x_d^2 + eps) * gamma          RMSNorm over D
 *   pair p = (y[2p], y[2p+1]) turned by the angle pos_a * base^(-i/n_a)
 * where the D/2 pairs form contiguous groups for the t, y and x axes of sizes
 * n_t = D/2 - 2*floor(D/6) and n_y = n_x = floor(D/6), i is the pair's index
 * in its group and pos_a the token's coordinate on that axis (t-major raster
 * order); a turn by phi maps (a, b) to (a cos phi - b sin phi,
 * a sin phi + b cos phi).  The result is rounded once to bf16 (nearest, ties
 * to even) and written, and the block summaries of step 1 are taken from the
 * written values in the same pass: they equal what sva_pool_blocks gives for
 * q_out and k_out.
 *   q_in, k_in       : bf16 [B, H, N, D] device, 16-byte aligned
 *   gamma_q, gamma_k : float32 [D] device, RMSNorm weights shared by the heads
 *   q_out, k_out     : bf16 [B, H, N, D] device, 16-byte aligned, written; each
 *                      may be its input (in place) but must not otherwise
 *                      overlap it
 *   q_pool, k_pool   : float32 [B, H, nB, D] device, written
 * Float32 arithmetic; the rotation angle is reduced modulo one turn in
 * float64 before its sine and cosine are taken.
 * SVA_ERR_INVALID_ARG for a null pointer, eps < 0, rope_base <= 1 or a
 * non-finite parameter. */
int sva_qknorm_rope_pool(const sva_problem* prob, const sva_rope_params* rope,
                         const void* q_in, const void* k_in, const float* gamma_q,
                         const float* gamma_k, void* q_out, void* k_out,
                         float* q_pool, float* k_pool, void* stream);

/* Steps 2-3: block scores and block selection ("score-based routing",
 * Appendix A.2.2).
 *   q_pool, k_pool : float32 [B, H, nB, D] device (from sva_pool_blocks)
 *   kmax           : columns of kv_idx, >= sva_max_keep(...)
 *   kv_idx         : int32 [B, H, nB, kmax] device, written: kept KV blocks of
 *                    each query block in ascending order, padded with -1
 *   kv_count       : int32 [B, H, nB] device, written: number of kept blocks
 *   mask           : uint8 [B, H, nB, nB] device or NULL; if given, written
 *                    with 1 for kept (i, j) and 0 elsewhere
 * Scores are accumulated in float64; ties in score are broken toward the lower
 * block index.  Requires nB <= SVA_SELECT_MAX_BLOCKS. */
int sva_select_blocks(const sva_problem* prob, const sva_select_params* sel,
                      const float* q_pool, const float* k_pool, int32_t kmax,
                      int32_t* kv_idx, int32_t* kv_count, uint8_t* mask,
                      void* stream);

/* Step 4: attention over the kept blocks only (Section 4.2.2: the kept blocks
 * are computed exactly).
 *   q, k, v   : bf16 [B, H, N, D] device
 *   kv_idx    : int32 [B, H, nB, kmax] device; entries outside [0, nB) are
 *               skipped, as are entries at or beyond kv_count
 *   kv_count  : int32 [B, H, nB] device; values are clamped to [0, kmax]
 *   out       : [B, H, N, D] device, bf16 or float32 per out_dtype, written for
 *               every valid token; a query block with no valid kept block gets
 *               zeros
 *   lse       : float32 [B, H, N] device or NULL; natural-log log-sum-exp of
 *               the scaled logits of each query (-inf for an empty row)
 * bf16 MFMA products with float32 accumulation and an online softmax in
 * float32.  Duplicate entries in a row are attended twice.
 * Performance: the fast kernels finish a query block in one pass; a block
 * whose row sums would overflow float32 (logits rising by more than about
 * 2^63 within one kept block), whose inputs hold Inf or NaN, or, at block 64
 * with D = 128 and long rows, whose pair of lists is not strictly increasing
 * and in range, is marked through its output and redone by a per-block
 * rescaling kernel on a small grid (correct, but many times slower per
 * block).  Lists as sva_select_blocks writes them never take that path. */
int sva_sparse_attention(const sva_problem* prob, const void* q, const void* k,
                         const void* v, const int32_t* kv_idx,
                         const int32_t* kv_count, int32_t kmax, void* out,
                         float* lse, void* stream);

/* The dense fallback (Appendix A.2.2 keeps layers 0-1 dense): step 4 with
 * every block kept.  Arguments as for sva_sparse_attention. */
int sva_dense_attention(const sva_problem* prob, const void* q, const void* k,
                        const void* v, void* out, float* lse, void* stream);

/* ---- First-order remainder of the dropped blocks (Section 4.2.2: the
 * non-critical blocks are compensated by a first-order Taylor approximation
 * instead of dropped; the paper gives no formula, so this is the reading
 * implemented).  For query q of query block i and a key block j that row i
 * does not keep (n_j valid tokens, block means qbar_i, kbar_j, vbar_j), every
 * exp(c q.k_t) of the block is expanded to first order about the block's mean
 * key, exp(c q.kbar_j) (1 + c q.(k_t - kbar_j)), with the weight of the
 * first-order term then taken at the block-mean query (the block-mean form):
 *   exp(c q.k_t) ~ exp(c q.kbar_j) + exp(c qbar_i.kbar_j) c q.(k_t - kbar_j)
 * so the block adds n_j exp(c q.kbar_j) to the row sum and
 * n_j exp(c q.kbar_j) vbar_j + exp(c qbar_i.kbar_j) c M_j q to the numerator,
 * with the block moment M_j[e][d] = sum_t V[t][e] (K[t][d] - kbar_j[d]).  The
 * block-mean weight makes the first-order terms of a query block one D x D
 * matrix; with the query's own weight (the plain expansion) each query would
 * contract every dropped block's moment, about three times the kept-block
 * FLOPs at 15% density.  A block is dropped for row i when no in-range entry
 * of the row's list names it.  The result is exact where every key of a
 * dropped block equals the block mean and equals dense attention when every
 * block is kept.  Otherwise it differs from the plain expansion by
 * (exp(c qbar_i.kbar_j) - exp(c q.kbar_j)) c M_j q per dropped block, first
 * order in the key deviations where a block's queries differ by order one.
 * Requires nB <= SVA_REMAINDER_MAX_BLOCKS. ---- */
#define SVA_REMAINDER_MAX_BLOCKS 4096

/* Device workspace that sva_sparse_attention_remainder needs to process all
 * B*H (batch, head) pairs in one pass, in bytes (about B*H*(N*D*4 +
 * nB*D*D*4) + smaller parts; 5.7 GB for B=1, H=48, N=111600, D=128, S=128).
 * Host only. */
int sva_remainder_workspace(const sva_problem* prob, size_t* bytes);

/* The workspace for passes of `heads` consecutive (batch, head) pairs
 * (1 <= heads <= B*H; heads = B*H gives sva_remainder_workspace).  A
 * smaller workspace makes sva_sparse_attention_remainder process the pairs
 * in groups, with the same results; 119 MB per pair at the sizes above.
 * SVA_ERR_SHAPE for heads out of range.  Host only. */
int sva_remainder_workspace_heads(const sva_problem* prob, int32_t heads, size_t* bytes);

/* The block means and moments of the remainder.
 *   k, v     : bf16 [B, H, N, D] device
 *   kbar     : bf16 [B, H, nB, D] device, written: mean of K over the block's
 *              valid tokens (float32 sum, rounded once)
 *   vbar     : bf16 [B, H, nB, D] device, written: the same for V
 *   moments  : bf16 [B, H, nB, D, D] device, written: M_j[e][d] (d fastest),
 *              computed as sum_t V[t][e] K[t][d] - (sum_t V[t][e]) (sum_t
 *              K[t][d]) / n_j from the exact bf16 products with float32 sums,
 *              rounded once
 * All pointers 16-byte aligned. */
int sva_block_moments(const sva_problem* prob, const void* k, const void* v, void* kbar,
                      void* vbar, void* moments, void* stream);

/* Attention over the kept blocks plus the first-order remainder of the dropped
 * ones.  Arguments as for sva_sparse_attention, plus:
 *   q_pool, k_pool : float32 [B, H, nB, D] device, the block means from
 *                    sva_pool_blocks (or sva_qknorm_rope_pool); 16-byte aligned
 *   workspace      : device memory, 256-byte aligned, owned by the caller;
 *                    its contents on entry do not matter and on return are
 *                    unspecified.  With sva_remainder_workspace bytes every
 *                    (batch, head) pair is done in one pass; with less (at
 *                    least sva_remainder_workspace_heads(prob, 1)) the pairs
 *                    are done in consecutive groups of as many as fit, each
 *                    group's kernels one after the other on `stream`, with
 *                    the same results; SVA_ERR_SHAPE below one pair's size
 *   out, lse       : the compensated output and its log-sum-exp (lse may be
 *                    NULL), written for every valid token
 * Steps (all on `stream`): the kept blocks exactly with a float32 output into
 * the workspace; the block moments; the weights exp(c qbar_i.kbar_j - r_i) of
 * the dropped blocks with r_i = max_j c qbar_i.kbar_j; T_i = sum of those
 * weights times M_j; then per query block an online softmax over the pooled
 * keys of its dropped blocks (bf16 MFMA, weights n_j), plus exp(r_i) c T_i q,
 * merged with the kept part and normalised once.  The reference of each row's
 * softmax starts at max(LSE of the kept part, r_i), so the output is finite as
 * long as a query's largest logit against the kept keys or a dropped block's
 * mean key is within about 80 (natural-log units) of r_i. */
int sva_sparse_attention_remainder(const sva_problem* prob, const void* q, const void* k,
                                   const void* v, const float* q_pool, const float* k_pool,
                                   const int32_t* kv_idx, const int32_t* kv_count, int32_t kmax,
                                   void* workspace, size_t workspace_bytes, void* out, float* lse,
                                   void* stream);

/* ---- feat_norm token pruning (Section 4.2.3 token pruning; Appendix A.2.2
 * keeps 50% of the video tokens by the feat_norm saliency score in the LTX-2.3
 * refinement stage; the paper prints no formula, so this is the reading
 * implemented).  Hidden states are bf16 [B, N, C] (C fastest), 16-byte
 * aligned, C a multiple of 8. ---- */
typedef struct sva_tokens {
  int32_t batch;     /* B >= 1                                                   */
  int32_t tokens;    /* N >= 1                                                   */
  int32_t channels;  /* C >= 8, a multiple of 8                                  */
} sva_tokens;

/* Tokens kept per batch entry: k = clamp(ceil(r*N - 1e-6), 1, N) for a keep
 * ratio r in (0, 1].  Host only. */
int sva_token_keep_count(const sva_tokens* t, double keep_ratio, int32_t* k);

/* Bytes of device workspace sva_token_select needs (batch * 33024).  Host only. */
int sva_token_select_workspace(const sva_tokens* t, size_t* bytes);

/* Scores and kept tokens.
 *   x         : bf16 [B, N, C] device
 *   scores    : float64 [B, N] device, written: sum over c of x[b, n, c]^2
 *               (the squared L2 norm, accumulated in float64)
 *   kept_idx  : int32 [B, k] device, written: per batch entry the k tokens
 *               with the largest score (ties to the lower index), ascending
 *   kept_pos  : int32 [B, N] device, written: a kept token's position in
 *               kept_idx, -1 for a dropped token
 *   workspace : device memory of at least sva_token_select_workspace bytes,
 *               8-byte aligned, owned by the caller; its contents on entry do
 *               not matter.  Calls that share a workspace must not overlap
 *               (order them on one stream).
 * k as sva_token_keep_count gives it.  For x holding Inf or NaN the choice
 * among those tokens is unspecified (it stays within bounds).
 * SVA_ERR_SHAPE when workspace_bytes is too small. */
int sva_token_select(const sva_tokens* t, double keep_ratio, const void* x, double* scores,
                     int32_t* kept_idx, int32_t* kept_pos, void* workspace, size_t workspace_bytes,
                     void* stream);

/* sva_token_select for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same kernels and results, with the workspace in a static
 * device array of SVA_TOKEN_SELECT_NOALLOC_MAX_BATCH * 33024 bytes (528 KB)
 * that each GPU the library runs on holds until the process ends.  Arguments
 * as for sva_token_select, without the workspace; the caller still passes the
 * outputs.  The call allocates nothing (no hipMalloc, hipFree or allocating
 * library routine); its first call on a device looks the array's address up
 * once.  Every call on one GPU shares that GPU's array: calls that overlap on
 * one GPU (unordered streams, several host threads) race, so order them on
 * one stream.  SVA_ERR_SHAPE for more than SVA_TOKEN_SELECT_NOALLOC_MAX_BATCH
 * batch entries, SVA_ERR_HIP when the address lookup fails. */
#define SVA_TOKEN_SELECT_NOALLOC_MAX_BATCH 16
int sva_token_select_noalloc(const sva_tokens* t, double keep_ratio, const void* x, double* scores,
                             int32_t* kept_idx, int32_t* kept_pos, void* stream);

/* x_kept[b, j, :] = x[b, kept_idx[b, j], :] for j < k (an index outside
 * [0, N) gives a row of zeros).
 *   x: bf16 [B, N, C]; kept_idx: int32 [B, k]; x_kept: bf16 [B, k, C], written. */
int sva_token_gather(const sva_tokens* t, int32_t k, const void* x, const int32_t* kept_idx,
                     void* x_kept, void* stream);

/* Reconstruction after the pruned span: out[b, n, :] = y_kept[b, p, :] where
 * p = kept_pos[b, n] is in [0, k), else base[b, n, :] (a dropped token keeps
 * its input).
 *   y_kept: bf16 [B, k, C]; kept_pos: int32 [B, N]; base, out: bf16 [B, N, C];
 *   out must not overlap y_kept; it may be base (in place). */
int sva_token_scatter(const sva_tokens* t, int32_t k, const void* y_kept, const int32_t* kept_pos,
                      const void* base, void* out, void* stream);

/* ---- 8-bit (fp8 e4m3) attention (Section 4.2.4 points to the SageAttention
 * series: 8-bit attention with outlier smoothing; no formula is given, so
 * this is the reading implemented).  Codes are OCP e4m3 bytes (round to
 * nearest even); every scale is a power of two 2^e, e in [-127, 127], the
 * smallest with (group's largest magnitude) <= 448 * 2^e.  D in {64, 112, 128}.
 * Np = nB * S (sva_fp8_padded_len); code rows past N are zero.  D' = D
 * rounded up to a multiple of 64 (sva_fp8_code_dim: 64, 128, 128); code
 * channels D .. D'-1 are zero and have exponent 0. ---- */
typedef struct sva_fp8_tensors {
  void* q8;          /* u8 [B, H, Np, D']: Q codes, one exponent per query block */
  void* k8;          /* u8 [B, H, Np, D']: codes of K - k_mean, one exponent per key block */
  void* v8;          /* u8 [B, H, Np/64, D', 64]: V codes in 64-key tiles, channel-major
                        inside a tile; one exponent per channel */
  int32_t* q_exp;    /* [B, H, nB] */
  int32_t* k_exp;    /* [B, H, nB] */
  int32_t* v_exp;    /* [B, H, D'] */
  void* k_mean;      /* bf16 [B, H, D]: K's channel mean over the N tokens, rounded
                        once to bf16 (the smoothing vector; every logit of a query
                        moves by the same amount, so the softmax is unchanged) */
} sva_fp8_tensors;

/* Np = nB * S, the padded token count of the code tensors.  Host only.
 * SVA_ERR_UNSUPPORTED for D outside {64, 112, 128}. */
int sva_fp8_padded_len(const sva_problem* prob, int32_t* np);

/* D', the channel count of the code tensors.  Host only. */
int sva_fp8_code_dim(const sva_problem* prob, int32_t* dp);

/* Quantise bf16 Q, K, V [B, H, N, D] into the code tensors and exponents of
 * `out` (all device memory the caller owns; k_mean is written too).  Q
 * carries the softmax scale: it is multiplied by lambda = c * log2(e) (c =
 * prob->softmax_scale, or 1/sqrt(D) when that is <= 0, in double; lambda
 * rounded once to float32) and the float32 product is quantised, so the code
 * product is the logit in base-2 units.  K is smoothed first (K - k_mean, in
 * float32).  Pointers 16-byte aligned (exponent arrays 4). */
int sva_quantize_fp8(const sva_problem* prob, const void* q, const void* k, const void* v,
                     const sva_fp8_tensors* out, void* stream);

/* Block-sparse attention on quantised inputs, with the kept-block lists of
 * sva_select_blocks (kmax <= 2047, else SVA_ERR_UNSUPPORTED).  The softmax
 * scale is the one the Q codes carry (prob->softmax_scale is not read here).
 * The unnormalised probabilities are rounded to e4m3 before the PV product and
 * l sums those rounded weights.  out: bf16 or f32 [B, H, N, D] as
 * prob->out_dtype; lse (optional) f32 [B, H, N], natural log.  k_mean is not
 * read. */
int sva_sparse_attention_fp8(const sva_problem* prob, const sva_fp8_tensors* in, const int32_t* kv_idx,
                             const int32_t* kv_count, int32_t kmax, void* out, float* lse, void* stream);

/* The same with every block kept (nB <= 2047). */
int sva_dense_attention_fp8(const sva_problem* prob, const sva_fp8_tensors* in, void* out, float* lse,
                            void* stream);

/* Static text for a status code. */
const char* sva_status_string(int status);

/* SVA_VERSION_MAJOR * 100 + SVA_VERSION_MINOR. */
int sva_version(void);

#ifdef __cplusplus
}
#endif

#endif /* SVA_H */
