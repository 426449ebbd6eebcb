// Host side of the C ABI declared in include/sva.h: argument validation and
// dispatch.  Every check runs before any HIP call, so invalid arguments return
// a status without touching the device.
#include <math.h>
#include <stddef.h>
#include <stdint.h>

#include <algorithm>

#include "../../include/sva.h"
#include "sva_internal.h"

namespace {

using sva::Dims;
using sva::SelectRule;

constexpr double kCountEps = 1e-6;   // guards ceil() against ratio*nB landing a hair above an integer

bool aligned(const void* p, size_t n) { return (reinterpret_cast<uintptr_t>(p) % n) == 0; }

int check_problem(const sva_problem* p, Dims* d) {
  if (!p) return SVA_ERR_INVALID_ARG;
  if (p->batch < 1 || p->heads < 1 || p->seq_len < 1 || p->head_dim < 1 || p->block_size < 1)
    return SVA_ERR_INVALID_ARG;
  if (p->grid_t < 1 || p->grid_h < 1 || p->grid_w < 1) return SVA_ERR_INVALID_ARG;
  if (p->out_dtype != SVA_BF16 && p->out_dtype != SVA_F32) return SVA_ERR_INVALID_ARG;
  if (!(p->softmax_scale == p->softmax_scale) || isinf(p->softmax_scale)) return SVA_ERR_INVALID_ARG;
  const int64_t thw = (int64_t)p->grid_t * p->grid_h * p->grid_w;
  if (thw != (int64_t)p->seq_len) return SVA_ERR_SHAPE;
  if (p->head_dim != 64 && p->head_dim != 112 && p->head_dim != 128) return SVA_ERR_UNSUPPORTED;
  if (p->block_size != 64 && p->block_size != 128) return SVA_ERR_UNSUPPORTED;
  const int64_t nB = ((int64_t)p->seq_len + p->block_size - 1) / p->block_size;
  const int64_t rows = (int64_t)p->batch * p->heads * nB;
  if (rows > INT32_MAX) return SVA_ERR_SHAPE;
  // element offsets are formed in 64-bit; the per-head offset bh*N*D must fit too
  const int64_t elems = (int64_t)p->batch * p->heads * p->seq_len * p->head_dim;
  if (elems / p->head_dim / p->seq_len != (int64_t)p->batch * p->heads) return SVA_ERR_SHAPE;
  if ((int64_t)p->batch * p->heads * p->seq_len > INT32_MAX) return SVA_ERR_SHAPE;
  if (d) {
    d->B = p->batch;
    d->H = p->heads;
    d->N = p->seq_len;
    d->D = p->head_dim;
    d->S = p->block_size;
    d->nB = (int)nB;
    d->frame_tokens = (int)((int64_t)p->grid_h * p->grid_w > INT32_MAX ? INT32_MAX
                                                                        : (int64_t)p->grid_h * p->grid_w);
    d->scale = p->softmax_scale > 0.0 ? p->softmax_scale : 1.0 / sqrt((double)p->head_dim);
    d->out_f32 = p->out_dtype == SVA_F32;
  }
  return SVA_OK;
}

int check_tokens(const sva_tokens* t) {
  if (!t) return SVA_ERR_INVALID_ARG;
  if (t->batch < 1 || t->tokens < 1 || t->channels < 8 || t->channels % 8 != 0) return SVA_ERR_INVALID_ARG;
  // row offsets are formed in 64-bit, row counts in 32-bit
  if ((int64_t)t->batch * t->tokens > INT32_MAX) return SVA_ERR_SHAPE;
  return SVA_OK;
}

int check_select(const sva_select_params* s, const Dims& d, SelectRule* r) {
  if (!s) return SVA_ERR_INVALID_ARG;
  SelectRule out{};
  out.mode = s->mode;
  if (s->mode == SVA_SELECT_TOPK) {
    if (s->topk < 0) return SVA_ERR_INVALID_ARG;
    int64_t k;
    if (s->topk > 0) {
      k = s->topk;
    } else {
      if (!(s->keep_ratio > 0.0 && s->keep_ratio <= 1.0)) return SVA_ERR_INVALID_ARG;
      k = (int64_t)ceil(s->keep_ratio * d.nB - kCountEps);
    }
    if (k < 1) k = 1;
    if (k > d.nB) k = d.nB;
    out.k = (int)k;
    out.cap = out.k;
  } else if (s->mode == SVA_SELECT_CUMMASS) {
    if (!(s->mass_threshold > 0.0 && s->mass_threshold <= 1.0)) return SVA_ERR_INVALID_ARG;
    if (!(s->max_keep_ratio > 0.0 && s->max_keep_ratio <= 1.0)) return SVA_ERR_INVALID_ARG;
    int nf = 0;
    if (s->force_first_frame) {
      const int64_t f = ((int64_t)d.frame_tokens + d.S - 1) / d.S;
      nf = (int)(f < d.nB ? f : d.nB);
    }
    int64_t cap = (int64_t)ceil(s->max_keep_ratio * d.nB - kCountEps);
    if (cap > d.nB) cap = d.nB;
    if (cap < nf) cap = nf;
    if (cap < 1) cap = 1;
    out.cap = (int)cap;
    out.n_forced = nf;
    out.tau = s->mass_threshold;
  } else {
    return SVA_ERR_INVALID_ARG;
  }
  if (r) *r = out;
  return SVA_OK;
}

int hip_status(hipError_t e) { return e == hipSuccess ? SVA_OK : SVA_ERR_HIP; }

static_assert(sva::kRemMaxBlocks == SVA_REMAINDER_MAX_BLOCKS, "remainder block limit");

// Byte offsets of the remainder workspace's parts, each 256-byte aligned.
struct RemLayout {
  size_t oa, lsea, kbar, vbar, mom, E, r, T, total;
};

RemLayout rem_layout(const Dims& d) {
  const size_t bh = (size_t)d.B * d.H, N = d.N, D = d.D;
  const size_t nbp = (size_t)sva::rem_padded_blocks(d.nB);
  auto up = [](size_t x) { return (x + 255) & ~(size_t)255; };
  RemLayout L{};
  size_t off = 0;
  L.oa = off;   off += up(bh * N * D * 4);
  L.lsea = off; off += up(bh * N * 4);
  L.kbar = off; off += up(bh * nbp * D * 2);
  L.vbar = off; off += up(bh * nbp * D * 2);
  L.mom = off;  off += up(bh * nbp * D * D * 2);
  L.E = off;    off += up(bh * nbp * (size_t)sva::rem_weight_rows(d.nB) * 2);
  L.r = off;    off += up(bh * nbp * 4);
  L.T = off;    off += up(bh * nbp * D * D * 2);
  L.total = off;
  return L;
}

// The dims of a run of `heads` consecutive (b, h) pairs of d, taken as one
// batch entry of `heads` heads (the kernels index the flattened b*H + h).
Dims group_dims(const Dims& d, int heads) {
  Dims g = d;
  g.B = 1;
  g.H = heads;
  return g;
}

int check_remainder(const sva_problem* prob, Dims* d) {
  const int st = check_problem(prob, d);
  if (st != SVA_OK) return st;
  if (d->nB > sva::kRemMaxBlocks) return SVA_ERR_UNSUPPORTED;
  const int64_t nbp = sva::rem_padded_blocks(d->nB);
  const int64_t bh = (int64_t)d->B * d->H;
  // grids: one workgroup per (b, h, padded block), and per (b, h, column tile, row group)
  if (bh * nbp > INT32_MAX) return SVA_ERR_SHAPE;
  if (bh * ((int64_t)d->D * d->D / 128) * ((d->nB + sva::kRemGemmRows - 1) / sva::kRemGemmRows) > INT32_MAX)
    return SVA_ERR_SHAPE;
  return SVA_OK;
}

}  // namespace

// ---- fp8 (e4m3) quantisation and attention ----

namespace {
int fp8_code_dim(int D) { return (D + 63) / 64 * 64; }

int check_fp8(const sva_problem* prob, Dims* d) {
  const int st = check_problem(prob, d);
  if (st != SVA_OK) return st;
  // (D = 112 is carried as 128 code channels, the last 16 zero)
  // per-head byte ranges of the padded codes are 32-bit buffer offsets
  if ((int64_t)d->nB * d->S * fp8_code_dim(d->D) > INT32_MAX) return SVA_ERR_SHAPE;
  return SVA_OK;
}

int check_fp8_tensors(const sva_fp8_tensors* t, bool need_mean) {
  if (!t || !t->q8 || !t->k8 || !t->v8 || !t->q_exp || !t->k_exp || !t->v_exp) return SVA_ERR_INVALID_ARG;
  if (need_mean && !t->k_mean) return SVA_ERR_INVALID_ARG;
  if (!aligned(t->q8, 16) || !aligned(t->k8, 16) || !aligned(t->v8, 16) || !aligned(t->q_exp, 4) ||
      !aligned(t->k_exp, 4) || !aligned(t->v_exp, 4) || (need_mean && !aligned(t->k_mean, 16)))
    return SVA_ERR_ALIGNMENT;
  return SVA_OK;
}

sva::Fp8AttnArgs fp8_attn_args(const Dims& d, const sva_fp8_tensors* t, const int32_t* kv_idx,
                               const int32_t* kv_count, int32_t kmax, void* out, float* lse) {
  sva::Fp8AttnArgs a{};
  a.q8 = static_cast<const uint8_t*>(t->q8);
  a.k8 = static_cast<const uint8_t*>(t->k8);
  a.v8 = static_cast<const uint8_t*>(t->v8);
  a.q_exp = t->q_exp;
  a.k_exp = t->k_exp;
  a.v_exp = t->v_exp;
  a.kv_idx = kv_idx;
  a.kv_count = kv_count;
  a.kmax = kmax;
  a.out = out;
  a.lse = lse;
  return a;
}
}  // namespace

extern "C" {

int sva_version(void) { return SVA_VERSION_MAJOR * 100 + SVA_VERSION_MINOR; }

const char* sva_status_string(int status) {
  switch (status) {
    case SVA_OK: return "ok";
    case SVA_ERR_INVALID_ARG: return "invalid argument";
    case SVA_ERR_SHAPE: return "inconsistent or oversized shape";
    case SVA_ERR_ALIGNMENT: return "misaligned pointer";
    case SVA_ERR_UNSUPPORTED: return "unsupported head_dim, block_size or block count";
    case SVA_ERR_HIP: return "HIP runtime error at launch";
    default: return "unknown status";
  }
}

int sva_num_blocks(const sva_problem* prob, int32_t* n_blocks) {
  if (!n_blocks) return SVA_ERR_INVALID_ARG;
  Dims d;
  const int st = check_problem(prob, &d);
  if (st != SVA_OK) return st;
  *n_blocks = d.nB;
  return SVA_OK;
}

int sva_max_keep(const sva_problem* prob, const sva_select_params* sel, int32_t* kmax) {
  if (!kmax) return SVA_ERR_INVALID_ARG;
  Dims d;
  int st = check_problem(prob, &d);
  if (st != SVA_OK) return st;
  SelectRule r;
  st = check_select(sel, d, &r);
  if (st != SVA_OK) return st;
  *kmax = r.cap;
  return SVA_OK;
}

int sva_pool_blocks(const sva_problem* prob, const void* q, const void* k, float* q_pool,
                    float* k_pool, void* stream) {
  Dims d;
  const int st = check_problem(prob, &d);
  if (st != SVA_OK) return st;
  if (!q || !k || !q_pool || !k_pool) return SVA_ERR_INVALID_ARG;
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(q_pool, 4) || !aligned(k_pool, 4))
    return SVA_ERR_ALIGNMENT;
  return hip_status(sva::launch_pool(d, static_cast<const uint16_t*>(q),
                                     static_cast<const uint16_t*>(k), q_pool, k_pool,
                                     static_cast<hipStream_t>(stream)));
}

int sva_qknorm_rope_pool(const sva_problem* prob, const sva_rope_params* rope, const void* q_in,
                         const void* k_in, const float* gamma_q, const float* gamma_k, void* q_out,
                         void* k_out, float* q_pool, float* k_pool, void* stream) {
  Dims d;
  const int st = check_problem(prob, &d);
  if (st != SVA_OK) return st;
  if (!rope || !q_in || !k_in || !gamma_q || !gamma_k || !q_out || !k_out || !q_pool || !k_pool)
    return SVA_ERR_INVALID_ARG;
  if (!isfinite(rope->eps) || rope->eps < 0.0 || !isfinite(rope->rope_base) || rope->rope_base <= 1.0)
    return SVA_ERR_INVALID_ARG;
  if (!aligned(q_in, 16) || !aligned(k_in, 16) || !aligned(q_out, 16) || !aligned(k_out, 16) ||
      !aligned(gamma_q, 4) || !aligned(gamma_k, 4) || !aligned(q_pool, 4) || !aligned(k_pool, 4))
    return SVA_ERR_ALIGNMENT;
  // an output is either its input (in place) or disjoint from it
  const size_t bytes = (size_t)d.B * d.H * d.N * d.D * 2;
  auto overlap = [bytes](const void* x, const void* y) {
    const uintptr_t a = reinterpret_cast<uintptr_t>(x), b = reinterpret_cast<uintptr_t>(y);
    return a != b && a < b + bytes && b < a + bytes;
  };
  if (overlap(q_in, q_out) || overlap(k_in, k_out)) return SVA_ERR_INVALID_ARG;
  sva::RopeArgs a{};
  a.q_in = static_cast<const uint16_t*>(q_in);
  a.k_in = static_cast<const uint16_t*>(k_in);
  a.gamma_q = gamma_q;
  a.gamma_k = gamma_k;
  a.q_out = static_cast<uint16_t*>(q_out);
  a.k_out = static_cast<uint16_t*>(k_out);
  a.q_pool = q_pool;
  a.k_pool = k_pool;
  a.grid_h = prob->grid_h;
  a.grid_w = prob->grid_w;
  a.eps = (float)rope->eps;
  a.base = rope->rope_base;
  return hip_status(sva::launch_qknorm_rope_pool(d, a, static_cast<hipStream_t>(stream)));
}

int sva_token_keep_count(const sva_tokens* t, double keep_ratio, int32_t* k) {
  if (!k) return SVA_ERR_INVALID_ARG;
  const int st = check_tokens(t);
  if (st != SVA_OK) return st;
  if (!(keep_ratio > 0.0) || keep_ratio > 1.0) return SVA_ERR_INVALID_ARG;
  int64_t kk = (int64_t)ceil(keep_ratio * t->tokens - kCountEps);
  if (kk < 1) kk = 1;
  if (kk > t->tokens) kk = t->tokens;
  *k = (int32_t)kk;
  return SVA_OK;
}

int sva_token_select_workspace(const sva_tokens* t, size_t* bytes) {
  if (!bytes) return SVA_ERR_INVALID_ARG;
  const int st = check_tokens(t);
  if (st != SVA_OK) return st;
  *bytes = (size_t)t->batch * sva::kTokenSelectWsStride;
  return SVA_OK;
}

int sva_token_select(const sva_tokens* t, double keep_ratio, const void* x, double* scores,
                     int32_t* kept_idx, int32_t* kept_pos, void* workspace, size_t workspace_bytes,
                     void* stream) {
  int32_t k;
  const int st = sva_token_keep_count(t, keep_ratio, &k);
  if (st != SVA_OK) return st;
  if (!x || !scores || !kept_idx || !kept_pos || !workspace) return SVA_ERR_INVALID_ARG;
  if (workspace_bytes < (size_t)t->batch * sva::kTokenSelectWsStride) return SVA_ERR_SHAPE;
  if (!aligned(x, 16) || !aligned(scores, 8) || !aligned(kept_idx, 4) || !aligned(kept_pos, 4) ||
      !aligned(workspace, 8))
    return SVA_ERR_ALIGNMENT;
  return hip_status(sva::launch_token_select(t->batch, t->tokens, t->channels, k,
                                             static_cast<const uint16_t*>(x), scores, kept_idx,
                                             kept_pos, workspace, static_cast<hipStream_t>(stream)));
}

int sva_token_select_noalloc(const sva_tokens* t, double keep_ratio, const void* x, double* scores,
                             int32_t* kept_idx, int32_t* kept_pos, void* stream) {
  static_assert(SVA_TOKEN_SELECT_NOALLOC_MAX_BATCH == sva::kTokenSelectStaticBatch, "static batch");
  int32_t k;
  const int st = sva_token_keep_count(t, keep_ratio, &k);
  if (st != SVA_OK) return st;
  if (!x || !scores || !kept_idx || !kept_pos) return SVA_ERR_INVALID_ARG;
  if (t->batch > SVA_TOKEN_SELECT_NOALLOC_MAX_BATCH) return SVA_ERR_SHAPE;
  if (!aligned(x, 16) || !aligned(scores, 8) || !aligned(kept_idx, 4) || !aligned(kept_pos, 4))
    return SVA_ERR_ALIGNMENT;
  void* ws = nullptr;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  if (sva::token_select_scratch(s, &ws) != hipSuccess) return SVA_ERR_HIP;
  return hip_status(sva::launch_token_select(t->batch, t->tokens, t->channels, k,
                                             static_cast<const uint16_t*>(x), scores, kept_idx,
                                             kept_pos, ws, s));
}

int sva_token_gather(const sva_tokens* t, int32_t k, const void* x, const int32_t* kept_idx,
                     void* x_kept, void* stream) {
  const int st = check_tokens(t);
  if (st != SVA_OK) return st;
  if (k < 1 || k > t->tokens) return SVA_ERR_SHAPE;
  if (!x || !kept_idx || !x_kept) return SVA_ERR_INVALID_ARG;
  if (!aligned(x, 16) || !aligned(x_kept, 16) || !aligned(kept_idx, 4)) return SVA_ERR_ALIGNMENT;
  return hip_status(sva::launch_token_gather(t->batch, t->tokens, t->channels, k,
                                             static_cast<const uint16_t*>(x), kept_idx,
                                             static_cast<uint16_t*>(x_kept),
                                             static_cast<hipStream_t>(stream)));
}

int sva_token_scatter(const sva_tokens* t, int32_t k, const void* y_kept, const int32_t* kept_pos,
                      const void* base, void* out, void* stream) {
  const int st = check_tokens(t);
  if (st != SVA_OK) return st;
  if (k < 1 || k > t->tokens) return SVA_ERR_SHAPE;
  if (!y_kept || !kept_pos || !base || !out) return SVA_ERR_INVALID_ARG;
  if (!aligned(y_kept, 16) || !aligned(base, 16) || !aligned(out, 16) || !aligned(kept_pos, 4))
    return SVA_ERR_ALIGNMENT;
  const uintptr_t o = reinterpret_cast<uintptr_t>(out), y = reinterpret_cast<uintptr_t>(y_kept);
  const size_t out_bytes = (size_t)t->batch * t->tokens * t->channels * 2;
  const size_t y_bytes = (size_t)t->batch * k * t->channels * 2;
  if (o < y + y_bytes && y < o + out_bytes) return SVA_ERR_INVALID_ARG;   // out overlaps y_kept
  const uintptr_t bs = reinterpret_cast<uintptr_t>(base);
  if (bs != o && bs < o + out_bytes && o < bs + out_bytes) return SVA_ERR_INVALID_ARG;
  return hip_status(sva::launch_token_scatter(t->batch, t->tokens, t->channels, k,
                                              static_cast<const uint16_t*>(y_kept), kept_pos,
                                              static_cast<const uint16_t*>(base),
                                              static_cast<uint16_t*>(out),
                                              static_cast<hipStream_t>(stream)));
}

int sva_select_blocks(const sva_problem* prob, const sva_select_params* sel, const float* q_pool,
                      const float* k_pool, int32_t kmax, int32_t* kv_idx, int32_t* kv_count,
                      uint8_t* mask, void* stream) {
  Dims d;
  int st = check_problem(prob, &d);
  if (st != SVA_OK) return st;
  SelectRule r;
  st = check_select(sel, d, &r);
  if (st != SVA_OK) return st;
  if (!q_pool || !k_pool || !kv_idx || !kv_count) return SVA_ERR_INVALID_ARG;
  if (!aligned(q_pool, 4) || !aligned(k_pool, 4) || !aligned(kv_idx, 4) || !aligned(kv_count, 4))
    return SVA_ERR_ALIGNMENT;
  if (d.nB > SVA_SELECT_MAX_BLOCKS) return SVA_ERR_UNSUPPORTED;
  if (kmax < r.cap) return SVA_ERR_SHAPE;
  return hip_status(sva::launch_select(d, r, q_pool, k_pool, kmax, kv_idx, kv_count, mask,
                                       static_cast<hipStream_t>(stream)));
}

int sva_sparse_attention(const sva_problem* prob, const void* q, const void* k, const void* v,
                         const int32_t* kv_idx, const int32_t* kv_count, int32_t kmax, void* out,
                         float* lse, void* stream) {
  Dims d;
  const int st = check_problem(prob, &d);
  if (st != SVA_OK) return st;
  if (!q || !k || !v || !kv_idx || !kv_count || !out) return SVA_ERR_INVALID_ARG;
  if (kmax < 1) return SVA_ERR_SHAPE;
  if ((int64_t)d.B * d.H * d.nB * kmax > ((int64_t)1 << 40)) return SVA_ERR_SHAPE;
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(out, 16) ||
      !aligned(kv_idx, 4) || !aligned(kv_count, 4) || (lse && !aligned(lse, 4)))
    return SVA_ERR_ALIGNMENT;
  return hip_status(sva::launch_attention(
      d, true, static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k),
      static_cast<const uint16_t*>(v), kv_idx, kv_count, kmax, out, lse,
      static_cast<hipStream_t>(stream)));
}

int sva_remainder_workspace(const sva_problem* prob, size_t* bytes) {
  if (!bytes) return SVA_ERR_INVALID_ARG;
  Dims d;
  const int st = check_remainder(prob, &d);
  if (st != SVA_OK) return st;
  *bytes = rem_layout(d).total;
  return SVA_OK;
}

int sva_remainder_workspace_heads(const sva_problem* prob, int32_t heads, size_t* bytes) {
  if (!bytes) return SVA_ERR_INVALID_ARG;
  Dims d;
  const int st = check_remainder(prob, &d);
  if (st != SVA_OK) return st;
  if (heads < 1 || (int64_t)heads > (int64_t)d.B * d.H) return SVA_ERR_SHAPE;
  *bytes = rem_layout(group_dims(d, heads)).total;
  return SVA_OK;
}

int sva_block_moments(const sva_problem* prob, const void* k, const void* v, void* kbar, void* vbar,
                      void* moments, void* stream) {
  Dims d;
  const int st = check_remainder(prob, &d);
  if (st != SVA_OK) return st;
  if (!k || !v || !kbar || !vbar || !moments) return SVA_ERR_INVALID_ARG;
  if (!aligned(k, 16) || !aligned(v, 16) || !aligned(kbar, 16) || !aligned(vbar, 16) || !aligned(moments, 16))
    return SVA_ERR_ALIGNMENT;
  sva::RemMomentArgs a{};
  a.k = static_cast<const uint16_t*>(k);
  a.v = static_cast<const uint16_t*>(v);
  a.kbar = static_cast<uint16_t*>(kbar);
  a.vbar = static_cast<uint16_t*>(vbar);
  a.mom = static_cast<uint16_t*>(moments);
  a.N = d.N;
  a.nB = d.nB;
  a.rows = d.nB;
  return hip_status(sva::launch_block_moments(d, a, static_cast<hipStream_t>(stream)));
}

namespace {

// One pass of the remainder over the (b, h) pairs that d describes, its
// intermediates in the workspace laid out by rem_layout(d).
hipError_t remainder_pass(const Dims& d, const uint16_t* q, const uint16_t* k, const uint16_t* v,
                          const float* q_pool, const float* k_pool, const int32_t* kv_idx, const int32_t* kv_count,
                          int32_t kmax, unsigned char* ws, void* out, float* lse, hipStream_t s) {
  const RemLayout L = rem_layout(d);
  float* oa = reinterpret_cast<float*>(ws + L.oa);
  float* lsea = reinterpret_cast<float*>(ws + L.lsea);
  uint16_t* kbar = reinterpret_cast<uint16_t*>(ws + L.kbar);
  uint16_t* vbar = reinterpret_cast<uint16_t*>(ws + L.vbar);
  uint16_t* mom = reinterpret_cast<uint16_t*>(ws + L.mom);
  const int nbp = sva::rem_padded_blocks(d.nB);

  // the kept blocks exactly, in float32 (merged once, at the end)
  Dims df = d;
  df.out_f32 = true;
  hipError_t e = sva::launch_attention(df, true, q, k, v, kv_idx, kv_count, kmax, oa, lsea, s);
  if (e != hipSuccess) return e;

  sva::RemMomentArgs ma{};
  ma.k = k;
  ma.v = v;
  ma.kbar = kbar;
  ma.vbar = vbar;
  ma.mom = mom;
  ma.N = d.N;
  ma.nB = d.nB;
  ma.rows = nbp;
  if ((e = sva::launch_block_moments(d, ma, s)) != hipSuccess) return e;

  sva::RemWeightArgs wa{};
  wa.q_pool = q_pool;
  wa.k_pool = k_pool;
  wa.kv_idx = kv_idx;
  wa.kv_count = kv_count;
  wa.E = reinterpret_cast<uint16_t*>(ws + L.E);
  wa.r = reinterpret_cast<float*>(ws + L.r);
  wa.nB = d.nB;
  wa.nBp = nbp;
  wa.nBr = sva::rem_weight_rows(d.nB);
  wa.kmax = kmax;
  wa.scale = (float)d.scale;

  sva::RemGemmArgs ga{};
  ga.E = wa.E;
  ga.mom = mom;
  ga.T = reinterpret_cast<uint16_t*>(ws + L.T);
  ga.nB = d.nB;
  ga.nBp = nbp;
  ga.nBr = wa.nBr;
  ga.DD = d.D * d.D;
  ga.n_wg = 0;                      // set by the launcher

  sva::RemAttnArgs aa{};
  aa.q = q;
  aa.kbar = kbar;
  aa.vbar = vbar;
  aa.kv_idx = kv_idx;
  aa.kv_count = kv_count;
  aa.T = ga.T;
  aa.r = wa.r;
  aa.o_a = oa;
  aa.lse_a = lsea;
  aa.out = out;
  aa.lse = lse;
  aa.N = d.N;
  aa.nB = d.nB;
  aa.nBp = nbp;
  aa.kmax = kmax;
  aa.n_rows = 0;                    // set by the launcher
  aa.scale = (float)d.scale;
  aa.scale_log2 = (float)(d.scale * 1.4426950408889634);
  return sva::launch_remainder(d, wa, ga, aa, s);
}

}  // namespace

int sva_sparse_attention_remainder(const sva_problem* prob, const void* q, const void* k, const void* v,
                                   const float* q_pool, const float* k_pool, const int32_t* kv_idx,
                                   const int32_t* kv_count, int32_t kmax, void* workspace,
                                   size_t workspace_bytes, void* out, float* lse, void* stream) {
  Dims d;
  const int st = check_remainder(prob, &d);
  if (st != SVA_OK) return st;
  if (!q || !k || !v || !q_pool || !k_pool || !kv_idx || !kv_count || !workspace || !out)
    return SVA_ERR_INVALID_ARG;
  if (kmax < 1) return SVA_ERR_SHAPE;
  if ((int64_t)d.B * d.H * d.nB * kmax > ((int64_t)1 << 40)) return SVA_ERR_SHAPE;
  // as many (b, h) pairs per pass as the workspace holds: all of them with
  // sva_remainder_workspace bytes, at least one
  const int bh = d.B * d.H;
  int group = bh;
  if (workspace_bytes < rem_layout(d).total) {
    group = (int)std::min<size_t>((size_t)bh, workspace_bytes / std::max<size_t>(1, rem_layout(group_dims(d, 1)).total));
    while (group > 0 && rem_layout(group_dims(d, group)).total > workspace_bytes) --group;
    if (group < 1) return SVA_ERR_SHAPE;
  }
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(out, 16) || !aligned(q_pool, 16) ||
      !aligned(k_pool, 16) || !aligned(kv_idx, 4) || !aligned(kv_count, 4) || (lse && !aligned(lse, 4)) ||
      !aligned(workspace, 256))
    return SVA_ERR_ALIGNMENT;
  hipStream_t s = static_cast<hipStream_t>(stream);
  unsigned char* ws = static_cast<unsigned char*>(workspace);
  const size_t nd = (size_t)d.N * d.D, nbd = (size_t)d.nB * d.D;
  const size_t out_elem = d.out_f32 ? 4 : 2;
  for (int h0 = 0; h0 < bh; h0 += group) {
    const int g = std::min(group, bh - h0);
    const hipError_t e = remainder_pass(
        group_dims(d, g), static_cast<const uint16_t*>(q) + h0 * nd, static_cast<const uint16_t*>(k) + h0 * nd,
        static_cast<const uint16_t*>(v) + h0 * nd, q_pool + h0 * nbd, k_pool + h0 * nbd,
        kv_idx + (size_t)h0 * d.nB * kmax, kv_count + (size_t)h0 * d.nB, kmax, ws,
        static_cast<unsigned char*>(out) + h0 * nd * out_elem, lse ? lse + (size_t)h0 * d.N : nullptr, s);
    if (e != hipSuccess) return SVA_ERR_HIP;
  }
  return SVA_OK;
}

int sva_dense_attention(const sva_problem* prob, const void* q, const void* k, const void* v,
                        void* out, float* lse, void* stream) {
  Dims d;
  const int st = check_problem(prob, &d);
  if (st != SVA_OK) return st;
  if (!q || !k || !v || !out) return SVA_ERR_INVALID_ARG;
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(out, 16) ||
      (lse && !aligned(lse, 4)))
    return SVA_ERR_ALIGNMENT;
  return hip_status(sva::launch_attention(
      d, false, static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k),
      static_cast<const uint16_t*>(v), nullptr, nullptr, 1, out, lse,
      static_cast<hipStream_t>(stream)));
}

int sva_fp8_padded_len(const sva_problem* prob, int32_t* np) {
  if (!np) return SVA_ERR_INVALID_ARG;
  Dims d;
  const int st = check_fp8(prob, &d);
  if (st != SVA_OK) return st;
  *np = d.nB * d.S;
  return SVA_OK;
}

int sva_fp8_code_dim(const sva_problem* prob, int32_t* dp) {
  if (!dp) return SVA_ERR_INVALID_ARG;
  Dims d;
  const int st = check_fp8(prob, &d);
  if (st != SVA_OK) return st;
  *dp = fp8_code_dim(d.D);
  return SVA_OK;
}

int sva_quantize_fp8(const sva_problem* prob, const void* q, const void* k, const void* v,
                     const sva_fp8_tensors* out, void* stream) {
  Dims d;
  int st = check_fp8(prob, &d);
  if (st != SVA_OK) return st;
  if (!q || !k || !v) return SVA_ERR_INVALID_ARG;
  if ((st = check_fp8_tensors(out, true)) != SVA_OK) return st;
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16)) return SVA_ERR_ALIGNMENT;
  sva::Fp8QuantArgs a{};
  a.q = static_cast<const uint16_t*>(q);
  a.k = static_cast<const uint16_t*>(k);
  a.v = static_cast<const uint16_t*>(v);
  a.q8 = static_cast<uint8_t*>(out->q8);
  a.k8 = static_cast<uint8_t*>(out->k8);
  a.v8 = static_cast<uint8_t*>(out->v8);
  a.q_exp = out->q_exp;
  a.k_exp = out->k_exp;
  a.v_exp = out->v_exp;
  a.k_mean = static_cast<uint16_t*>(out->k_mean);
  a.q_mul = (float)(d.scale * 1.4426950408889634);   // the softmax scale in base 2, carried by Q
  return hip_status(sva::launch_quantize_fp8(d, a, static_cast<hipStream_t>(stream)));
}

int sva_sparse_attention_fp8(const sva_problem* prob, const sva_fp8_tensors* in, const int32_t* kv_idx,
                             const int32_t* kv_count, int32_t kmax, void* out, float* lse, void* stream) {
  Dims d;
  int st = check_fp8(prob, &d);
  if (st != SVA_OK) return st;
  if ((st = check_fp8_tensors(in, false)) != SVA_OK) return st;
  if (!kv_idx || !kv_count || !out) return SVA_ERR_INVALID_ARG;
  if (kmax < 1) return SVA_ERR_SHAPE;
  if (kmax > sva::kFp8MaxList) return SVA_ERR_UNSUPPORTED;
  if (!aligned(out, 16) || !aligned(kv_idx, 4) || !aligned(kv_count, 4) || (lse && !aligned(lse, 4)))
    return SVA_ERR_ALIGNMENT;
  return hip_status(sva::launch_attention_fp8(d, true, fp8_attn_args(d, in, kv_idx, kv_count, kmax, out, lse),
                                              static_cast<hipStream_t>(stream)));
}

int sva_dense_attention_fp8(const sva_problem* prob, const sva_fp8_tensors* in, void* out, float* lse,
                            void* stream) {
  Dims d;
  int st = check_fp8(prob, &d);
  if (st != SVA_OK) return st;
  if ((st = check_fp8_tensors(in, false)) != SVA_OK) return st;
  if (!out) return SVA_ERR_INVALID_ARG;
  if (d.nB > sva::kFp8MaxList) return SVA_ERR_UNSUPPORTED;
  if (!aligned(out, 16) || (lse && !aligned(lse, 4))) return SVA_ERR_ALIGNMENT;
  return hip_status(sva::launch_attention_fp8(d, false, fp8_attn_args(d, in, nullptr, nullptr, 1, out, lse),
                                              static_cast<hipStream_t>(stream)));
}

}  // extern "C"
