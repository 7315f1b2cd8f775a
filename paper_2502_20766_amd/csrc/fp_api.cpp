// Host side of the C ABI: argument checks, workspace layout, launch order.
//
// Nothing here allocates device memory or synchronises: every call validates on the host,
// carves the caller's workspace, and enqueues kernels on the caller's stream.
#include <math.h>
#include <stdio.h>
#include <string.h>

#include "fp_internal.h"

namespace {

thread_local char g_last_error[256] = "";

constexpr size_t kAlign = 256;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

struct Dims {
  fp::SeqTable st;
  int64_t total_tokens;
  int64_t nb_total;
  int64_t tri_total;
  int64_t ch_total;
};

fp_status check_shape(const fp_shape *sh, Dims *dm) {
  if (!sh || !sh->cu_seqlens) return FP_ERR_INVALID_ARG;
  if (sh->batch < 1 || sh->num_q_heads < 1 || sh->num_kv_heads < 1 || sh->head_dim < 1 ||
      sh->block < 1)
    return FP_ERR_INVALID_ARG;
  if (sh->num_q_heads % sh->num_kv_heads != 0) return FP_ERR_INVALID_ARG;
  if (sh->batch > FP_MAX_BATCH) return FP_ERR_UNSUPPORTED;
  if (sh->head_dim != 64 && sh->head_dim != 128) return FP_ERR_UNSUPPORTED;
  if (sh->block != 128 && sh->block != 64) return FP_ERR_UNSUPPORTED;
  if (sh->num_kv_heads > 1024 || sh->num_q_heads > 8192) return FP_ERR_UNSUPPORTED;
  if (sh->cu_seqlens[0] != 0) return FP_ERR_INVALID_ARG;
  memset(dm, 0, sizeof(*dm));
  fp::SeqTable &st = dm->st;
  st.n_seq = sh->batch;
  // score chunk: the longest of 1024, 512, 256 keys that still gives the line-sum kernel
  // kScoreWorkgroups (sequence chunk, query head) workgroups
  st.ch_len = fp::kScoreChunkMin;
  for (int len = fp::kScoreChunk; len > fp::kScoreChunkMin; len /= 2) {
    int64_t chunks = 0;
    for (int s = 0; s < sh->batch; ++s)
      chunks += ((int64_t)sh->cu_seqlens[s + 1] - sh->cu_seqlens[s] + len - 1) / len;
    if (chunks * sh->num_q_heads >= fp::kScoreWorkgroups) {
      st.ch_len = len;
      break;
    }
  }
  int64_t nb_acc = 0, tri_acc = 0, ch_acc = 0;
  int max_nb = 0;
  for (int s = 0; s < sh->batch; ++s) {
    const int64_t n = (int64_t)sh->cu_seqlens[s + 1] - sh->cu_seqlens[s];
    if (n < 1) return FP_ERR_INVALID_ARG;
    const int64_t nb = (n + sh->block - 1) / sh->block;
    if (nb > 8192) return FP_ERR_UNSUPPORTED;   // up to 1M tokens (512k at block 64)
    st.cu[s] = sh->cu_seqlens[s];
    st.nb_off[s] = (int32_t)nb_acc;
    st.tri_off[s] = tri_acc;
    st.ch_off[s] = (int32_t)ch_acc;
    nb_acc += nb;
    tri_acc += nb * (nb + 1) / 2;
    ch_acc += (n + st.ch_len - 1) / st.ch_len;
    if (nb > max_nb) max_nb = (int)nb;
  }
  const int64_t T = sh->cu_seqlens[sh->batch];
  if (T > (int64_t)0x7FFFFFFF / 2) return FP_ERR_UNSUPPORTED;
  if (nb_acc > (1 << 20)) return FP_ERR_UNSUPPORTED;
  st.cu[sh->batch] = (int32_t)T;
  st.nb_off[sh->batch] = (int32_t)nb_acc;
  st.tri_off[sh->batch] = tri_acc;
  st.ch_off[sh->batch] = (int32_t)ch_acc;
  st.max_nb = max_nb;
  dm->total_tokens = T;
  dm->nb_total = nb_acc;
  dm->tri_total = tri_acc;
  dm->ch_total = ch_acc;
  // the flattened per-head index space must stay addressable with int32 offsets per head
  if (tri_acc * (int64_t)sh->num_q_heads > ((int64_t)1 << 40)) return FP_ERR_UNSUPPORTED;
  return FP_OK;
}

// A softmax scale argument: finite and >= 0 (0 selects 1 / sqrt(d)).
bool scale_ok(float s) { return s >= 0.f && !isnan(s) && !isinf(s); }
float resolved_scale(float s, int head_dim) {
  return s > 0.f ? s : 1.0f / sqrtf((float)head_dim);
}

fp_status check_params(const fp_shape *sh, const fp_params *p) {
  if (!(p->gamma > 0.f) || !(p->gamma <= 1.f) || isnan(p->gamma)) return FP_ERR_INVALID_ARG;
  if (!(p->tau >= 0.f) || !(p->tau <= 1.f)) return FP_ERR_INVALID_ARG;
  if (p->min_budget_blocks < 0) return FP_ERR_INVALID_ARG;
  if (p->min_budget_blocks > FP_MAX_MIN_BUDGET) return FP_ERR_UNSUPPORTED;
  if (!scale_ok(p->softmax_scale)) return FP_ERR_INVALID_ARG;
  if (p->force_pattern < -1 || p->force_pattern > 1) return FP_ERR_INVALID_ARG;
  if (p->max_budget_blocks < 0 || p->max_budget_blocks == 1) return FP_ERR_INVALID_ARG;
  if (p->max_budget_blocks > 0 && p->max_budget_blocks < p->min_budget_blocks)
    return FP_ERR_INVALID_ARG;
  if (p->qa_mode < 0 || p->qa_mode > 1) return FP_ERR_INVALID_ARG;
  if (p->vs_granularity < 0 || p->vs_granularity > 1) return FP_ERR_INVALID_ARG;
  (void)sh;
  return FP_OK;
}

// Workspace layout of fp_select; returns the total size, fills pointers when base != 0.
size_t select_layout(const fp_shape *sh, const Dims &dm, char *base, fp::SelectArgs *a) {
  const int64_t hq = sh->num_q_heads, hkv = sh->num_kv_heads, d = sh->head_dim, b = sh->block;
  const int64_t problems = (int64_t)sh->batch * hq * 2;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = align_up(off + bytes);
    return base ? base + o : nullptr;
  };
  char *chunk_stats = take(sizeof(float2) * dm.ch_total * hq * b);
  char *row_stats = take(sizeof(float2) * sh->batch * hq * b);
  char *kbar = take(sizeof(float) * dm.nb_total * hkv * d);
  char *qbar = take(sizeof(float) * dm.nb_total * hq * d);
  char *a_v = take(sizeof(float) * hq * dm.total_tokens);
  char *a_s = take(sizeof(float) * hq * dm.total_tokens);
  char *av_blk = take(sizeof(float) * hq * dm.nb_total);
  char *as_blk = take(sizeof(float) * hq * dm.nb_total);
  char *pat_logit = take(sizeof(float) * hq * dm.nb_total);
  char *pat_ahat = take(sizeof(double) * hq * dm.nb_total);
  char *vs_marks = take(4 * hq * dm.nb_total);
  char *flat = take(sizeof(float) * hq * dm.tri_total);
  char *sel = take(sizeof(fp::SelState) * problems);
  char *hist_cnt = take(sizeof(uint32_t) * problems * fp::kHistBuckets);
  char *hist_mass = take(sizeof(unsigned long long) * problems * fp::kHistBuckets);
  if (a) {
    a->chunk_stats = (float2 *)chunk_stats;
    a->row_stats = (float2 *)row_stats;
    a->kbar = (float *)kbar;
    a->qbar = (float *)qbar;
    a->a_v = (float *)a_v;
    a->a_s = (float *)a_s;
    a->av_blk = (float *)av_blk;
    a->as_blk = (float *)as_blk;
    a->pat_logit = (float *)pat_logit;
    a->pat_ahat = (double *)pat_ahat;
    a->vs_marks = (uint8_t *)vs_marks;
    a->flat = (float *)flat;
    a->sel = (fp::SelState *)sel;
    a->hist_cnt = (uint32_t *)hist_cnt;
    a->hist_mass = (unsigned long long *)hist_mass;
  }
  return off;
}

// attention workspace: ordered item records [Hq][NB] int4, 8 queue counters, then the V^T
// tiles [Hkv][NB][block * d] bf16
// Attention workspace: ordered item records (16 B per query head and block), 8 queue
// counters, V^T tiles, and the items' sort keys (8 B) and records in id order (16 B).
size_t attn_layout(const fp_shape *sh, const Dims &dm) {
  const size_t items = (size_t)dm.nb_total * sh->num_q_heads;
  return align_up(16 * items) + align_up(8 * sizeof(int32_t)) +
         align_up(2 * (size_t)dm.nb_total * sh->num_kv_heads * sh->block * sh->head_dim) +
         align_up(8 * items) + align_up(16 * items);
}

fp_status hip_fail(hipError_t e, const char *what) {
  snprintf(g_last_error, sizeof(g_last_error), "%s: %s", what, hipGetErrorString(e));
  return FP_ERR_HIP;
}

}  // namespace

extern "C" {

fp_status fp_indices_size(const fp_shape *shape, size_t *kb_idx_elems, size_t *kb_cnt_elems) {
  Dims dm;
  fp_status st = check_shape(shape, &dm);
  if (st != FP_OK) return st;
  if (!kb_idx_elems || !kb_cnt_elems) return FP_ERR_INVALID_ARG;
  *kb_idx_elems = (size_t)(dm.tri_total * shape->num_q_heads);
  *kb_cnt_elems = (size_t)(dm.nb_total * shape->num_q_heads);
  return FP_OK;
}

fp_status fp_select_workspace_size(const fp_shape *shape, const fp_params *params,
                                   size_t *bytes) {
  Dims dm;
  fp_status st = check_shape(shape, &dm);
  if (st != FP_OK) return st;
  if (!params || !bytes) return FP_ERR_INVALID_ARG;
  if ((st = check_params(shape, params)) != FP_OK) return st;
  *bytes = params->gamma >= 1.f ? 0 : select_layout(shape, dm, nullptr, nullptr);
  return FP_OK;
}

fp_status fp_attn_workspace_size(const fp_shape *shape, size_t *bytes) {
  Dims dm;
  fp_status st = check_shape(shape, &dm);
  if (st != FP_OK) return st;
  if (!bytes) return FP_ERR_INVALID_ARG;
  *bytes = attn_layout(shape, dm);
  return FP_OK;
}

fp_status fp_validate(const fp_shape *shape, const fp_params *params, size_t ws_bytes) {
  Dims dm;
  fp_status st = check_shape(shape, &dm);
  if (st != FP_OK) return st;
  if (params) {
    if ((st = check_params(shape, params)) != FP_OK) return st;
    const size_t need = params->gamma >= 1.f ? 0 : select_layout(shape, dm, nullptr, nullptr);
    if (ws_bytes < need) return FP_ERR_WORKSPACE;
  } else {
    if (ws_bytes < attn_layout(shape, dm)) return FP_ERR_WORKSPACE;
  }
  return FP_OK;
}

fp_status fp_select(const fp_shape *shape, const void *q, const void *k, const fp_params *params,
                    fp_indices *out, void *ws, size_t ws_bytes, void *stream) {
  fp_status st = fp_validate(shape, params, ws_bytes);
  if (st != FP_OK) return st;
  if (!q || !k || !out || !out->kb_idx || !out->kb_cnt || !out->pattern || !out->js ||
      !out->units)
    return FP_ERR_INVALID_ARG;
  Dims dm;
  check_shape(shape, &dm);
  fp::SelectArgs a;
  memset(&a, 0, sizeof(a));
  a.st = dm.st;
  a.q = (const uint16_t *)q;
  a.k = (const uint16_t *)k;
  a.hq = shape->num_q_heads;
  a.hkv = shape->num_kv_heads;
  a.d = shape->head_dim;
  a.block = shape->block;
  a.total_tokens = (int32_t)dm.total_tokens;
  a.nb_total = (int32_t)dm.nb_total;
  a.tri_total = dm.tri_total;
  a.scale = resolved_scale(params->softmax_scale, shape->head_dim);
  a.gamma = params->gamma;
  a.tau = params->tau;
  a.min_budget = params->min_budget_blocks;
  a.force_pattern = params->force_pattern;
  a.max_budget = params->max_budget_blocks;
  a.qa_mode = params->qa_mode;
  a.vs_granularity = params->vs_granularity;
  a.kb_idx = out->kb_idx;
  a.kb_cnt = out->kb_cnt;
  a.pattern = out->pattern;
  a.js = out->js;
  a.units = out->units;
  out->softmax_scale = a.scale;
  hipStream_t s = (hipStream_t)stream;
  hipError_t e;
  if (params->gamma >= 1.f) {
    e = fp::launch_dense_lists(a, s);
    return e == hipSuccess ? FP_OK : hip_fail(e, "fp_select(dense)");
  }
  if (!ws) return FP_ERR_INVALID_ARG;
  select_layout(shape, dm, (char *)ws, &a);
  e = fp::launch_select_pipeline(a, s);
  return e == hipSuccess ? FP_OK : hip_fail(e, "fp_select");
}

fp_status fp_sparse_attn(const fp_shape *shape, const void *q, const void *k, const void *v,
                         const fp_indices *idx, void *o, void *ws, size_t ws_bytes,
                         void *stream) {
  fp_status st = fp_validate(shape, nullptr, ws_bytes);
  if (st != FP_OK) return st;
  if (!q || !k || !v || !o || !idx || !idx->kb_idx || !idx->kb_cnt || !ws)
    return FP_ERR_INVALID_ARG;
  if (!scale_ok(idx->softmax_scale)) return FP_ERR_INVALID_ARG;
  Dims dm;
  check_shape(shape, &dm);
  fp::AttnArgs a;
  memset(&a, 0, sizeof(a));
  a.st = dm.st;
  a.q = (const uint16_t *)q;
  a.k = (const uint16_t *)k;
  a.v = (const uint16_t *)v;
  a.o = (uint16_t *)o;
  a.kb_idx = idx->kb_idx;
  a.kb_cnt = idx->kb_cnt;
  a.hq = shape->num_q_heads;
  a.hkv = shape->num_kv_heads;
  a.d = shape->head_dim;
  a.block = shape->block;
  a.nb_total = (int32_t)dm.nb_total;
  a.tri_total = dm.tri_total;
  a.scale_log2 = resolved_scale(idx->softmax_scale, shape->head_dim) * 1.4426950408889634f;
  a.items = (int4 *)ws;
  a.queue = (int32_t *)((char *)ws + align_up(16 * dm.nb_total * shape->num_q_heads));
  a.vt = (uint16_t *)((char *)a.queue + align_up(8 * sizeof(int32_t)));
  a.sort_keys = (unsigned long long *)((char *)a.vt +
                                       align_up(2 * (size_t)dm.nb_total * shape->num_kv_heads *
                                                shape->block * shape->head_dim));
  a.sort_recs = (int4 *)((char *)a.sort_keys + align_up(8 * dm.nb_total * shape->num_q_heads));
  hipError_t e = fp::launch_sparse_attn(a, (hipStream_t)stream);
  return e == hipSuccess ? FP_OK : hip_fail(e, "fp_sparse_attn");
}

fp_status fp_sparse_attn_noalloc(const fp_shape *shape, const void *q, const void *k,
                                 const void *v, const fp_indices *idx, void *o, void *stream) {
  Dims dm;
  fp_status st = check_shape(shape, &dm);
  if (st != FP_OK) return st;
  const size_t need = attn_layout(shape, dm);
  if (need > (size_t)FP_NOALLOC_SCRATCH_BYTES) {
    snprintf(g_last_error, sizeof(g_last_error),
             "fp_sparse_attn_noalloc: the problem needs %zu workspace bytes, more than the "
             "fixed scratch of %zu",
             need, (size_t)FP_NOALLOC_SCRATCH_BYTES);
    return FP_ERR_WORKSPACE;
  }
  if (!q || !k || !v || !o || !idx || !idx->kb_idx || !idx->kb_cnt) return FP_ERR_INVALID_ARG;
  if (!scale_ok(idx->softmax_scale)) return FP_ERR_INVALID_ARG;
  void *ws = nullptr;
  const hipError_t e = fp::noalloc_scratch(&ws);
  if (e != hipSuccess) return hip_fail(e, "fp_sparse_attn_noalloc(scratch)");
  return fp_sparse_attn(shape, q, k, v, idx, o, ws, (size_t)FP_NOALLOC_SCRATCH_BYTES, stream);
}

const char *fp_status_string(fp_status status) {
  switch (status) {
    case FP_OK: return "FP_OK";
    case FP_ERR_INVALID_ARG: return "FP_ERR_INVALID_ARG: invalid argument";
    case FP_ERR_UNSUPPORTED: return "FP_ERR_UNSUPPORTED: configuration not supported";
    case FP_ERR_WORKSPACE: return "FP_ERR_WORKSPACE: workspace too small";
    case FP_ERR_HIP: return "FP_ERR_HIP: HIP runtime error";
  }
  return "unknown fp_status";
}

const char *fp_last_error(void) { return g_last_error; }

}  // extern "C"
