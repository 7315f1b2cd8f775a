/*
 * flexprefill.h -- C ABI of an MI355X (gfx950) implementation of FlexPrefill's
 * context-aware sparse prefill attention (Lai et al., "FlexPrefill: A Context-Aware
 * Sparse Attention Mechanism for Efficient Long-Sequence Inference", ICLR 2025).
 *
 * Two calls make up the method (Algorithm 1):
 *   fp_select       pattern search (Algorithm 2) + index search (Algorithm 3 for
 *                   vertical-slash heads, Algorithm 4 for query-aware heads),
 *                   producing per-head lists of key blocks for every query block;
 *   fp_sparse_attn  A(Q, K, V, S): causal attention restricted to those blocks
 *                   (Section 2, sparse attention with the mask M_S).
 *
 * Conventions shared by every entry point
 *  - Tensors are packed "THD": Q and O are [T][Hq][d], K and V are [T][Hkv][d],
 *    bf16 (raw 16-bit patterns), d contiguous, T = total tokens of all sequences.
 *    Sequence s occupies tokens [cu_seqlens[s], cu_seqlens[s+1]).
 *  - Query head h reads KV head h / (Hq / Hkv) (grouped-query attention).
 *  - Every device pointer is caller-owned device memory; the library never
 *    allocates, frees, or synchronises, and never throws across the ABI.
 *  - The compute calls enqueue kernel launches only (no memset or copy nodes, no host
 *    waits), so they can be captured into a HIP graph and replayed; the first call of
 *    fp_sparse_attn_noalloc on a device resolves its scratch address and belongs
 *    outside a capture.
 *  - All arguments are checked on the host before anything is enqueued; on a
 *    failed check the first failing status is returned and nothing is enqueued.
 *  - Work is enqueued on `stream` (a hipStream_t; NULL = the default stream) and
 *    completes asynchronously: outputs are valid once the caller has synchronised.
 *  - A launch failure returns FP_ERR_HIP; fp_last_error() then names it.
 *  - Calls that share a workspace or output buffers must not overlap in time.
 */
#ifndef FLEXPREFILL_H
#define FLEXPREFILL_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum fp_status {
  FP_OK = 0,
  FP_ERR_INVALID_ARG = 1,  /* null pointer, bad shape, out-of-range parameter */
  FP_ERR_UNSUPPORTED = 2,  /* valid but not implemented (e.g. head_dim 96)     */
  FP_ERR_WORKSPACE = 3,    /* workspace smaller than the *_workspace_size()   */
  FP_ERR_HIP = 4           /* a HIP runtime call or kernel launch failed       */
} fp_status;

/* Per-head pattern codes written to fp_indices.pattern. */
#define FP_PATTERN_QUERY_AWARE 0    /* Algorithm 4 ("query_specific")            */
#define FP_PATTERN_VERTICAL_SLASH 1 /* Algorithm 3                               */
#define FP_PATTERN_DENSE 2          /* gamma >= 1: every causal block, no search */

#define FP_MAX_BATCH 64             /* sequences per call                        */
#define FP_MAX_MIN_BUDGET 64        /* largest min_budget_blocks accepted        */

/* Problem shape. */
typedef struct fp_shape {
  int32_t batch;              /* number of packed sequences, 1..FP_MAX_BATCH          */
  const int32_t *cu_seqlens;  /* HOST array [batch+1]: cu[0] = 0, non-decreasing;    */
                              /* T = cu[batch]; every sequence has >= 1 token        */
  int32_t num_q_heads;        /* Hq >= 1                                              */
  int32_t num_kv_heads;       /* Hkv >= 1, Hq % Hkv == 0                              */
  int32_t head_dim;           /* d in {64, 128}                                       */
  int32_t block;              /* block_size: 128 (the paper's setting, Section 4.1)  */
                              /* or 64; at most 8192 blocks per sequence             */
} fp_shape;

/* Method parameters (Algorithm 1 inputs tau, gamma; Section 4.1 guards). */
typedef struct fp_params {
  float gamma;                /* cumulative-attention threshold, (0, 1]; gamma >= 1   */
                              /* selects every causal block (full attention)          */
  float tau;                  /* JS-distance threshold, [0, 1]; a head is query-aware */
                              /* iff D_JS < tau (so tau = 0 makes every head VS)      */
  int32_t min_budget_blocks;  /* each query-block row keeps >= min(m, I+1) key        */
                              /* blocks; 0..FP_MAX_MIN_BUDGET (paper: 1024 tokens = 8)*/
  float softmax_scale;        /* 0 => 1/sqrt(head_dim)                                */
  int32_t force_pattern;      /* -1 decide by JS; 0 force query-aware; 1 force VS     */
  int32_t max_budget_blocks;  /* 0: no cap; M >= 2 (and >= min_budget_blocks): every  */
                              /* row keeps <= M key blocks -- 0 and I, then the rest  */
                              /* in top-up order (appendix "maximum budget limit")    */
  int32_t qa_mode;            /* query-aware selection: 0 over the flattened pooled   */
                              /* map (Algorithm 4); 1 per query block, each row of    */
                              /* the map reaching gamma (appendix "flatten ablation") */
  int32_t vs_granularity;     /* vertical-slash lines: 0 token lines (Algorithm 3);   */
                              /* 1 block-pooled: key blocks and offset blocks of      */
                              /* lines are the selection units                        */
} fp_params;

/* Outputs of fp_select (caller-allocated device buffers; sizes from fp_indices_size).
 * Rows are (sequence s, query head h, query block I), I in [0, nb_s), nb_s = ceil(n_s/b).
 *   kb_idx : int32 [kb_idx_elems]; row (s,h,I) starts at
 *            h * TRI + tri_off[s] + I*(I+1)/2, where tri_off[s] = sum_{s'<s} nb_s'(nb_s'+1)/2
 *            and TRI = tri_off[batch]; it holds kb_cnt of that row key-block indices,
 *            strictly ascending, each in [0, I], always containing 0 and I.
 *   kb_cnt : int32 [kb_cnt_elems]; row (s,h,I) at h * NB + nb_off[s] + I,
 *            nb_off[s] = sum_{s'<s} nb_s', NB = nb_off[batch].
 *   pattern: uint8 [batch * Hq], FP_PATTERN_* per (s, h) at s*Hq + h.
 *   js     : float [batch * Hq], D_JS per (s, h) (negative when not computed).
 *   units  : int32 [batch * Hq * 2], per (s, h): {K, 0} for query-aware heads (units
 *            selected by Algorithm 4; with qa_mode 1 the sum over query blocks of
 *            their K), {K_v, K_s} for vertical-slash heads (lines, or blocks of lines
 *            with vs_granularity 1), {all, 0} when dense.
 *            Diagnostics only. */
typedef struct fp_indices {
  int32_t *kb_idx;
  int32_t *kb_cnt;
  uint8_t *pattern;
  float *js;
  int32_t *units;
  float softmax_scale;  /* HOST field: the scale the lists were selected with.  fp_select */
                        /* writes the scale it used (params->softmax_scale, or 1/sqrt(d) */
                        /* when that is 0); fp_sparse_attn attends with this scale (0 =>  */
                        /* 1/sqrt(d)), so selection and attention share one scale.        */
} fp_indices;

/* Element counts of fp_indices.kb_idx and .kb_cnt for `shape`.  Host only. */
fp_status fp_indices_size(const fp_shape *shape, size_t *kb_idx_elems, size_t *kb_cnt_elems);

/* Device workspace bytes needed by fp_select / fp_sparse_attn.  Host only.
 * fp_select: 0 when gamma >= 1 (every causal block is listed without any scoring).
 * fp_sparse_attn: the work order (16 bytes per query head and block), 8 counters, one
 * transposed copy of V (2 * Hkv * NB * block * d bytes, NB = sum of ceil(n_s / block)) and
 * the work order's sort keys and unsorted records (24 bytes per query head and block),
 * written at the start of every call. */
fp_status fp_select_workspace_size(const fp_shape *shape, const fp_params *params,
                                   size_t *bytes);
fp_status fp_attn_workspace_size(const fp_shape *shape, size_t *bytes);

/* Host-only argument check used by fp_select (params != NULL) and fp_sparse_attn
 * (params == NULL): shape, parameters and workspace size.  Touches no device. */
fp_status fp_validate(const fp_shape *shape, const fp_params *params, size_t ws_bytes);

/* Pattern search + index selection (Algorithm 1 up to S; Algorithms 2-4).
 * q: [T][Hq][d] bf16, k: [T][Hkv][d] bf16 (device).  ws: device workspace of
 * ws_bytes >= fp_select_workspace_size().  Enqueues the writes of every device buffer of
 * *out and sets out->softmax_scale on the host. */
fp_status fp_select(const fp_shape *shape, const void *q, const void *k,
                    const fp_params *params, fp_indices *out, void *ws,
                    size_t ws_bytes, void *stream);

/* Block-sparse causal attention O = A(Q, K, V, S) (Section 2): query i of block I
 * attends to keys j <= i whose key block is listed in row (s, h, I) of idx, with the
 * softmax scale idx->softmax_scale (0 => 1/sqrt(d); finite, >= 0).
 * q, o: [T][Hq][d] bf16; k, v: [T][Hkv][d] bf16; idx->kb_idx, idx->kb_cnt as written by
 * fp_select (pattern, js and units unused).  Listed blocks outside [0, I] are skipped; a
 * query row with no visible key gets O = 0. */
fp_status fp_sparse_attn(const fp_shape *shape, const void *q, const void *k,
                         const void *v, const fp_indices *idx, void *o, void *ws,
                         size_t ws_bytes, void *stream);

/* Size of the fixed device scratch array used by fp_sparse_attn_noalloc (one per GPU). */
#define FP_NOALLOC_SCRATCH_BYTES (64u << 20)

/* fp_sparse_attn without a workspace argument, for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc).  Same arguments, result and checks as fp_sparse_attn; the workspace is a
 * fixed FP_NOALLOC_SCRATCH_BYTES device array inside the library (one per GPU, held until
 * the process ends), so the call itself allocates nothing.  Problems whose
 * fp_attn_workspace_size exceeds FP_NOALLOC_SCRATCH_BYTES are rejected with
 * FP_ERR_WORKSPACE before anything is enqueued (fp_last_error() says why).  Every call on
 * one GPU uses the same array: calls that overlap in time on one GPU (other streams, other
 * host threads) race and give undefined results. */
fp_status fp_sparse_attn_noalloc(const fp_shape *shape, const void *q, const void *k,
                                 const void *v, const fp_indices *idx, void *o, void *stream);

/* Static description of a status code. */
const char *fp_status_string(fp_status status);

/* Text of the last FP_ERR_HIP seen by this thread ("" if none). */
const char *fp_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* FLEXPREFILL_H */
