// Internal declarations shared by the host orchestration and the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/flexprefill.h"

namespace fp {

// Longest key chunk owned by one workgroup of the representative-score kernels.  Short
// problems use chunks of 512 or 256 keys (SeqTable::ch_len) so that those kernels still
// get enough workgroups to fill the GPU.
constexpr int kScoreChunk = 1024;
constexpr int kScoreChunkMin = 256;
// workgroups of the line-sum kernel wanted before the chunk is shortened (4 per CU)
constexpr int kScoreWorkgroups = 1024;
constexpr int kHistBuckets = 2048;     // radix-select digit: 11 bits

// Per-call table of packed sequences, passed by value to every kernel.
struct SeqTable {
  int32_t n_seq;
  int32_t max_nb;
  int32_t cu[FP_MAX_BATCH + 1];       // token offsets
  int32_t nb_off[FP_MAX_BATCH + 1];   // prefix sums of nb_s = ceil(n_s / block)
  int32_t ch_len;                     // keys per score chunk: 1024, 512 or 256
  int32_t ch_off[FP_MAX_BATCH + 1];   // prefix sums of ceil(n_s / ch_len)
  int64_t tri_off[FP_MAX_BATCH + 1];  // prefix sums of nb_s (nb_s + 1) / 2
};

// Everything a kernel of the selection pipeline needs.
struct SelectArgs {
  SeqTable st;
  const uint16_t *q;       // [T][Hq][d] bf16
  const uint16_t *k;       // [T][Hkv][d] bf16
  int32_t hq, hkv, d, block;
  int32_t total_tokens;    // T
  int32_t nb_total;        // NB
  int64_t tri_total;       // TRI
  float scale;             // softmax scale
  float gamma, tau;
  int32_t min_budget;
  int32_t force_pattern;
  int32_t max_budget;      // 0 = no cap
  int32_t qa_mode;         // 0 flattened map (Algorithm 4), 1 per query block
  int32_t vs_granularity;  // 0 token lines (Algorithm 3), 1 block-pooled lines
  // workspace
  float2 *chunk_stats;     // [ch_total][Hq][block] (max, sum) in log2 units
  float2 *row_stats;       // [n_seq][Hq][block]
  float *kbar;             // [NB][Hkv][d]
  float *qbar;             // [NB][Hq][d]
  float *a_v;              // [Hq][T]
  float *a_s;              // [Hq][T]
  float *av_blk;           // [Hq][NB] a_v summed per key block (block-pooled lines)
  float *as_blk;           // [Hq][NB] a_s summed per offset block
  float *pat_logit;        // [Hq][NB] scale * q_bar . K_bar_J of the pattern search
  double *pat_ahat;        // [Hq][NB] a_hat[J] = a_v summed per key block
  uint8_t *vs_marks;       // [Hq][NB][4] per key block / diagonal: column, diagonal (full
                           // rows), diagonal (partial last row), diagonal + 1
  float *flat;             // [Hq][TRI]
  struct SelState *sel;    // [n_seq][Hq][2]
  uint32_t *hist_cnt;      // [n_seq][Hq][2][kHistBuckets]
  unsigned long long *hist_mass;  // [n_seq][Hq][2][kHistBuckets]
  // outputs
  int32_t *kb_idx;
  int32_t *kb_cnt;
  uint8_t *pattern;
  float *js;
  int32_t *units;
};

// State of one cumulative-mass selection problem (one score vector).
struct SelState {
  unsigned long long total;       // fixed-point mass of all units
  unsigned long long thr;         // ceil(gamma * total)
  unsigned long long mass_above;  // mass of keys above the current digit range
  uint32_t cnt_above;             // number of keys above the current digit range
  uint32_t prefix;                // key bits fixed so far
  uint32_t key;                   // final threshold key
  uint32_t need_eq;               // units with key == `key` to take (lowest ids first)
  uint32_t n_eq;                  // units with key == `key`
  int32_t idcut;                  // last id taken among key == `key`
  int32_t k;                      // units selected
  int32_t mode;                   // 0 active, 1 take all, 2 inactive (other pattern)
  int32_t n;                      // number of units
  int32_t pad;
};

struct AttnArgs {
  SeqTable st;
  const uint16_t *q, *k, *v;
  uint16_t *o;
  const int32_t *kb_idx;
  const int32_t *kb_cnt;
  int32_t hq, hkv, d, block;
  int32_t nb_total;
  int64_t tri_total;
  float scale_log2;        // softmax scale * log2(e)
  int4 *items;             // [Hkv][G * NB] workspace: ordered item records per KV group
  int32_t *queue;          // [8] workspace: per-XCD work-queue counters
  int32_t mix;             // set by the launcher: an XCD's KV groups served interleaved
  uint16_t *vt;            // [Hkv][NB][B * d] workspace: V^T tiles per key block
  unsigned long long *sort_keys;  // [Hkv][G * NB] workspace: items' sort keys
  int4 *sort_recs;         // [Hkv][G * NB] workspace: item records in item-id order
};

// Device address of the current device's fixed scratch array (fp_noalloc.hip).
hipError_t noalloc_scratch(void **out);

// Launchers (each returns the hipError_t of its launch).
hipError_t launch_sparse_attn(const AttnArgs &a, hipStream_t s);
hipError_t launch_select_pipeline(const SelectArgs &a, hipStream_t s);
hipError_t launch_dense_lists(const SelectArgs &a, hipStream_t s);
hipError_t launch_qa_rows(const SelectArgs &a, hipStream_t s);

}  // namespace fp
