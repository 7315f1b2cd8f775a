// Representative-block attention scores and block pooling for gfx950.
//
// For every (sequence, query head) the last b' = min(block, n) queries Q_hat attend
// causally to all keys (Section 3, "Representative Query Selection"; Algorithm 3 first
// step).  From A_hat = softmax(Q_hat K^T / sqrt d) two line scores are reduced:
//   a_v[j] = sum_r A_hat[r, j] / b'            (vertical lines, Algorithm 3)
//   a_s[o] = sum_r A_hat[r, i_r - o] / b'      (slash lines, offset o = i - j)
// A_hat is never stored: pass 1 computes each row's max and sum of exp per chunk of
// 1024 keys (512 or 256 for short problems, so that the passes still fill the GPU), a
// combine kernel merges the chunks, pass 2 recomputes the scores tile by tile, sums the
// columns in registers (one key per lane) and the diagonals through an LDS tile.  Every
// sum is in a fixed order (no float atomics), so results are bit-reproducible for a given
// shape.  Each pass-2 workgroup owns the slash offsets whose last-row key falls in its
// chunk and recomputes the 128 keys before the chunk so that it sees those diagonals whole.
//
// Block pooling (avgpool with window block_size, aligned at token 0 of each sequence): K̄
// (every KV head) is summed by pass 1 from the K tiles it streams anyway, Q̄ (query-aware
// heads only) by a separate streaming kernel.
#include <type_traits>

#include "fp_internal.h"

namespace fp {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kThreads = 256;
constexpr int KT = 64;             // keys per tile of the statistics pass

__device__ __forceinline__ int seq_of_chunk(const SeqTable &st, int c) {
  int s = 0;
  while (s + 1 < st.n_seq && st.ch_off[s + 1] <= c) ++s;
  return s;
}

__device__ __forceinline__ int seq_of_block(const SeqTable &st, int blk) {
  int s = 0;
  while (s + 1 < st.n_seq && st.nb_off[s + 1] <= blk) ++s;
  return s;
}

template <int D>
__device__ __forceinline__ int k_swz(int chunk, int key) {
  if constexpr (D == 128) return chunk ^ (key & 15);
  else return chunk ^ ((key >> 1) & 7);
}

// Keys [kt, kt + TK) of KV head g (rows past n are zero), staged through the registers of
// NT threads: the next tile is loaded while the current one is in use, then stored to LDS
// swizzled.  The loads go through a buffer resource over the tile's rows that ends at the
// sequence's last key (its range check returns zero past it): the per-thread offset is
// fixed and the tile and iteration steps are scalar.
template <int D, int NT = kThreads, int TK = KT>
struct KTile {
  static constexpr int KCH = D / 8;                     // 16-byte chunks per key
  static constexpr int CH = TK * KCH;                   // chunks per tile
  static constexpr int NIT = CH >= NT ? CH / NT : 1;    // chunks per thread (threads past
                                                        // CH stay idle)
  static_assert(CH < NT || NIT * NT == CH, "tile chunks must divide over the threads");
  static_assert(KCH == 8 || KCH == 16, "head dim 64 or 128");
  uint4 v[NIT];
  __device__ __forceinline__ void load(const uint16_t *kbase, int64_t kv_row, int kt, int n,
                                       int tid) {
    const uint64_t p = (uint64_t)(uintptr_t)(kbase + (int64_t)kt * kv_row);
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)p);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(p >> 32));
    const int row_bytes = (int)kv_row * 2;
    const int nrec = __builtin_amdgcn_readfirstlane(min(TK, n - kt) * row_bytes);
    const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(
        (void *)(uintptr_t)(((uint64_t)hi << 32) | lo), (short)0, nrec, 0x00020000);
    const int voff = (tid / KCH) * row_bytes + (tid % KCH) * 16;
#pragma unroll
    for (int it = 0; it < NIT; ++it) {
      if (CH < NT && tid >= CH) continue;
      const auto x = __builtin_amdgcn_raw_buffer_load_b128(
          r, voff, __builtin_amdgcn_readfirstlane(it * (NT / KCH) * row_bytes), 0);
      v[it] = make_uint4(x[0], x[1], x[2], x[3]);
    }
  }
  __device__ __forceinline__ void store(uint16_t *Ks, int tid) const {
#pragma unroll
    for (int it = 0; it < NIT; ++it) {
      const int c = it * NT + tid;
      if (CH < NT && c >= CH) continue;
      const int key = c / KCH;
      *reinterpret_cast<uint4 *>(Ks + key * D + k_swz<D>(c % KCH, key) * 8) = v[it];
    }
  }
};

// Scores of 64 keys x the wave's 32 query rows: two 32x32 MFMA blocks.  KEY_ROWS: S^T (lane
// holds query row lane % 32 and 16 keys); otherwise S (lane holds key lane % 32 of the
// sub-block and 16 query rows).  The fragments are the same, only the operand order differs.
template <int D, bool KEY_ROWS = true>
__device__ __forceinline__ void tile_scores(const uint16_t *Ks, const bf16x8 *qf, int lr, int lh,
                                            f32x16 *sacc) {
#pragma unroll
  for (int b2 = 0; b2 < 2; ++b2) {
    sacc[b2] = f32x16{};
    const int key = b2 * 32 + lr;
#pragma unroll
    for (int k = 0; k < D / 16; ++k) {
      const bf16x8 kf =
          *reinterpret_cast<const bf16x8 *>(Ks + key * D + k_swz<D>(2 * k + lh, key) * 8);
      if constexpr (KEY_ROWS)
        sacc[b2] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[k], sacc[b2], 0, 0, 0);
      else
        sacc[b2] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qf[k], kf, sacc[b2], 0, 0, 0);
    }
  }
}

// Load the Q_hat^T fragments of the wave's query rows (rows past b' are zero).
template <int D>
__device__ __forceinline__ void load_qhat(const SelectArgs &a, int tok0, int n, int h, int r,
                                          int lh, bf16x8 *qf) {
  const int bp = min(a.block, n);
  if (r < bp) {
    const uint16_t *qp = a.q + ((int64_t)(tok0 + n - bp + r) * a.hq + h) * D + 8 * lh;
#pragma unroll
    for (int k = 0; k < D / 16; ++k) qf[k] = *reinterpret_cast<const bf16x8 *>(qp + 16 * k);
  } else {
#pragma unroll
    for (int k = 0; k < D / 16; ++k) qf[k] = bf16x8{};
  }
}

// ---------------------------------------------------------------- pass 1: row max / sum

// HG query heads of one KV group per workgroup, RW waves of 32 representative rows each
// (4 at block 128, 2 at block 64), sharing every K tile: the chunk's K is read once for HG
// heads (HG = 4 fits in 128 registers per lane, so the 16 waves of a block-128 workgroup
// are resident together).  The workgroup holding the first heads
// of its KV group also writes K̄ for the chunk's key blocks: each thread adds up its
// 16-byte pieces of the block's tiles (all in one column of 8 dimensions), the lanes of a
// wave holding one column are summed by a fixed xor tree, and the waves' partial sums in
// order through LDS.
template <int D, int HG, int RW>
__global__ __launch_bounds__(64 * RW * HG) void rep_stats(SelectArgs a) {
  constexpr int NT = 64 * RW * HG;
  using Tile = KTile<D, NT>;
  constexpr int NSLOT = (Tile::CH < NT ? Tile::CH : NT) / 64;   // waves holding tile pieces
  __shared__ __attribute__((aligned(16))) uint16_t Ks[KT * D];
  __shared__ float kpart[NSLOT][D];          // per wave: sums over its keys of the block
  const int c = blockIdx.x;
  const int h = blockIdx.y * HG + (int)threadIdx.x / (64 * RW);
  const int s = seq_of_chunk(a.st, c);
  const int tok0 = a.st.cu[s];
  const int n = a.st.cu[s + 1] - tok0;
  const int bp = min(a.block, n);
  const int c0 = (c - a.st.ch_off[s]) * a.st.ch_len;
  const int c1 = min(c0 + a.st.ch_len, n);
  const int tid = threadIdx.x, w = (tid >> 6) % RW, lane = tid & 63, lr = lane & 31, lh = lane >> 5;
  const int r = 32 * w + lr;                 // representative row of this lane
  const int irow = n - bp + r;               // its absolute position i_r
  const int G = a.hq / a.hkv;
  const int64_t kv_row = (int64_t)a.hkv * D;
  const uint16_t *kbase = a.k + (int64_t)tok0 * kv_row + (int64_t)(h / G) * D;
  const float sl2 = a.scale * 1.4426950408889634f;

  bf16x8 qf[D / 16];
  load_qhat<D>(a, tok0, n, h, r, lh, qf);
  float m = -INFINITY, l = 0.f;
  // K̄ of this chunk's blocks: by the workgroup of the KV group's first heads
  const bool pool = (blockIdx.y * HG) % G == 0;
  // thread tid's pieces of a tile are chunks it * NT + tid: keys (it * NT + tid) / KCH, all
  // in column tid % KCH (NT is a multiple of KCH)
  float ksum[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  Tile tile;
  tile.load(kbase, kv_row, c0, n, tid);
  for (int kt = c0; kt < c1; kt += KT) {
    __syncthreads();
    // the tile ends a key block (tiles never straddle one: chunks start on a block
    // boundary and KT divides the block)
    const bool block_end = (kt + KT) % a.block == 0 || kt + KT >= c1;
    if (pool) {
#pragma unroll
      for (int it = 0; it < Tile::NIT; ++it) {
        if (Tile::CH < NT && tid >= Tile::CH) continue;     // idle in the tile copy
        const uint32_t wv[4] = {tile.v[it].x, tile.v[it].y, tile.v[it].z, tile.v[it].w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          ksum[2 * i] += __uint_as_float(wv[i] << 16);
          ksum[2 * i + 1] += __uint_as_float(wv[i] & 0xFFFF0000u);
        }
      }
      if (block_end) {
        // the lanes of a wave with one column differ in the lane bits from KCH up: pairs
        // 16 and 32 apart are added by the row and half swaps (lower lane first), 8 apart
        // by a lane shuffle
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          if constexpr (Tile::KCH <= 8) ksum[e] += __shfl_xor(ksum[e], 8);
          const auto r16 = __builtin_amdgcn_permlane16_swap(__float_as_uint(ksum[e]),
                                                            __float_as_uint(ksum[e]), false, false);
          ksum[e] = __uint_as_float(r16[0]) + __uint_as_float(r16[1]);
          const auto r32 = __builtin_amdgcn_permlane32_swap(__float_as_uint(ksum[e]),
                                                            __float_as_uint(ksum[e]), false, false);
          ksum[e] = __uint_as_float(r32[0]) + __uint_as_float(r32[1]);
        }
        if (tid < Tile::CH && lane < Tile::KCH) {
#pragma unroll
          for (int e = 0; e < 8; ++e) kpart[tid / 64][lane * 8 + e] = ksum[e];
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) ksum[e] = 0.f;
      }
    }
    tile.store(Ks, tid);
    __syncthreads();
    if (pool && block_end && tid < D) {
      float sum = 0.f;
#pragma unroll
      for (int q = 0; q < NSLOT; ++q) sum += kpart[q][tid];
      const int J = kt / a.block;
      const int cntk = min(a.block, n - J * a.block);
      a.kbar[((int64_t)(a.st.nb_off[s] + J) * a.hkv + h / G) * D + tid] = sum / (float)cntk;
    }
    if (kt + KT < c1) tile.load(kbase, kv_row, kt + KT, n, tid);   // overlaps this tile
    f32x16 sacc[2];
    tile_scores<D>(Ks, qf, lr, lh, sacc);
    // tile max on the raw scores (the scale is positive and rounding is monotonic, so the
    // scaled max is the max of the scaled scores); the scale is folded into the exponent
    float mr = -INFINITY;
    // masking only in tiles that reach past the chunk, past the first row's position, or
    // in waves holding rows beyond b' (a wave-uniform test)
    const bool edge = kt + KT > c1 || kt + KT - 1 > n - bp + 32 * w || 32 * w + 31 >= bp;
    if (edge) {
#pragma unroll
      for (int b2 = 0; b2 < 2; ++b2)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int j = kt + b2 * 32 + 8 * (v >> 2) + 4 * lh + (v & 3);
          if (j >= c1 || j > irow || r >= bp) sacc[b2][v] = -INFINITY;
          mr = fmaxf(mr, sacc[b2][v]);
        }
    } else {
#pragma unroll
      for (int b2 = 0; b2 < 2; ++b2)
#pragma unroll
        for (int v = 0; v < 16; ++v) mr = fmaxf(mr, sacc[b2][v]);
    }
    const float mn = fmaxf(m, mr * sl2);
    const float mu = (mn == -INFINITY) ? 0.f : mn;
    float acc = 0.f;
#pragma unroll
    for (int b2 = 0; b2 < 2; ++b2)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc += __builtin_amdgcn_exp2f(fmaf(sacc[b2][v], sl2, -mu));
    l = l * __builtin_amdgcn_exp2f(m - mu) + acc;
    m = mn;
  }
  // merge the two lanes that share the row (l and l^32)
  auto pm = __builtin_amdgcn_permlane32_swap(__float_as_uint(m), __float_as_uint(m), false, false);
  auto pl = __builtin_amdgcn_permlane32_swap(__float_as_uint(l), __float_as_uint(l), false, false);
  const float ma = __uint_as_float(pm[0]), mb = __uint_as_float(pm[1]);
  const float la = __uint_as_float(pl[0]), lb = __uint_as_float(pl[1]);
  const float mm = fmaxf(ma, mb);
  const float mu = (mm == -INFINITY) ? 0.f : mm;
  // fixed order: lower half's partial first
  const float lt = la * __builtin_amdgcn_exp2f(ma - mu) + lb * __builtin_amdgcn_exp2f(mb - mu);
  // rows r >= block do not exist (the RW waves cover exactly the block's rows; kept as a guard)
  if (lh == 0 && r < a.block)
    a.chunk_stats[((int64_t)c * a.hq + h) * a.block + r] = make_float2(mm, lt);
}

// (m1, l1) + (m2, l2) in log2 units: the max and the sum of exp2 rescaled to it.
__device__ __forceinline__ float2 merge_stats(float2 p, float2 q) {
  const float mn = fmaxf(p.x, q.x);
  const float mu = (mn == -INFINITY) ? 0.f : mn;
  return make_float2(mn, p.y * __builtin_amdgcn_exp2f(p.x - mu) + q.y * __builtin_amdgcn_exp2f(q.x - mu));
}

// Merge the chunk statistics of each representative row: one wave per row, lane i merges
// chunks i, i + 64, ... in order, then a butterfly over the lanes in which each pair is
// merged lower lane first (every lane computes the same value; the result is fixed).
__global__ __launch_bounds__(256) void rep_stats_combine(SelectArgs a) {
  const int s = blockIdx.x, h = blockIdx.y;
  const int r = blockIdx.z * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (r >= a.block) return;
  float2 acc = make_float2(-INFINITY, 0.f);
  for (int c = a.st.ch_off[s] + lane; c < a.st.ch_off[s + 1]; c += 64)
    acc = merge_stats(acc, a.chunk_stats[((int64_t)c * a.hq + h) * a.block + r]);
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const float2 o = make_float2(__shfl_xor(acc.x, off), __shfl_xor(acc.y, off));
    acc = (lane & off) ? merge_stats(o, acc) : merge_stats(acc, o);
  }
  if (lane == 0) a.row_stats[((int64_t)s * a.hq + h) * a.block + r] = acc;
}

// ---------------------------------------------------------------- pass 2: line sums

// 32-key tiles: each of the RW waves (one per 32 representative rows: 4 at block 128, 2 at
// block 64) computes S = Q_hat K^T for its 32 rows and the tile's 32 keys with one MFMA
// block, so a lane holds one key and 16 rows and the column sums (vertical lines) are
// in-lane adds plus one half-wave swap.  The weights go to an LDS tile whose diagonals
// (slash lines) are summed by the workgroup.  The small tile keeps the LDS and register
// footprint low enough for several workgroups per CU, which hides the latency of the
// barrier-separated phases.
constexpr int LKT = 32;                        // keys per line-pass tile
constexpr int LPITCH = LKT + 1;                // odd pitch: diagonal reads are conflict free
constexpr int LPAD = LKT - 1;                  // zero rows above and below the weight rows

template <int D, int RW>
__global__ __launch_bounds__(64 * RW) __attribute__((amdgpu_waves_per_eu(RW))) void rep_lines(
    SelectArgs a) {
  constexpr int NT = 64 * RW;                  // threads: one wave per 32 representative rows
  constexpr int ROWS = 32 * RW;                // rows of the weight tile (the block size)
  __shared__ __attribute__((aligned(16))) uint16_t Ks[LKT * D];   // K tile
  // Â tile, [row][key], with LPAD zero rows on both sides: every diagonal of the tile is
  // then LKT reads at fixed offsets (the rows past b' hold zero weights)
  __shared__ float Pt[(LPAD + ROWS + LPAD) * LPITCH];
  __shared__ float acc_s[kScoreChunk];         // owned slash offsets
  __shared__ float red[RW][LKT];               // per wave: column sums of the tile
  const int c = blockIdx.x;
  const int h = blockIdx.y;
  const int s = seq_of_chunk(a.st, c);
  const int tok0 = a.st.cu[s];
  const int n = a.st.cu[s + 1] - tok0;
  const int bp = min(a.block, n);
  const int c0 = (c - a.st.ch_off[s]) * a.st.ch_len;
  const int c1 = min(c0 + a.st.ch_len, n);
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, lr = lane & 31, lh = lane >> 5;
  const int r = 32 * w + lr;
  const int G = a.hq / a.hkv;
  const int64_t kv_row = (int64_t)a.hkv * D;
  const uint16_t *kbase = a.k + (int64_t)tok0 * kv_row + (int64_t)(h / G) * D;
  const float sl2 = a.scale * 1.4426950408889634f;
  // a tile column's sum over the waves, in wave order
  auto sum_waves = [&](int col) {
    float sv = red[0][col];
#pragma unroll
    for (int q = 1; q < RW; ++q) sv += red[q][col];
    return sv;
  };

  // Â[r, j] = exp2(s_rj * sl2 - m_r) / (l_r * b') = exp2(s_rj * sl2 - m_r - log2(l_r * b')).
  // Lane (lr, lh) holds key lr of the tile for the 16 rows rv(v) = 32 w + 8 (v / 4) + 4 lh
  // + v % 4.
  // (the 16 row statistics are loaded unconditionally, rows past b' clamped, so that the
  // loads are in flight together)
  float rm[16];
  float2 rst[16];
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const int rv = 32 * w + 8 * (v >> 2) + 4 * lh + (v & 3);
    rst[v] = a.row_stats[((int64_t)s * a.hq + h) * a.block + min(rv, bp - 1)];
  }
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const int rv = 32 * w + 8 * (v >> 2) + 4 * lh + (v & 3);
    rm[v] = rv < bp ? rst[v].x + __builtin_amdgcn_logf(rst[v].y * (float)bp) : 0.f;
  }
  bf16x8 qf[D / 16];
  load_qhat<D>(a, tok0, n, h, r, lh, qf);
  for (int i = tid; i < a.st.ch_len; i += NT) acc_s[i] = 0.f;
  for (int i = tid; i < LPAD * LPITCH; i += NT) {
    Pt[i] = 0.f;
    Pt[(LPAD + ROWS) * LPITCH + i] = 0.f;
  }

  // keys [c0 - ROWS, c0) are recomputed for the diagonals owned by this chunk (a diagonal
  // spans at most b' <= ROWS keys)
  const int kstart = max(c0 - ROWS, 0);
  // two barriers per tile: after the weights (every wave's K reads are then done, so the
  // next K tile, already in registers, is stored over the current one) and after the
  // diagonal pass
  KTile<D, NT, LKT> tile;
  tile.load(kbase, kv_row, kstart, n, tid);
  tile.store(Ks, tid);
  if (kstart + LKT < c1) tile.load(kbase, kv_row, kstart + LKT, n, tid);
  __syncthreads();
  for (int kt = kstart; kt < c1; kt += LKT) {
    f32x16 sacc = {};
#pragma unroll
    for (int k = 0; k < D / 16; ++k) {
      const bf16x8 kf =
          *reinterpret_cast<const bf16x8 *>(Ks + lr * D + k_swz<D>(2 * k + lh, lr) * 8);
      sacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qf[k], kf, sacc, 0, 0, 0);
    }
    // masking only in tiles that reach past the sequence or the first row's position, or
    // in waves holding rows beyond b' (a wave-uniform test)
    const bool edge = kt + LKT > n || kt + LKT - 1 > n - bp + 32 * w || 32 * w + 31 >= bp;
    const int j = kt + lr;
    float cs = 0.f;
    auto weights = [&](auto masked) {
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int rv = 32 * w + 8 * (v >> 2) + 4 * lh + (v & 3);
        float p = __builtin_amdgcn_exp2f(sacc[v] * sl2 - rm[v]);
        if constexpr (decltype(masked)::value)
          p = ((j < n) & (j <= n - bp + rv) & (rv < bp)) ? p : 0.f;
        Pt[(LPAD + rv) * LPITCH + lr] = p;
        cs += p;
      }
    };
    if (edge) weights(std::true_type{});
    else weights(std::false_type{});
    // vertical lines: this lane's 16 rows, then the other lane half's (lower half first),
    // then the four waves in order after the barrier
    if (kt >= c0) {
      const auto pr =
          __builtin_amdgcn_permlane32_swap(__float_as_uint(cs), __float_as_uint(cs), false, false);
      if (lh == 0) red[w][lr] = __uint_as_float(pr[0]) + __uint_as_float(pr[1]);
    }
    __syncthreads();
    if (kt + LKT < c1) {
      tile.store(Ks, tid);
      if (kt + 2 * LKT < c1) tile.load(kbase, kv_row, kt + 2 * LKT, n, tid);   // next-next tile
    }
    // slash lines: diagonal o with last-row key jl = n - 1 - o meets this tile for
    // jl in [kt, kt + LKT + bp - 1); its element in row rr is key jl - (bp - 1) + rr - kt,
    // so starting from row rr0 = bp - 1 - (jl - kt) (which may lie in the zero rows) it is
    // LKT elements at stride LPITCH + 1; eight partial sums in a fixed order
    const int jl = kt + tid;
    if (tid < LKT + bp - 1 && jl >= c0 && jl < c1) {
      const float *dp = Pt + (LPAD + bp - 1 - (jl - kt)) * LPITCH;
      float d[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int i = 0; i < LKT; i += 8)
#pragma unroll
        for (int u = 0; u < 8; ++u) d[u] += dp[(i + u) * (LPITCH + 1)];
      const float ds = ((d[0] + d[1]) + (d[2] + d[3])) + ((d[4] + d[5]) + (d[6] + d[7]));
      acc_s[jl - c0] += ds;
    }
    if (kt >= c0 && tid < LKT) {
      const int jj = kt + tid;
      if (jj < c1)
        a.a_v[(int64_t)h * a.total_tokens + tok0 + jj] =
            sum_waves(tid);
    }
    __syncthreads();
  }
  for (int i = tid; i < c1 - c0; i += NT) {
    const int jl = c0 + i;
    a.a_s[(int64_t)h * a.total_tokens + tok0 + (n - 1 - jl)] = acc_s[i];
  }
}

// ---------------------------------------------------------------- block pooling

// out[(blk) * H + head][d] = mean over the block's tokens of x[token][head][d].
// Launched with grid (NB, H); heads whose pattern differs from `only_pattern` are
// skipped when `pattern` is non-null.
template <int D>
__global__ __launch_bounds__(kThreads) void pool_blocks(SeqTable st, const uint16_t *x, int H,
                                                        int block, float *out,
                                                        const uint8_t *pattern, int hq,
                                                        int only_pattern) {
  constexpr int CH = D / 8;              // 16-byte chunks per row
  constexpr int PH = kThreads / CH;      // token phases
  __shared__ float part[PH][D];
  const int blk = blockIdx.x, head = blockIdx.y;
  const int s = seq_of_block(st, blk);
  if (pattern && pattern[s * hq + head] != only_pattern) return;
  const int tok0 = st.cu[s];
  const int n = st.cu[s + 1] - tok0;
  const int J = blk - st.nb_off[s];
  const int t0 = J * block;
  const int cntk = min(block, n - t0);
  const int tid = threadIdx.x, ch = tid % CH, ph = tid / CH;
  float acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  for (int t = ph; t < cntk; t += PH) {
    const uint4 v = *reinterpret_cast<const uint4 *>(x + ((int64_t)(tok0 + t0 + t) * H + head) * D +
                                                     ch * 8);
    const uint32_t wv[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      acc[2 * i] += __uint_as_float(wv[i] << 16);
      acc[2 * i + 1] += __uint_as_float(wv[i] & 0xFFFF0000u);
    }
  }
#pragma unroll
  for (int i = 0; i < 8; ++i) part[ph][ch * 8 + i] = acc[i];
  __syncthreads();
  if (tid < D) {
    float sum = 0.f;
    for (int p = 0; p < PH; ++p) sum += part[p][tid];
    out[((int64_t)blk * H + head) * D + tid] = sum / (float)cntk;
  }
}

}  // namespace

hipError_t launch_rep_scores(const SelectArgs &a, hipStream_t stream) {
  const int ch_total = a.st.ch_off[a.st.n_seq];
  dim3 grid(ch_total, a.hq);
  // 4 (or 2) query heads of one KV group per workgroup when the group size allows
  const int G = a.hq / a.hkv;
  int hg = G % 4 == 0 ? 4 : (G % 2 == 0 ? 2 : 1);
  // short problems: fewer heads per workgroup, so that the grid still covers the GPU
  while (hg > 1 && (int64_t)ch_total * (a.hq / hg) < 512) hg /= 2;
  // one wave per 32 representative rows: 4 per head at block 128, 2 at block 64
  const int rw = a.block == 64 ? 2 : 4;
  const dim3 grid_g(ch_total, a.hq / hg), block_g(64 * rw * hg);
  auto stats = [&](auto dc, auto rwc) {
    constexpr int D = decltype(dc)::value, RW = decltype(rwc)::value;
    if (hg == 4) hipLaunchKernelGGL((rep_stats<D, 4, RW>), grid_g, block_g, 0, stream, a);
    else if (hg == 2) hipLaunchKernelGGL((rep_stats<D, 2, RW>), grid_g, block_g, 0, stream, a);
    else hipLaunchKernelGGL((rep_stats<D, 1, RW>), grid_g, block_g, 0, stream, a);
  };
  using I128 = std::integral_constant<int, 128>;
  using I64 = std::integral_constant<int, 64>;
  using I4 = std::integral_constant<int, 4>;
  using I2 = std::integral_constant<int, 2>;
  if (a.d == 128) {
    if (rw == 4) stats(I128{}, I4{});
    else stats(I128{}, I2{});
  } else {
    if (rw == 4) stats(I64{}, I4{});
    else stats(I64{}, I2{});
  }
  hipLaunchKernelGGL(rep_stats_combine, dim3(a.st.n_seq, a.hq, (a.block + 3) / 4), dim3(256), 0,
                     stream, a);
  if (a.d == 128) {
    if (rw == 4) hipLaunchKernelGGL((rep_lines<128, 4>), grid, dim3(64 * rw), 0, stream, a);
    else hipLaunchKernelGGL((rep_lines<128, 2>), grid, dim3(64 * rw), 0, stream, a);
  } else {
    if (rw == 4) hipLaunchKernelGGL((rep_lines<64, 4>), grid, dim3(64 * rw), 0, stream, a);
    else hipLaunchKernelGGL((rep_lines<64, 2>), grid, dim3(64 * rw), 0, stream, a);
  }
  return hipGetLastError();
}

hipError_t launch_pool_q_query_aware(const SelectArgs &a, hipStream_t stream) {
  if (a.d == 128)
    hipLaunchKernelGGL(pool_blocks<128>, dim3(a.nb_total, a.hq), dim3(kThreads), 0, stream, a.st,
                       a.q, a.hq, a.block, a.qbar, (const uint8_t *)a.pattern, a.hq,
                       FP_PATTERN_QUERY_AWARE);
  else
    hipLaunchKernelGGL(pool_blocks<64>, dim3(a.nb_total, a.hq), dim3(kThreads), 0, stream, a.st,
                       a.q, a.hq, a.block, a.qbar, (const uint8_t *)a.pattern, a.hq,
                       FP_PATTERN_QUERY_AWARE);
  return hipGetLastError();
}

}  // namespace fp
