// Block-sparse causal flash-attention forward for gfx950: O = A(Q, K, V, S).
//
// A(Q, K, V, S) is the sparse attention of Section 2 of the FlexPrefill paper: softmax over
// the keys of S_i only (mask M_S = -inf elsewhere), with S_i inside the causal set j <= i.
// S is given at block granularity: for every (sequence, query head, query block I) an
// ascending list of key blocks J <= I.
//
// One workgroup = one (sequence, query head, query block) row of B queries; B/32 waves of
// 32 query rows each.  Per selected key block, in stages of B/2 keys:
//   * K tile [keys][d] is staged in LDS row-major with a 16-byte-chunk XOR swizzle;
//   * V is transposed once per call (VtTile / store_vt, in the preparation launch) into
//     16-key steps of V^T, [step][d][16 keys], already in the swizzled LDS order, so its
//     stage copy is linear and each V^T fragment is one conflict-free ds_read_b128;
//   * S^T = K Q^T on v_mfma_f32_32x32x16_bf16 (Q^T fragments live in registers), so each
//     lane owns one query row and half of the stage's keys: the row max needs one lane
//     swap.  K rows are read with bits 2 and 3 of the row index swapped, which makes the
//     keys a lane holds in S^T exactly the 8 consecutive keys its P^T B-operand needs;
//   * online softmax in the log2 domain (exp2 with log2(e) folded into the scale); a row's
//     reference max moves (with the O rescale) only when a score rises more than 2^8 in
//     weight terms above it, so most stages skip the rescale;
//   * the two LDS stage buffers alternate within each key block (every row takes an even
//     number of stages), so the unrolled stage pair reads them at constant offsets;
//   * O^T += V^T P^T on the same MFMA, and O^T keeps one query row per lane, so the
//     rescale by exp2(m_old - m_new) is per lane.
// A persistent grid walks each KV group's (sequence, query head, query block) items in a
// locality order (longest lists first in buckets, lists that start alike adjacent), every
// group served by the same XCD(s), so that items running together share K/V tiles in L2.
#include <algorithm>
#include <type_traits>

#include "fp_internal.h"
#include "fp_sort.h"

namespace fp {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));

// Block size B (queries per query block = keys per key block) is 128 or 64.  A workgroup
// is one query block: B/32 waves of 32 query rows.  Keys go through LDS in stages of B/2
// keys (two stages per key block), each stage made of 32-key MFMA sub-blocks.
template <int B>
struct Geo {
  static constexpr int WAVES = B / 32;
  static constexpr int THREADS = 64 * WAVES;
  static constexpr int KEYS = B / 2;            // keys per stage
  static constexpr int SUB = KEYS / 32;         // 32-key sub-blocks per stage
  static constexpr int WG_PER_CU = 512 / THREADS;  // two waves per SIMD
};

__device__ __forceinline__ float wave_pair_max(float x) {
  // lanes l and l^32 exchange values; max of both halves of the swap is symmetric
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

__device__ __forceinline__ float wave_pair_sum(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// acc + the sum of N 16-key steps' bf16 weights -- exactly the values the P V products
// use -- two per v_dot2_f32_bf16 against (1, 1), steps in order.
template <int N>
__device__ __forceinline__ float sum_weights(const bf16x8 (&pf)[N], float acc) {
  const bf16x2 one = {(__bf16)1.0f, (__bf16)1.0f};
#pragma unroll
  for (int i = 0; i < N; ++i)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const bf16x2 pair = {pf[i][2 * e], pf[i][2 * e + 1]};
      acc = __builtin_amdgcn_fdot2_f32_bf16(pair, one, acc, false);
    }
  return acc;
}

// Geometry of one stage in LDS: K row-major [key][d], V^T as [16-key step][d][16 keys]
// (bf16, 16-byte units placed by vt_unit).
template <int D, int B>
struct Stage {
  static constexpr int RB = 2 * D;                 // bytes per key row
  static constexpr int CPR = RB / 16;              // 16-byte chunks per row
  static constexpr int KEYS = Geo<B>::KEYS;
  static constexpr int BYTES = KEYS * RB;          // one tile (K or V)
  static constexpr int RPI = 1024 / RB;            // rows written by one wave-wide DMA
  static constexpr int DMA_PER_WAVE = BYTES / 1024 / Geo<B>::WAVES;
};

// 16-byte chunk swizzles (XOR, so the same function maps logical <-> physical).
// K: the 32 rows read by one half-wave at the same chunk land on distinct banks.
template <int D>
__device__ __forceinline__ int swz_k(int y, int r) {
  if constexpr (D == 128) return y ^ (r & 15);
  else return y ^ ((r >> 1) & 7);
}
// V^T: 16-byte unit of (head dim d, key half lh) inside one 16-key step of 2 d units per d.
// The 16 lanes that read one step at the same lh (d = d0 .. d0 + 15) land in 16 distinct
// 16-byte bank groups, and so do each 8 of them; the placement is additive in d / 32 and
// in the step, so a lane's reads differ only by immediate offsets.
__device__ __forceinline__ int vt_unit(int d, int lh) {
  return 16 * (d >> 3) + 8 * (lh ^ ((d >> 3) & 1)) + (d & 7);
}

// Per-lane byte offsets of the DMA slots of one stage, relative to the stage's first key
// row (K) or first byte (V^T): slot i of wave w covers LDS bytes [(DMA_PER_WAVE w + i)
// * 1024, +1024); for K lane l fills 16 bytes of tile row r with the logical chunk whose
// swizzled position is the lane's slot, for V^T (stored in LDS order) the copy is linear.
// A wave's slots are contiguous so that one M0 value serves all of them: the instruction's
// immediate offset (i * 1024) moves both the LDS destination and the source address, and
// the per-lane offsets below have it taken off.  The descriptor's range check applies to
// the sum, so K rows past the valid range still read as zero.
template <int D, int B>
struct DmaOffsets {
  uint32_t k[Stage<D, B>::DMA_PER_WAVE];
  uint32_t v;
};

template <int D, int B>
__device__ __forceinline__ DmaOffsets<D, B> dma_offsets(uint32_t row_bytes, int w, int lane) {
  using S = Stage<D, B>;
  DmaOffsets<D, B> o;
#pragma unroll
  for (int i = 0; i < S::DMA_PER_WAVE; ++i) {
    const int q = w * S::DMA_PER_WAVE + i;
    const int r = q * S::RPI + lane / S::CPR;
    const int phys = lane % S::CPR;
    o.k[i] = r * row_bytes + swz_k<D>(phys, r) * 16 - i * 1024;
  }
  o.v = w * S::DMA_PER_WAVE * 1024 + lane * 16;
  return o;
}

// Buffer descriptor over [base, base + nrec) with out-of-range reads returning zero.  The
// inputs are made wave-uniform first so the descriptor always lives in scalar registers
// (a descriptor the compiler believes divergent would be issued once per distinct lane
// value in a loop).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t uniform_rsrc(const void *base, int nrec) {
  const uint64_t p = (uint64_t)(uintptr_t)base;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)p);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(p >> 32));
  return __builtin_amdgcn_make_buffer_rsrc((void *)(uintptr_t)(((uint64_t)hi << 32) | lo),
                                           (short)0, __builtin_amdgcn_readfirstlane(nrec),
                                           0x00020000);
}

// Wave-wide 16-byte DMAs into LDS slots I .. N-1, slot i at i * 1024 past `dst` (the
// immediate offset moves the source address by the same amount), with a per-lane offset
// per slot (K) or one shared by all slots (V^T).
template <int I, int N>
__device__ __forceinline__ void dma_slots(__amdgpu_buffer_rsrc_t r,
                                          __attribute__((address_space(3))) void *dst,
                                          const uint32_t *voff) {
  if constexpr (I < N) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, dst, 16, voff[I], 0, I * 1024, 0);
    dma_slots<I + 1, N>(r, dst, voff);
  }
}
template <int I, int N>
__device__ __forceinline__ void dma_slots(__amdgpu_buffer_rsrc_t r,
                                          __attribute__((address_space(3))) void *dst,
                                          uint32_t voff) {
  if constexpr (I < N) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, dst, 16, voff, 0, I * 1024, 0);
    dma_slots<I + 1, N>(r, dst, voff);
  }
}

// Issue the DMA of one stage: keys k0 .. k0+KEYS-1 of the sequence, K through a buffer
// descriptor whose range ends at the last valid key row (rows past the sequence end read
// as zeros and are masked by the caller), V^T as the stage's contiguous tile (zero past
// the sequence end).
template <int D, int B>
__device__ __forceinline__ void stage_dma(uint8_t *ks, uint8_t *vs, const uint16_t *kbase,
                                          const uint16_t *vt_tile, int64_t kv_row, int k0,
                                          int kvalid, const DmaOffsets<D, B> &off) {
  using S = Stage<D, B>;
  const int nrec = (kvalid - 1) * (int)kv_row * 2 + 2 * D;
  const __amdgpu_buffer_rsrc_t rk = uniform_rsrc(kbase + (int64_t)k0 * kv_row, nrec);
  const __amdgpu_buffer_rsrc_t rv = uniform_rsrc(vt_tile, S::BYTES);
  static_assert((S::DMA_PER_WAVE - 1) * 1024 < 4096, "immediate offsets are 12 bits");
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  auto *kd = (__attribute__((address_space(3))) void *)(ks + w * S::DMA_PER_WAVE * 1024);
  auto *vd = (__attribute__((address_space(3))) void *)(vs + w * S::DMA_PER_WAVE * 1024);
  dma_slots<0, S::DMA_PER_WAVE>(rk, kd, off.k);
  dma_slots<0, S::DMA_PER_WAVE>(rv, vd, off.v);
}

// Small LDS accesses whose ordering against the in-flight LDS DMA is handled by the
// caller (so the compiler adds no vmcnt wait of its own).
__device__ __forceinline__ int lds_read_i32(uint32_t addr) {
  int v;
  asm volatile("ds_read_b32 %0, %1\n\ts_waitcnt lgkmcnt(0)" : "=v"(v) : "v"(addr));
  return v;
}
__device__ __forceinline__ int4 lds_read_i32x4(uint32_t addr) {
  int4 v;
  asm volatile("ds_read_b128 %0, %1\n\ts_waitcnt lgkmcnt(0)" : "=v"(v) : "v"(addr));
  return v;
}
__device__ __forceinline__ void lds_write_i32(uint32_t addr, int v) {
  asm volatile("ds_write_b32 %0, %1" ::"v"(addr), "v"(v) : "memory");
}

// One unit of work: the B queries of (sequence s, query head h, query block I).
struct Row {
  int valid;
  int I, h, g, cnt, tok0, n;
  int nb0;                        // global index of the sequence's first key block
  int J0, J1;                     // first two listed key blocks (-1 if absent)
  const __attribute__((address_space(4))) int32_t *list;
};

constexpr int kChunk = 16;   // consecutive ordered items kept together on one XCD
constexpr int kMixItems = 8;    // at most this many items per workgroup: groups interleaved
constexpr float kLazyLog2 = 8.f;  // rise of a row's max (log2 units) that moves its reference

// Item v of XCD x's work queue -> (KV group g, index j into g's ordered items), false once
// the queue is exhausted (every later v is then exhausted too).
//  * Hkv a multiple of 4, at least 8: XCDs x and x + 4 serve groups x % 4, x % 4 + 4, ... in
//    turn, each group's ordered items dealt to the two in alternate chunks of kChunk.  Only
//    4 groups' K/V are then read at a time, a working set that fits the last-level cache
//    (8 Llama-3-8B groups at 128k hold 512 MB of K/V), and similar items stay on one L2;
//  * Hkv divides 8: the 8/Hkv XCDs that share group g = x mod Hkv take its ordered items in
//    chunks of kChunk, dealt round-robin, so similar items stay on one XCD's L2;
//  * otherwise XCD x takes the whole lists of groups x, x + 8, ... in turn (XCDs without a
//    group only steal).
// With `mix` (short problems: few items per workgroup) an XCD that serves several groups
// takes their items alternately, one from each, instead of one group after the other: each
// group's items are ordered longest first, so the longest items of every group start in
// the first round instead of the later groups' after the earlier groups' short ones.
__device__ __forceinline__ bool queue_item(int x, int v, int hkv, int n_g, int mix, int &g,
                                           int &j) {
  if (hkv % 4 == 0 && hkv >= 8) {
    const int half = x >> 2;                        // which XCD of the pair
    const int nch = (n_g + kChunk - 1) / kChunk;    // chunks per group
    int taken = ((nch - half + 1) / 2) * kChunk;    // items of one group this XCD takes
    if (((nch - 1) & 1) == half) taken -= nch * kChunk - n_g;   // it holds the short chunk
    if (taken <= 0) return false;
    int q, vv;
    if (mix) {                                      // the XCD's groups item by item
      const int ng = hkv / 4;
      if (v >= ng * taken) return false;
      q = v % ng;
      vv = v / ng;
    } else {                                        // one group after the other
      q = v / taken;
      vv = v % taken;
    }
    g = (x & 3) + 4 * q;
    j = ((vv / kChunk) * 2 + half) * kChunk + vv % kChunk;
    return g < hkv && j < n_g;
  }
  if (8 % hkv == 0) {
    const int r = 8 / hkv;
    g = x % hkv;
    j = ((v / kChunk) * r + x / hkv) * kChunk + v % kChunk;
    return j < n_g;
  }
  if (mix) {                                        // the XCD's groups item by item
    const int ng = x < hkv ? (hkv - x + 7) / 8 : 0;
    if (v >= ng * n_g) return false;
    g = x + 8 * (v % ng);
    j = v / ng;
    return true;
  }
  g = x + 8 * (v / n_g);
  j = v % n_g;
  return g < hkv;
}

// Item record: {sequence s (6 bits) | query head within the group kk (13) | query block I
// (13), listed blocks (clamped to I + 1), first listed block, second listed block (-1 when
// absent)}.
__device__ __forceinline__ int4 item_record(const SeqTable &st, const int32_t *kb_idx,
                                            const int32_t *kb_cnt, int nb_total,
                                            int64_t tri_total, int G, int g, int s, int kk,
                                            int I) {
  const int h = g * G + kk;
  const int cnt = max(0, min(kb_cnt[(int64_t)h * nb_total + st.nb_off[s] + I], I + 1));
  const int32_t *list = kb_idx + (int64_t)h * tri_total + st.tri_off[s] + (int64_t)I * (I + 1) / 2;
  int4 r;
  r.x = (int)(((uint32_t)s << 26) | ((uint32_t)kk << 13) | (uint32_t)I);
  r.y = cnt;
  r.z = cnt > 0 ? list[0] : -1;
  r.w = cnt > 1 ? list[1] : -1;
  return r;
}

__device__ __forceinline__ const __attribute__((address_space(4))) int32_t *
row_list(const AttnArgs &a, int h, int s, int I) {
  return (const __attribute__((address_space(4))) int32_t *)(a.kb_idx + (int64_t)h * a.tri_total +
                                                           a.st.tri_off[s] +
                                                           (int64_t)I * (I + 1) / 2);
}

// The same row with every field made wave-uniform (readfirstlane), so that the compiler
// keeps it in scalar registers whatever control flow it came through.
__device__ __forceinline__ Row uniform_row(const Row &r) {
  Row u;
  u.valid = __builtin_amdgcn_readfirstlane(r.valid);
  u.I = __builtin_amdgcn_readfirstlane(r.I);
  u.h = __builtin_amdgcn_readfirstlane(r.h);
  u.g = __builtin_amdgcn_readfirstlane(r.g);
  u.cnt = __builtin_amdgcn_readfirstlane(r.cnt);
  u.tok0 = __builtin_amdgcn_readfirstlane(r.tok0);
  u.n = __builtin_amdgcn_readfirstlane(r.n);
  u.nb0 = __builtin_amdgcn_readfirstlane(r.nb0);
  u.J0 = __builtin_amdgcn_readfirstlane(r.J0);
  u.J1 = __builtin_amdgcn_readfirstlane(r.J1);
  const uint64_t p = (uint64_t)(uintptr_t)r.list;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)p);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(p >> 32));
  u.list = (const __attribute__((address_space(4))) int32_t *)(uintptr_t)(((uint64_t)hi << 32) | lo);
  return u;
}

// First key of stage `half` of key block J in row r, or -1 when the stage has no keys.
template <int B>
__device__ __forceinline__ int stage_first_key(const Row &r, int J, int half) {
  if (J < 0 || J > r.I) return -1;
  const int k0 = J * B + Geo<B>::KEYS * half;
  return k0 < r.n ? k0 : -1;
}

// Persistent kernel: gridDim.x workgroups, all resident; workgroup b first takes item b / 8
// of the queue of XCD x = b % 8 (the XCD the hardware places it on), then pulls the next
// items of that queue through an atomic counter and, once it is empty, those of the other
// XCDs' queues in turn.  The stages of consecutive rows form one
// stream: the next row's identity and block list are fetched over the current row's
// stages (one dependent step per stage, each step's loads covered by the wait for the
// stage's K/V copy) and its first K/V copy is issued at the top of the current row's last
// stage.
template <int D, int B>
__global__ __launch_bounds__(Geo<B>::THREADS) __attribute__((amdgpu_waves_per_eu(2, 2)))
void sparse_fa_fwd(AttnArgs a) {
  using S = Stage<D, B>;
  constexpr int BM = B;                   // queries per workgroup (one query block)
  constexpr int KS = D / 16;
  constexpr int DB = D / 32;
  __shared__ __attribute__((aligned(1024))) uint8_t lds[4 * S::BYTES];  // [2 stages][K, V]
  __shared__ int fetch_slot[2];           // queue positions handed from thread 0 to all
  __shared__ __attribute__((aligned(16))) int4 rec_slot;   // next row's item record

  const int G = a.hq / a.hkv;
  const int n_g = G * a.nb_total;         // items per KV group
  const int P = gridDim.x;                // a multiple of 8
  const int P8 = P / 8;                   // items per queue taken by the first wave of rows
  const int x0 = blockIdx.x & 7;
  const int tid = threadIdx.x;
  const int w = tid >> 6;
  const int lane = tid & 63;
  const int lr = lane & 31;
  const int lh = lane >> 5;
  const int qrow = 32 * w + lr;           // this lane's query row within the block
  const float c = a.scale_log2;
  // a rise of kLazyLog2 in log2 units, in raw logit units (c > 0; clamped to stay finite)
  const float lazy_raw = fminf(kLazyLog2 / c, 3.0e38f);
  const int64_t kv_row = (int64_t)a.hkv * D;  // elements between consecutive tokens

  // a row from its item record {packed (s, kk, I), blocks, first block, second block}
  auto row_from = [&](int g, int32_t packed, int cnt, int j0, int j1) {
    Row r;
    const int s = (uint32_t)packed >> 26;
    r.valid = 1;
    r.g = g;
    r.h = g * G + ((packed >> 13) & 0x1FFF);
    r.I = packed & 0x1FFF;
    r.tok0 = a.st.cu[s];
    r.n = a.st.cu[s + 1] - r.tok0;
    r.nb0 = a.st.nb_off[s];
    r.cnt = cnt;
    r.J0 = j0;
    r.J1 = j1;
    r.list = row_list(a, r.h, s, r.I);
    return r;
  };

  // ---- first row: item blockIdx / 8 of this XCD's queue, read directly
  Row cur;
  cur.valid = 0;
  {
    int g, j;
    if (queue_item(x0, blockIdx.x >> 3, a.hkv, n_g, a.mix, g, j)) {
      const int4 rec = a.items[(int64_t)g * n_g + j];
      cur = row_from(g, __builtin_amdgcn_readfirstlane(rec.x), __builtin_amdgcn_readfirstlane(rec.y),
                     __builtin_amdgcn_readfirstlane(rec.z), __builtin_amdgcn_readfirstlane(rec.w));
    }
  }

  // ---- next-row fetch, spread over the current row:
  //   row setup: thread 0 takes a queue position (atomic), retired with the row's Q loads
  //              and published in LDS                                       -> fs 1
  //   fs 1 (first stage top, after the barrier): position known; if that queue is empty,
  //         positions of the next queues are taken right away; else lanes 0-3 of wave 0
  //         copy the item record into LDS (LDS DMA)                         -> fs 2
  //   fs 2 (next stage top, covered by its wait and barrier): next row complete -> fs 4
  // No load result stays in flight in a register across the stage loop (the compiler
  // would otherwise wait for it, and with it for the K/V DMA, inside the stages).
  // The next row is kept as its raw item record (and KV group) until it is used: the
  // derived Row fields would hold scalar registers over the whole current row.
  int nxt_valid = 0, nxt_g = 0, nxt_x = 0, nxt_y = 0, nxt_z = 0, nxt_w = 0;
  auto next_row = [&]() { return row_from(nxt_g, nxt_x, nxt_y, nxt_z, nxt_w); };
  int fs = 4, qi = 0, n_fetch = 0, fetch_g = 0;
  const uint32_t rec_off = 4u * (uint32_t)(tid & 3);   // record dword of lanes 0-3
  const uint32_t slot_addr =
      (uint32_t)(uintptr_t)(__attribute__((address_space(3))) int *)fetch_slot;
  const uint32_t rec_addr =
      (uint32_t)(uintptr_t)(__attribute__((address_space(3))) int4 *)&rec_slot;
  // workgroup barrier without a memory fence: the callers wait for exactly the memory
  // operations the other waves depend on (LDS DMA by vmcnt, LDS writes by lgkmcnt)
  auto barrier = [&]() {
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
  };
  // thread 0 takes the next position of queue (x0 + qi) and publishes it in slot n_fetch;
  // the atomic's return is consumed at once (the caller places this where a wait is paid
  // anyway)
  auto take_position = [&]() {
    if (tid == 0) {
      const int p = atomicAdd(a.queue + ((x0 + qi) & 7), 1);
      lds_write_i32(slot_addr + 4 * (n_fetch & 1), p);
    }
    // the fetch state stays wave-uniform across the thread-0 branch above
    qi = __builtin_amdgcn_readfirstlane(qi);
    n_fetch = __builtin_amdgcn_readfirstlane(n_fetch);
  };
  // one step; call after a barrier that follows the publication of slot n_fetch
  auto fetch_step = [&]() {
    if (fs == 1) {
      while (true) {
        qi = __builtin_amdgcn_readfirstlane(qi);
        const int x = (x0 + qi) & 7;
        const int v =
            P8 + __builtin_amdgcn_readfirstlane(lds_read_i32(slot_addr + 4 * (n_fetch & 1)));
        ++n_fetch;
        int g, j;
        if (queue_item(x, v, a.hkv, n_g, a.mix, g, j)) {
          fetch_g = g;
          if (tid < 4) {
            const __amdgpu_buffer_rsrc_t rr = uniform_rsrc(a.items + (int64_t)g * n_g + j, 16);
            __builtin_amdgcn_raw_ptr_buffer_load_lds(
                rr, (__attribute__((address_space(3))) void *)&rec_slot, 4, rec_off, 0, 0, 0);
          }
          fs = 2;
          fetch_g = __builtin_amdgcn_readfirstlane(fetch_g);
          n_fetch = __builtin_amdgcn_readfirstlane(n_fetch);
          qi = __builtin_amdgcn_readfirstlane(qi);
          break;
        }
        if (++qi == 8) {                // every queue drained: no next row
          fs = 4;
          break;
        }
        take_position();                // rare: this queue is empty, try the next one now
        barrier();
      }
    } else if (fs == 2) {
      const int4 rec = lds_read_i32x4(rec_addr);
      nxt_valid = 1;
      nxt_g = fetch_g;
      nxt_x = __builtin_amdgcn_readfirstlane(rec.x);
      nxt_y = __builtin_amdgcn_readfirstlane(rec.y);
      nxt_z = __builtin_amdgcn_readfirstlane(rec.z);
      nxt_w = __builtin_amdgcn_readfirstlane(rec.w);
      fs = 4;
    }
    // (the compiler's uniformity analysis does not always see through the loop above)
    fs = __builtin_amdgcn_readfirstlane(fs);
    qi = __builtin_amdgcn_readfirstlane(qi);
    n_fetch = __builtin_amdgcn_readfirstlane(n_fetch);
    nxt_valid = __builtin_amdgcn_readfirstlane(nxt_valid);
  };
  // complete the fetch now (rows with fewer stages than fetch steps)
  auto fetch_finish = [&]() {
    while (fs < 4) {
      if (fs == 2) {
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        barrier();
      }
      fetch_step();
    }
  };
  auto load_q = [&](const Row &r, bf16x8 (&qf)[KS]) {
    const int qr = min(r.I * BM + qrow, r.n - 1);
    const uint16_t *qp = a.q + ((int64_t)(r.tok0 + qr) * a.hq + r.h) * D + 8 * lh;
#pragma unroll
    for (int k = 0; k < KS; ++k) qf[k] = *reinterpret_cast<const bf16x8 *>(qp + 16 * k);
  };

  const DmaOffsets<D, B> doff = dma_offsets<D, B>((uint32_t)(kv_row * 2), w, lane);
  // per-lane V^T fragment address (relative to a V^T stage) of d-block 0, step 0: d-block
  // db adds 1 KB, step t adds 32 D bytes
  const uint32_t vaddr_rel = 16 * vt_unit(lr, lh);
  // per-lane K fragment addresses (relative to a K stage) of sub-block 0; sub-block 1 is
  // 32 rows further (the swizzles repeat every 32 rows).  MFMA row lr reads key row
  // kr = lr with bits 2 and 3 swapped, so that S^T element v of lane (lr, lh) is key
  // 16 (v / 8) + 8 lh + v % 8 of the sub-block.
  const int kr = (lr & ~12) | ((lr >> 1) & 4) | ((lr << 1) & 8);
  uint32_t kaddr_rel[KS];
#pragma unroll
  for (int k = 0; k < KS; ++k) kaddr_rel[k] = kr * S::RB + swz_k<D>(2 * k + lh, kr) * 16;
  const uint32_t lds_base = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint8_t *)lds;
  auto issue = [&](const Row &r, int k0, int into) {
    const uint16_t *kb = a.k + (int64_t)r.tok0 * kv_row + (int64_t)r.g * D;
    const int jb = r.nb0 + (int)((uint32_t)k0 / B), koff = (int)((uint32_t)k0 % B);
    const uint16_t *vt = a.vt + ((int64_t)(r.g * a.nb_total + jb) * B + koff) * D;
    uint8_t *dst = lds + into * 2 * S::BYTES;
    stage_dma<D, B>(dst, dst + S::BYTES, kb, vt, kv_row, k0, min(S::KEYS, r.n - k0), doff);
  };

  if (!cur.valid) {                       // this XCD's queue had no first item: take one
    take_position();
    fs = 1;
    barrier();
    fetch_finish();
    if (!nxt_valid) return;
    cur = next_row();
    nxt_valid = 0;
  }
  int k0_next = stage_first_key<B>(cur, cur.J0, 0);
  if (k0_next >= 0) issue(cur, k0_next, 0);
  bf16x8 qf[KS];
  while (true) {
    // ---- row setup: Q^T fragments (lane owns query row q0 + qrow), zero state
    cur = uniform_row(cur);
    const int q0 = cur.I * BM;
    // the next row's queue position and this row's Q fragments load together, and both are
    // retired here: the stage loop then holds no pending register load, so the compiler
    // adds no wait before its MFMAs (which would also wait for the K/V DMA)
    if (qi < 8) {
      take_position();
      fs = 1;
    }
    fs = __builtin_amdgcn_readfirstlane(fs);
    load_q(cur, qf);
#pragma unroll
    for (int k = 0; k < KS; ++k) asm volatile("" : "+v"(qf[k]));
    f32x16 oacc[DB];
#pragma unroll
    for (int i = 0; i < DB; ++i) oacc[i] = f32x16{};
    float m_ref = -INFINITY;   // reference max (raw logit units) of this lane's row
    float mc = 0.f;             // m_ref * c (0 while m_ref is -inf)
    float m_trig = -INFINITY;   // m_ref + lazy_raw: a score above it moves the reference
    float l_run = 0.f;          // this lane's share of the row sum of the bf16 weights
    int J_cur = cur.J0;         // block of the stage being prefetched
    int J_pre = cur.J1;         // block after it
    // stage t covers keys J*B + (B/2)*(t&1) .. of block J = list[t >> 1]; a row with no
    // blocks still takes two (empty) stages so that its zero output is written.  Every row
    // has an even number of stages, so even stages read LDS buffer 0 and odd ones buffer 1;
    // the loop is unrolled by two, which makes each buffer's read offsets constants.
    const int n_stages = 2 * max(cur.cnt, 1);
    auto stage = [&](auto cbc, const int t) {
      const int CB = cbc;                        // LDS buffer of this stage's K/V tiles
      const int k0 = k0_next;
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // this wave's DMA of stage t landed
      barrier();                        // ... and every wave's; stage t-1 reads are done
      fetch_step();
      // the next stage is the row's next one, or the first stage of the next row
      k0_next = -1;
      if (t + 1 < n_stages) {
        if (CB == 0) {
          k0_next = stage_first_key<B>(cur, J_cur, 1);
        } else {
          J_cur = J_pre;
          J_pre = ((t >> 1) + 2 < cur.cnt) ? cur.list[(t >> 1) + 2] : -1;
          k0_next = stage_first_key<B>(cur, J_cur, 0);
        }
        if (k0_next >= 0) issue(cur, k0_next, CB ^ 1);
      } else {
        fetch_finish();
        if (nxt_valid) {
          const Row nr = next_row();
          k0_next = stage_first_key<B>(nr, nr.J0, 0);
          if (k0_next >= 0) issue(nr, k0_next, CB ^ 1);
        }
      }
      if (k0 < 0) return;
      const int kq = k0 - q0;             // key offset relative to the query block start
      const bool diag = kq >= 0;          // diagonal block: keys after the query are masked
      uint32_t ka[KS];                    // this stage's K fragment LDS addresses (sub-block 0)
#pragma unroll
      for (int k = 0; k < KS; ++k) ka[k] = lds_base + CB * 2 * S::BYTES + kaddr_rel[k];
      f32x16 sacc[2];
      auto qk_block = [&](auto b2c) {
        constexpr int b2 = decltype(b2c)::value;
        sacc[b2] = f32x16{};
        bf16x8 kf[KS];            // all K fragments in flight before the first MFMA
#pragma unroll
        for (int k = 0; k < KS; ++k)
          kf[k] = *reinterpret_cast<const bf16x8 *>(lds + (ka[k] - lds_base) + b2 * 32 * S::RB);
#pragma unroll
        for (int k = 0; k < KS; ++k)
          sacc[b2] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[k], qf[k], sacc[b2], 0, 0, 0);
      };
      // Move the reference max, rescaling O and the row sums, only when some row of the wave
      // sees a score more than kLazyLog2 (log2 units) above it; smaller rises keep the old
      // reference, so weights stay below 2^kLazyLog2 (bf16 and the float32 sums hold them
      // with the same relative precision as weights below 1) and most stages skip the
      // rescale.  While a row's reference is -inf its trigger is -inf too, so its first
      // visible score moves it; a row with no visible key keeps -inf (weights 0).  `mt` is
      // this lane's max over its half of the row's stage keys: the two lanes of a row share
      // the trigger, so the wave-wide vote needs no exchange, and only a moving reference
      // takes the row max across the lane pair.
      auto update_max = [&](float mt) {
        if (__ballot(mt > m_trig)) {
          const float m_new = fmaxf(m_ref, wave_pair_max(mt));
          const float alpha = __builtin_amdgcn_exp2f((m_ref - m_new) * c);
          const float a2 = (m_ref == m_new) ? 1.f : alpha;
          l_run *= a2;
#pragma unroll
          for (int i = 0; i < DB; ++i) oacc[i] *= a2;
          m_ref = m_new;
          const bool none = m_new == -INFINITY;
          mc = none ? 0.f : m_new * c;
          m_trig = none ? -INFINITY : m_new + lazy_raw;
        }
      };
      // ---- O^T += V^T P^T, 16 keys per step; one ds_read_b128 per V^T fragment
      const uint8_t *vs = lds + (CB * 2 + 1) * S::BYTES + vaddr_rel;
      auto pv_step = [&](auto tc, const bf16x8 &pf) {
        constexpr int t = decltype(tc)::value;
        bf16x8 vf[DB];
#pragma unroll
        for (int db = 0; db < DB; ++db)
          vf[db] = *reinterpret_cast<const bf16x8 *>(vs + db * 1024 + t * 32 * D);
#pragma unroll
        for (int db = 0; db < DB; ++db)
          oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[db], pf, oacc[db], 0, 0, 0);
      };
      // ---- the stage's scores, one running-max update for all its keys, the bf16 weights
      // (P^T steps of 16 keys) and their sum, then O^T += V^T P^T
      constexpr int SB = Geo<B>::SUB;
      qk_block(std::integral_constant<int, 0>{});
      if constexpr (SB == 2) qk_block(std::integral_constant<int, 1>{});
      if (diag) {
#pragma unroll
        for (int b2 = 0; b2 < SB; ++b2)
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int key = kq + b2 * 32 + 16 * (v >> 3) + 8 * lh + (v & 7);
            if (key > qrow) sacc[b2][v] = -INFINITY;
          }
      }
      float mt = -INFINITY;
#pragma unroll
      for (int b2 = 0; b2 < SB; ++b2)
#pragma unroll
        for (int v = 0; v < 16; ++v) mt = fmaxf(mt, sacc[b2][v]);
      update_max(mt);
      bf16x8 pf[2 * SB];
#pragma unroll
      for (int b2 = 0; b2 < SB; ++b2)
#pragma unroll
        for (int v = 0; v < 16; ++v)
          pf[2 * b2 + (v >> 3)][v & 7] = (__bf16)__builtin_amdgcn_exp2f(fmaf(sacc[b2][v], c, -mc));
      l_run = sum_weights(pf, l_run);
      pv_step(std::integral_constant<int, 0>{}, pf[0]);
      pv_step(std::integral_constant<int, 1>{}, pf[1]);
      if constexpr (SB == 2) {
        pv_step(std::integral_constant<int, 2>{}, pf[2]);
        pv_step(std::integral_constant<int, 3>{}, pf[3]);
      }
    };
    for (int t = 0; t < n_stages; t += 2) {
      stage(std::integral_constant<int, 0>{}, t);
      stage(std::integral_constant<int, 1>{}, t + 1);
    }

    // ---- normalise and store: lane holds query row qrow, d = 32db + 8(v/4) + 4lh + v%4
    const float l_tot = wave_pair_sum(l_run);
    const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
    if (q0 + qrow < cur.n) {
      uint16_t *op = a.o + ((int64_t)(cur.tok0 + q0 + qrow) * a.hq + cur.h) * D;
#pragma unroll
      for (int db = 0; db < DB; ++db) {
#pragma unroll
        for (int grp = 0; grp < 4; ++grp) {
          bf16x4 ov;
#pragma unroll
          for (int e = 0; e < 4; ++e) ov[e] = (__bf16)(oacc[db][4 * grp + e] * inv);
          *reinterpret_cast<bf16x4 *>(op + db * 32 + 8 * grp + 4 * lh) = ov;
        }
      }
    }
    if (!nxt_valid) break;
    cur = next_row();
    nxt_valid = 0;
  }
}

// number of rows (s, I) with I >= i0, over all sequences
__device__ __forceinline__ int rows_at_or_above(const SeqTable &st, int i0) {
  int c = 0;
  for (int s = 0; s < st.n_seq; ++s) {
    int nb = st.nb_off[s + 1] - st.nb_off[s];
    c += nb > i0 ? nb - i0 : 0;
  }
  return c;
}

// sequence holding global row r (nb_off ascending, n_seq <= 64)
__device__ __forceinline__ int seq_of_row(const SeqTable &st, int r) {
  int lo = 0, hi = st.n_seq;
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (st.nb_off[mid] <= r) lo = mid; else hi = mid;
  }
  return lo;
}

// V^T tiles for the attention stages: for KV head h and global key block gb (B keys of
// one sequence), the B x D slice of V is written as B/16 steps of [d][16 keys], each
// 16-byte unit (8 keys of one d) at vt_unit(d, key half) of its step -- the order the
// attention kernel keeps in LDS.  Keys past the sequence end are zero.  A tile goes
// through 256 threads: load() takes its rows of V into registers, to_lds() stores them in
// a [key][d] LDS tile (`tile`, B * D * 2 bytes; unit index XOR key % (D / 8)), and after a
// barrier store_vt() writes the transposed tile.
template <int D, int B>
struct VtTile {
  static constexpr int UPR = D / 8;              // 16-byte units per key row of the slice
  static constexpr int PER = B * UPR / 256;      // units per thread
  uint4 val[PER];
  __device__ __forceinline__ void load(const SeqTable &st, const uint16_t *v, int hkv, int gb,
                                       int h, int tid) {
    const int s = seq_of_row(st, gb);
    const int tok = st.cu[s] + (gb - st.nb_off[s]) * B;
    const int nvalid = min(B, st.cu[s + 1] - tok);
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int u = tid + 256 * i, key = u / UPR, c = u % UPR;
      val[i] = key < nvalid
                   ? *reinterpret_cast<const uint4 *>(v + ((int64_t)(tok + key) * hkv + h) * D + 8 * c)
                   : make_uint4(0, 0, 0, 0);
    }
  }
  __device__ __forceinline__ void to_lds(uint4 *tile, int tid) const {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int u = tid + 256 * i, key = u / UPR, c = u % UPR;
      tile[key * UPR + (c ^ (key % UPR))] = val[i];
    }
  }
};

template <int D, int B>
__device__ __forceinline__ void store_vt(const uint4 *tile, uint16_t *vt, int nb_total, int gb,
                                         int h, int tid) {
  constexpr int UPR = D / 8;
  const uint16_t *t16 = reinterpret_cast<const uint16_t *>(tile);
  uint4 *out = reinterpret_cast<uint4 *>(vt + ((int64_t)h * nb_total + gb) * B * D);
  for (int p = tid; p < B * UPR; p += 256) {
    const int step = p / (2 * D), w = p % (2 * D);
    const int d = 8 * (w >> 4) + (w & 7);
    const int lh = ((w >> 3) & 1) ^ ((w >> 4) & 1);
    uint32_t word[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int k0 = 16 * step + 8 * lh + 2 * e;
      const uint32_t lo = t16[(k0 * UPR + ((d >> 3) ^ (k0 % UPR))) * 8 + (d & 7)];
      const uint32_t hi = t16[((k0 + 1) * UPR + ((d >> 3) ^ ((k0 + 1) % UPR))) * 8 + (d & 7)];
      word[e] = lo | (hi << 16);
    }
    out[p] = make_uint4(word[0], word[1], word[2], word[3]);
  }
}

// The V^T tiles alone (used with the plain item order).  Grid: (NB, Hkv), 256 threads.
template <int D, int B>
__global__ __launch_bounds__(256) void stage_v_transposed(SeqTable st, const uint16_t *v, int hkv,
                                                          int nb_total, uint16_t *vt) {
  __shared__ uint4 tile[B * D / 8];
  VtTile<D, B> t;
  t.load(st, v, hkv, blockIdx.x, blockIdx.y, threadIdx.x);
  t.to_lds(tile, threadIdx.x);
  __syncthreads();
  store_vt<D, B>(tile, vt, nb_total, blockIdx.x, blockIdx.y, threadIdx.x);
}

// Plain item order, used when a group has too many items for the in-LDS sort: rows by query
// block descending (then sequence ascending), the G heads of a row adjacent.  Same for every
// group.  Also resets the queue counters.
__global__ void build_item_order_plain(SeqTable st, const int32_t *kb_idx, const int32_t *kb_cnt,
                                       int hq, int hkv, int64_t tri_total, int4 *items,
                                       int32_t *queue) {
  const int nb_total = st.nb_off[st.n_seq];
  const int G = hq / hkv;
  const int64_t n_g = (int64_t)G * nb_total;
  if (blockIdx.x == 0 && threadIdx.x < 8) queue[threadIdx.x] = 0;
  for (int pos = blockIdx.x * blockDim.x + threadIdx.x; pos < nb_total;
       pos += gridDim.x * blockDim.x) {
    int lo = 0, hi = st.max_nb;
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (rows_at_or_above(st, mid) > pos) lo = mid; else hi = mid;
    }
    int idx = pos - rows_at_or_above(st, lo + 1);
    int s = 0;
    for (; s < st.n_seq; ++s) {
      const int nb = st.nb_off[s + 1] - st.nb_off[s];
      if (nb > lo) {
        if (idx == 0) break;
        --idx;
      }
    }
    for (int g = 0; g < hkv; ++g)
      for (int kk = 0; kk < G; ++kk)
        items[g * n_g + (int64_t)pos * G + kk] =
            item_record(st, kb_idx, kb_cnt, nb_total, tri_total, G, g, s, kk, lo);
  }
}

constexpr int kSortItems = 16384;   // items per KV group sorted in LDS (128 KB of keys)
constexpr int kSortThreads = 1024;  // threads of a sorting workgroup

// The n keys at src (device memory) sorted ascending into key[] (kSortThreads * E slots of
// LDS, the slots past n padded with keys that sort last): each thread takes E consecutive
// keys into registers, the bitonic network exchanges them inside the thread, across lanes,
// and through key[] for strides that cross waves.
template <int E>
__device__ __forceinline__ void sort_keys(unsigned long long *key, const unsigned long long *src,
                                          int n) {
  const int tid = threadIdx.x;
  unsigned long long k[E];
#pragma unroll
  for (int e = 0; e < E; ++e) k[e] = tid * E + e < n ? src[tid * E + e] : ~0ull;
  bitonic_sort<kSortThreads, E>(k, key, tid);
  __syncthreads();                       // the network's last reads of key[] are done
#pragma unroll
  for (int e = 0; e < E; ++e) key[tid * E + e] = k[e];
  __syncthreads();
}

// Sort key and item record of item id = row * G + kk of KV group g.  The keys give the
// locality order of a group's items (s, head, I): ascending by
//   [1023 - min(blocks / 2, 1023)] [first three listed blocks after block 0] [item id],
// i.e. longest first in buckets of 2 blocks, and inside a bucket items whose lists start
// alike are adjacent, so that the items running at the same time on an XCD read the same
// K/V tiles through its L2 (heads of a row adjacent in id).  The list entries are read
// together, at indices clamped to the row's capacity I + 1.
__device__ __forceinline__ void item_key(const SeqTable &st, const int32_t *kb_idx,
                                         const int32_t *kb_cnt, int G, int64_t tri_total, int g,
                                         int id, unsigned long long &key, int4 &rec) {
  const int nb_total = st.nb_off[st.n_seq];
  const int r = id / G, kk = id % G;
  const int s = seq_of_row(st, r);
  const int I = r - st.nb_off[s];
  const int h = g * G + kk;
  const int32_t *list = kb_idx + (int64_t)h * tri_total + st.tri_off[s] + (int64_t)I * (I + 1) / 2;
  const int c_raw = kb_cnt[(int64_t)h * nb_total + r];
  int32_t l[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) l[t] = list[min(t, I)];
  const int cnt = max(0, min(c_raw, I + 1));
  unsigned long long e[3];
#pragma unroll
  for (int t = 0; t < 3; ++t) e[t] = cnt > t + 1 ? min((unsigned)l[t + 1], 0x1FFFu) : 0x1FFFu;
  const unsigned long long bucket = (unsigned long long)min(cnt >> 1, 1023);
  key = ((1023ull - bucket) << 53) | (e[0] << 40) | (e[1] << 27) | (e[2] << 14) |
        (unsigned long long)id;
  rec = make_int4((int)(((uint32_t)s << 26) | ((uint32_t)kk << 13) | (uint32_t)I), cnt,
                  cnt > 0 ? l[0] : -1, cnt > 1 ? l[1] : -1);
}

// Groups of more than kSortInline items have their keys and records built by item_keys
// (one thread per item, before the sort) instead of by the sorting workgroup itself.
constexpr int kSortInline = 4096;

// Keys and records of every item of groups larger than kSortInline: keys[g][id],
// recs[g][id].  Grid: (G * NB / 256, Hkv), 256 threads.
__global__ __launch_bounds__(256) void item_keys(SeqTable st, const int32_t *kb_idx,
                                                 const int32_t *kb_cnt, int hq, int hkv,
                                                 int64_t tri_total, unsigned long long *keys,
                                                 int4 *recs) {
  const int G = hq / hkv;
  const int n_g = G * st.nb_off[st.n_seq];
  const int g = blockIdx.y;
  const int id = blockIdx.x * blockDim.x + threadIdx.x;
  if (id >= n_g) return;
  unsigned long long key;
  int4 rec;
  item_key(st, kb_idx, kb_cnt, G, tri_total, g, id, key, rec);
  keys[(int64_t)g * n_g + id] = key;
  recs[(int64_t)g * n_g + id] = rec;
}

// One KV group's items in the order of their keys: the keys sorted in LDS, then each
// item's record copied to its place.  Groups of up to kSortInline items build their keys
// here (the records kept in LDS after the key slots), larger ones read those item_keys
// wrote.  Also resets the queue counters.
__device__ __forceinline__ void sort_group_items(const SeqTable &st, const int32_t *kb_idx,
                                                 const int32_t *kb_cnt, int hq, int hkv,
                                                 int64_t tri_total,
                                                 const unsigned long long *keys,
                                                 const int4 *recs, int4 *items, int32_t *queue,
                                                 int g, unsigned long long *key) {
  const int G = hq / hkv;
  const int n_g = G * st.nb_off[st.n_seq];
  if (g == 0 && threadIdx.x < 8) queue[threadIdx.x] = 0;
  // sort slots: a power of two, at least one per thread
  int np = kSortThreads;
  while (np < n_g) np <<= 1;
  const unsigned long long *src = keys + (int64_t)g * n_g;
  const int4 *rsrc = recs + (int64_t)g * n_g;
  if (n_g <= kSortInline) {
    static_assert(kSortInline * (8 + 16) <= kSortItems * 8, "keys and records exceed the LDS");
    int4 *rec = reinterpret_cast<int4 *>(key + np);
    for (int id = threadIdx.x; id < n_g; id += blockDim.x)
      item_key(st, kb_idx, kb_cnt, G, tri_total, g, id, key[id], rec[id]);
    __syncthreads();
    src = key;
    rsrc = rec;
  }
  // bitonic sort, ascending, np / kSortThreads keys per thread held in registers
  switch (np / kSortThreads) {
    case 1: sort_keys<1>(key, src, n_g); break;
    case 2: sort_keys<2>(key, src, n_g); break;
    case 4: sort_keys<4>(key, src, n_g); break;
    case 8: sort_keys<8>(key, src, n_g); break;
    default: sort_keys<16>(key, src, n_g); break;
  }
  for (int t = threadIdx.x; t < n_g; t += blockDim.x)
    items[(int64_t)g * n_g + t] = rsrc[(int)(key[t] & 0x3FFF)];
}


// One launch for both preparations of the attention: workgroups 0 .. Hkv-1 sort their KV
// group's items (as above), the others (about one per CU the sort leaves) write the V^T
// tiles, four at a time per workgroup (one per 256 threads).  1024 threads; 128 KB of LDS
// shared by both.
template <int D, int B>
__global__ __launch_bounds__(1024) void prepare_attn(SeqTable st, const int32_t *kb_idx,
                                                     const int32_t *kb_cnt, int hq, int hkv,
                                                     int64_t tri_total,
                                                     const unsigned long long *keys,
                                                     const int4 *recs, int4 *items,
                                                     int32_t *queue, const uint16_t *v,
                                                     int nb_total, uint16_t *vt) {
  static_assert(4 * B * D * 2 <= kSortItems * 8, "V^T tiles exceed the shared LDS");
  __shared__ __attribute__((aligned(16))) unsigned long long smem[kSortItems];
  if ((int)blockIdx.x < hkv) {
    sort_group_items(st, kb_idx, kb_cnt, hq, hkv, tri_total, keys, recs, items, queue,
                     blockIdx.x, smem);
    return;
  }
  // V^T workgroups: tiles t = gb * Hkv + h, four at a time (one per 256 threads); each
  // workgroup takes every step-th group of four, loading the next group's rows while it
  // writes the current group's transposed tiles
  const int q = threadIdx.x >> 8, tid = threadIdx.x & 255;
  uint4 *tile = reinterpret_cast<uint4 *>(smem) + q * (B * D / 8);
  const int ntiles = nb_total * hkv;
  const int step = ((int)gridDim.x - hkv) * 4;
  const int first = ((int)blockIdx.x - hkv) * 4;
  VtTile<D, B> cur;
  if (first + q < ntiles) cur.load(st, v, hkv, (first + q) / hkv, (first + q) % hkv, tid);
  for (int base = first; base < ntiles; base += step) {
    const int tc = base + q, tn = tc + step;
    if (tc < ntiles) cur.to_lds(tile, tid);
    __syncthreads();
    if (tn < ntiles) cur.load(st, v, hkv, tn / hkv, tn % hkv, tid);
    if (tc < ntiles) store_vt<D, B>(tile, vt, nb_total, tc / hkv, tc % hkv, tid);
    __syncthreads();
  }
}
}  // namespace

hipError_t launch_sparse_attn(const AttnArgs &a, hipStream_t stream) {
  const int G = a.hq / a.hkv;
  const int64_t n_g = (int64_t)G * a.nb_total;
  static int cus = 0;
  if (cus == 0) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        cus <= 0)
      cus = 256;
  }
  // item order and V^T tiles: one fused launch when the groups fit the in-LDS sort
  auto prepare = [&](auto dc, auto bc) {
    constexpr int D = decltype(dc)::value, B = decltype(bc)::value;
    if (n_g <= kSortItems) {
      if (n_g > kSortInline)
        hipLaunchKernelGGL(item_keys, dim3((int)((n_g + 255) / 256), a.hkv), dim3(256), 0,
                           stream, a.st, a.kb_idx, a.kb_cnt, a.hq, a.hkv, a.tri_total,
                           a.sort_keys, a.sort_recs);
      // V^T workgroups: one per CU left by the sorting ones (each holds all of a CU's LDS
      // it may use), no more than there are groups of four tiles
      const int groups = (a.nb_total * a.hkv + 3) / 4;
      const int vt_wgs = std::max(1, std::min(cus - a.hkv, groups));
      hipLaunchKernelGGL((prepare_attn<D, B>), dim3(a.hkv + vt_wgs), dim3(1024), 0,
                         stream, a.st, a.kb_idx, a.kb_cnt, a.hq, a.hkv, a.tri_total,
                         a.sort_keys, a.sort_recs, a.items, a.queue, a.v, a.nb_total, a.vt);
    } else {
      hipLaunchKernelGGL(build_item_order_plain, dim3((a.nb_total + 255) / 256), dim3(256), 0,
                         stream, a.st, a.kb_idx, a.kb_cnt, a.hq, a.hkv, a.tri_total, a.items,
                         a.queue);
      hipLaunchKernelGGL((stage_v_transposed<D, B>), dim3(a.nb_total, a.hkv), dim3(256), 0,
                         stream, a.st, a.v, a.hkv, a.nb_total, a.vt);
    }
  };
  using I128 = std::integral_constant<int, 128>;
  using I64 = std::integral_constant<int, 64>;
  if (a.block == 128) {
    if (a.d == 128) prepare(I128{}, I128{});
    else prepare(I64{}, I128{});
  } else {
    if (a.d == 128) prepare(I128{}, I64{});
    else prepare(I64{}, I64{});
  }
  // Persistent grid: resident workgroups for two waves per SIMD (a multiple of 8, one
  // share per XCD), no more than there are items.
  const int64_t total = n_g * a.hkv;
  auto grid = [&](int wg_per_cu) {
    return (int)std::min<int64_t>((wg_per_cu * cus / 8) * 8, (total + 7) / 8 * 8);
  };
  // groups interleaved on an XCD when there are at most kMixItems items per workgroup
  AttnArgs args = a;
  args.mix = total <= (int64_t)kMixItems * grid(a.block == 128 ? Geo<128>::WG_PER_CU
                                                                : Geo<64>::WG_PER_CU);
  if (a.block == 128) {
    if (a.d == 128)
      hipLaunchKernelGGL((sparse_fa_fwd<128, 128>), dim3(grid(Geo<128>::WG_PER_CU)),
                         dim3(Geo<128>::THREADS), 0, stream, args);
    else
      hipLaunchKernelGGL((sparse_fa_fwd<64, 128>), dim3(grid(Geo<128>::WG_PER_CU)),
                         dim3(Geo<128>::THREADS), 0, stream, args);
  } else {
    if (a.d == 128)
      hipLaunchKernelGGL((sparse_fa_fwd<128, 64>), dim3(grid(Geo<64>::WG_PER_CU)),
                         dim3(Geo<64>::THREADS), 0, stream, args);
    else
      hipLaunchKernelGGL((sparse_fa_fwd<64, 64>), dim3(grid(Geo<64>::WG_PER_CU)),
                         dim3(Geo<64>::THREADS), 0, stream, args);
  }
  return hipGetLastError();
}

}  // namespace fp
