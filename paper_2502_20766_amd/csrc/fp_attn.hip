// Block-sparse causal flash-attention forward for gfx950: O = A(Q, K, V, S).
//
// A(Q, K, V, S) is the sparse attention of Section 2 of the FlexPrefill paper: softmax over
// the keys of S_i only (mask M_S = -inf elsewhere), with S_i inside the causal set j <= i.
// S is given at block granularity: for every (sequence, query head, query block I) an
// ascending list of key blocks J <= I.
//
// One workgroup = one (sequence, query head, query block) row of 128 queries; 4 waves of
// 32 query rows each.  Per selected key block:
//   * K tile [128 keys][d] is staged in LDS row-major with a 16-byte-chunk XOR swizzle;
//   * V tile is staged transposed, Vt[d][128 keys], with an 8-byte-unit XOR swizzle, so
//     that both the K fragment (ds_read_b128) and the V^T fragment (2 x ds_read_b64) are
//     bank-conflict free;
//   * S^T = K Q^T on v_mfma_f32_32x32x16_bf16 (Q^T fragments live in registers), so each
//     lane owns one query row and 64 of the 128 keys: the row max needs one lane swap;
//   * online softmax in the log2 domain (exp2 with log2(e) folded into the scale), the
//     O rescale skipped when no row of the wave sees a new maximum;
//   * O^T += V^T P^T on the same MFMA: P^T is already in B-operand layout (the key order
//     inside each 16-key step is permuted identically on both operands), and O^T keeps
//     one query row per lane, so the rescale by exp2(m_old - m_new) is per lane.
// Each KV group's rows are dispatched longest first (by the blocks listed for the group's
// query heads); the G query heads that share a KV head are adjacent in dispatch order
// and on the same XCD.
#include "fp_internal.h"

namespace fp {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));

constexpr int BM = 128;  // queries per workgroup (one query block)
constexpr int BN = 128;  // keys per tile (one key block)
constexpr int kThreads = 256;

__device__ __forceinline__ float wave_pair_max(float x) {
  // lanes l and l^32 exchange values; max of both halves of the swap is symmetric
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

__device__ __forceinline__ float wave_pair_sum(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Geometry of one 64-key stage in LDS (K and V both row-major [key][d], bf16).
template <int D>
struct Stage {
  static constexpr int RB = 2 * D;                 // bytes per key row
  static constexpr int CPR = RB / 16;              // 16-byte chunks per row
  static constexpr int KEYS = 64;
  static constexpr int BYTES = KEYS * RB;          // one tile (K or V)
  static constexpr int RPI = 1024 / RB;            // rows written by one wave-wide DMA
  static constexpr int DMA_PER_WAVE = BYTES / 1024 / 4;
};

// 16-byte chunk swizzles (XOR, so the same function maps logical <-> physical).
// K: the 32 rows read by one half-wave at the same chunk land on distinct banks.
template <int D>
__device__ __forceinline__ int swz_k(int y, int r) {
  if constexpr (D == 128) return y ^ (r & 15);
  else return y ^ ((r >> 1) & 7);
}
// V: the 4 consecutive rows x 4 chunks read by one half-wave transposing load are distinct.
template <int D>
__device__ __forceinline__ int swz_v(int y, int r) {
  if constexpr (D == 128) return y ^ ((r & 3) << 2);
  else return y ^ (((r >> 1) & 1) << 2);
}

// Per-lane byte offsets of the DMA slots of one stage, relative to the stage's first key
// row: slot i of wave w covers LDS bytes [(4i + w) * 1024, +1024), lane l fills 16 bytes
// of tile row r with the logical chunk whose swizzled position is the lane's slot.
template <int D>
struct DmaOffsets {
  uint32_t k[Stage<D>::DMA_PER_WAVE];
  uint32_t v[Stage<D>::DMA_PER_WAVE];
};

template <int D>
__device__ __forceinline__ DmaOffsets<D> dma_offsets(uint32_t row_bytes, int w, int lane) {
  using S = Stage<D>;
  DmaOffsets<D> o;
#pragma unroll
  for (int i = 0; i < S::DMA_PER_WAVE; ++i) {
    const int r = (i * 4 + w) * S::RPI + lane / S::CPR;
    const int phys = lane % S::CPR;
    o.k[i] = r * row_bytes + swz_k<D>(phys, r) * 16;
    o.v[i] = r * row_bytes + swz_v<D>(phys, r) * 16;
  }
  return o;
}

// Issue the DMA of one 64-key stage: keys k0 .. k0+63 of the sequence through buffer
// descriptors whose range ends at the last valid key row, so rows past the sequence end
// read as zeros (and are masked by the caller).
template <int D>
__device__ __forceinline__ void stage_dma(uint8_t *ks, uint8_t *vs, const uint16_t *kbase,
                                          const uint16_t *vbase, int64_t kv_row, int k0,
                                          int kvalid, const DmaOffsets<D> &off) {
  using S = Stage<D>;
  const int nrec = (kvalid - 1) * (int)kv_row * 2 + 2 * D;
  const __amdgpu_buffer_rsrc_t rk =
      __builtin_amdgcn_make_buffer_rsrc((void *)(kbase + (int64_t)k0 * kv_row), (short)0, nrec,
                                        0x00020000);
  const __amdgpu_buffer_rsrc_t rv =
      __builtin_amdgcn_make_buffer_rsrc((void *)(vbase + (int64_t)k0 * kv_row), (short)0, nrec,
                                        0x00020000);
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
#pragma unroll
  for (int i = 0; i < S::DMA_PER_WAVE; ++i) {
    const int q = i * 4 + w;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(
        rk, (__attribute__((address_space(3))) void *)(ks + q * 1024), 16, off.k[i], 0, 0, 0);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(
        rv, (__attribute__((address_space(3))) void *)(vs + q * 1024), 16, off.v[i], 0, 0, 0);
  }
}

// One 16-key step of V^T fragments: DB d-blocks x 2 key halves of ds_read_b64_tr_b16.
// The loads and their lgkmcnt wait are one asm block, so the outputs are only defined
// once the data has arrived; the compiler's own (conservative) wait for the in-flight
// DMA of the next stage is thereby avoided.
template <int DB, int OFF0, int OFF1>
__device__ __forceinline__ void v_frags(const uint32_t (&addr)[DB], s16x4 (&lo)[DB],
                                        s16x4 (&hi)[DB]) {
  if constexpr (DB == 4) {
    asm volatile(
        "ds_read_b64_tr_b16 %0, %8 offset:%12\n\t"
        "ds_read_b64_tr_b16 %1, %8 offset:%13\n\t"
        "ds_read_b64_tr_b16 %2, %9 offset:%12\n\t"
        "ds_read_b64_tr_b16 %3, %9 offset:%13\n\t"
        "ds_read_b64_tr_b16 %4, %10 offset:%12\n\t"
        "ds_read_b64_tr_b16 %5, %10 offset:%13\n\t"
        "ds_read_b64_tr_b16 %6, %11 offset:%12\n\t"
        "ds_read_b64_tr_b16 %7, %11 offset:%13\n\t"
        "s_waitcnt lgkmcnt(0)"
        : "=&v"(lo[0]), "=&v"(hi[0]), "=&v"(lo[1]), "=&v"(hi[1]), "=&v"(lo[2]), "=&v"(hi[2]),
          "=&v"(lo[3]), "=&v"(hi[3])
        : "v"(addr[0]), "v"(addr[1]), "v"(addr[2]), "v"(addr[3]), "i"(OFF0), "i"(OFF1));
  } else {
    asm volatile(
        "ds_read_b64_tr_b16 %0, %4 offset:%6\n\t"
        "ds_read_b64_tr_b16 %1, %4 offset:%7\n\t"
        "ds_read_b64_tr_b16 %2, %5 offset:%6\n\t"
        "ds_read_b64_tr_b16 %3, %5 offset:%7\n\t"
        "s_waitcnt lgkmcnt(0)"
        : "=&v"(lo[0]), "=&v"(hi[0]), "=&v"(lo[1]), "=&v"(hi[1])
        : "v"(addr[0]), "v"(addr[1]), "i"(OFF0), "i"(OFF1));
  }
}

// One unit of work: the 128 queries of (sequence s, query head h, query block I).
struct Row {
  int valid;
  int I, h, g, cnt, tok0, n;
  int J0, J1;                     // first two listed key blocks (-1 if absent)
  const __attribute__((address_space(4))) int32_t *list;
};

// Work item v of XCD x's queue -> (KV group g, query head h, dispatch position pos).
// Item v of queue x is virtual block vb = 8v + x; the G query heads that share a KV head
// are adjacent items of one queue, and each KV group's positions follow its
// longest-first row order.
struct Item {
  int g, h, pos;
};
__device__ __forceinline__ Item item_of(int vb, int G, int hkv) {
  const int wg = (vb / (8 * G)) * 8 + (vb % 8);
  Item it;
  it.g = wg % hkv;
  it.h = it.g * G + (vb / 8) % G;
  it.pos = wg / hkv;
  return it;
}
// items in queue x: v with (v / G) * 8 + x < W, W = NB * Hkv
__device__ __forceinline__ int queue_len(int x, int G, int W) {
  return W > x ? G * ((W - x + 7) / 8) : 0;
}

__device__ __forceinline__ const __attribute__((address_space(4))) int32_t *
row_list(const AttnArgs &a, int h, int s, int I) {
  return (const __attribute__((address_space(4))) int32_t *)(a.kb_idx + (int64_t)h * a.tri_total +
                                                           a.st.tri_off[s] +
                                                           (int64_t)I * (I + 1) / 2);
}

// First key of stage `half` of key block J in row r, or -1 when the stage has no keys.
__device__ __forceinline__ int stage_first_key(const Row &r, int J, int half) {
  if (J < 0 || J > r.I) return -1;
  const int k0 = J * BN + 64 * half;
  return k0 < r.n ? k0 : -1;
}

// Persistent kernel: gridDim.x workgroups, all resident; workgroup b first takes virtual
// block b (so the first wave of rows is the non-persistent dispatch order), then pulls
// items from its XCD's queue (x = b % 8, the XCD the hardware places it on) and, once that
// is empty, from the other XCDs' queues in turn.  The stages of consecutive rows form one
// stream: the next row's identity and block list are fetched over the current row's
// stages (one dependent step per stage, each step's loads covered by the wait for the
// stage's K/V copy), its first K/V copy is issued at the top of the current row's last
// stage and its Q fragments load during that stage.
template <int D>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
void sparse_fa_fwd(AttnArgs a) {
  using S = Stage<D>;
  constexpr int KS = D / 16;
  constexpr int DB = D / 32;
  __shared__ __attribute__((aligned(1024))) uint8_t lds[4 * S::BYTES];  // [2 stages][K, V]
  __shared__ int fetch_slot[2];           // queue positions handed from thread 0 to all

  const int G = a.hq / a.hkv;
  const int W = a.nb_total * a.hkv;
  const int P = gridDim.x;                // a multiple of 8G
  const int P8 = P / 8;                   // items per queue taken by the first wave of rows
  const int x0 = blockIdx.x & 7;
  const int tid = threadIdx.x;
  const int w = tid >> 6;
  const int lane = tid & 63;
  const int lr = lane & 31;
  const int lh = lane >> 5;
  const int g16 = lane >> 4;
  const int i16 = lane & 15;
  const int qrow = 32 * w + lr;           // this lane's query row within the block
  const float c = a.scale_log2;
  const int64_t kv_row = (int64_t)a.hkv * D;  // elements between consecutive tokens

  // ---- first row: virtual block b, read directly
  Row cur;
  {
    const int vb = blockIdx.x;
    if ((vb / (8 * G)) * 8 + (vb % 8) >= W) return;
    const Item it = item_of(vb, G, a.hkv);
    const int packed = a.row_order[(int64_t)it.g * a.nb_total + it.pos];
    cur.valid = 1;
    cur.g = it.g;
    cur.h = it.h;
    const int s = packed >> 20;
    cur.I = packed & 0xFFFFF;
    cur.tok0 = a.st.cu[s];
    cur.n = a.st.cu[s + 1] - cur.tok0;
    cur.cnt = min(a.kb_cnt[(int64_t)cur.h * a.nb_total + a.st.nb_off[s] + cur.I], cur.I + 1);
    cur.list = row_list(a, cur.h, s, cur.I);
    cur.J0 = cur.cnt > 0 ? cur.list[0] : -1;
    cur.J1 = cur.cnt > 1 ? cur.list[1] : -1;
  }

  // ---- next-row fetch: a small state machine advanced once per stage
  //   fs 0: take a queue position (atomic by thread 0)        -> fs 1
  //   fs 1: position known; empty queue -> next queue (fs 1), else load row_order -> fs 2
  //   fs 2: (s, I) known; load the count and first two list entries      -> fs 3
  //   fs 3: row complete                                                  -> fs 4
  Row nxt;
  nxt.valid = 0;
  int fs = 0, qi = 0, n_fetch = 0;
  int ret_atomic = 0, ret_row = 0, ret_cnt = 0, ret_j0 = 0, ret_j1 = 0;
  auto fetch_issue = [&]() {
    if (tid == 0) ret_atomic = atomicAdd(a.queue + ((x0 + qi) & 7), 1);
  };
  // thread 0 publishes the position it received; runs before a barrier
  auto fetch_publish = [&]() {
    if (fs == 1 && tid == 0) fetch_slot[n_fetch & 1] = ret_atomic;
  };
  // one step; call after a barrier that follows fetch_publish
  auto fetch_step = [&]() {
    if (fs == 0) {
      fetch_issue();
      fs = 1;
    } else if (fs == 1) {
      const int x = (x0 + qi) & 7;
      const int v = P8 + __builtin_amdgcn_readfirstlane(fetch_slot[n_fetch & 1]);
      ++n_fetch;
      if (v >= queue_len(x, G, W)) {
        if (++qi == 8) {
          fs = 4;                       // every queue drained: no next row
        } else {
          fetch_issue();
        }
      } else {
        const Item it = item_of(8 * v + x, G, a.hkv);
        nxt.g = it.g;
        nxt.h = it.h;
        ret_row = *(a.row_order + (int64_t)it.g * a.nb_total + it.pos);
        fs = 2;
      }
    } else if (fs == 2) {
      const int packed = __builtin_amdgcn_readfirstlane(ret_row);
      const int s = packed >> 20;
      nxt.I = packed & 0xFFFFF;
      nxt.tok0 = a.st.cu[s];
      nxt.n = a.st.cu[s + 1] - nxt.tok0;
      nxt.list = row_list(a, nxt.h, s, nxt.I);
      const int32_t *lv = (const int32_t *)nxt.list;
      ret_cnt = a.kb_cnt[(int64_t)nxt.h * a.nb_total + a.st.nb_off[s] + nxt.I];
      ret_j0 = lv[0];
      ret_j1 = lv[nxt.I > 0 ? 1 : 0];   // list of block I has I + 1 slots
      fs = 3;
    } else if (fs == 3) {
      nxt.cnt = min(__builtin_amdgcn_readfirstlane(ret_cnt), nxt.I + 1);
      nxt.J0 = nxt.cnt > 0 ? __builtin_amdgcn_readfirstlane(ret_j0) : -1;
      nxt.J1 = nxt.cnt > 1 ? __builtin_amdgcn_readfirstlane(ret_j1) : -1;
      nxt.valid = 1;
      fs = 4;
    }
  };
  // complete the fetch now (rows with fewer stages than fetch steps)
  auto fetch_finish = [&]() {
    while (fs < 4) {
      if (fs == 1) {
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        fetch_publish();
        __syncthreads();
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

  const DmaOffsets<D> doff = dma_offsets<D>((uint32_t)(kv_row * 2), w, lane);
  // per-lane V^T fragment addresses (relative to a V stage), one per d-block
  uint32_t vaddr_rel[DB];
  {
    const int r_l = 4 * (g16 >> 1) + (i16 >> 2);       // row within a 16-key step
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      const int dcol = 32 * db + 16 * (g16 & 1) + 4 * (i16 & 3);
      vaddr_rel[db] = r_l * S::RB + swz_v<D>(dcol >> 3, r_l) * 16 + (dcol & 7) * 2;
    }
  }
  const uint32_t lds_base = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint8_t *)lds;
  auto issue = [&](const Row &r, int k0, int into) {
    const uint16_t *kb = a.k + (int64_t)r.tok0 * kv_row + (int64_t)r.g * D;
    const uint16_t *vbp = a.v + (int64_t)r.tok0 * kv_row + (int64_t)r.g * D;
    uint8_t *dst = lds + into * 2 * S::BYTES;
    stage_dma<D>(dst, dst + S::BYTES, kb, vbp, kv_row, k0, min(64, r.n - k0), doff);
  };

  int buf = 0;
  int k0_next = stage_first_key(cur, cur.J0, 0);
  if (k0_next >= 0) issue(cur, k0_next, buf);
  bf16x8 qf[KS];
  bool q_ready = false;
  while (true) {
    // ---- row setup: Q^T fragments (lane owns query row q0 + qrow), zero state
    const int q0 = cur.I * BM;
    if (!q_ready) load_q(cur, qf);
    q_ready = false;
    f32x16 oacc[DB];
#pragma unroll
    for (int i = 0; i < DB; ++i) oacc[i] = f32x16{};
    float m_ref = -INFINITY;   // reference max (raw logit units) of this lane's row
    float l_run = 0.f;          // this lane's share of the row sum (its 32 of 64 keys)
    int J_cur = cur.J0;         // block of the stage being prefetched
    int J_pre = cur.J1;         // block after it
    // stage t covers keys J*128 + 64*(t&1) .. +63 of block J = list[t >> 1]; a row with no
    // blocks still takes one (empty) stage so that its zero output is written
    const int n_stages = max(2 * cur.cnt, 1);
    for (int t = 0; t < n_stages; ++t) {
      const int k0 = k0_next;
      const uint8_t *ks = lds + buf * 2 * S::BYTES;
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // this wave's DMA of stage t landed
      fetch_publish();
      __syncthreads();                  // ... and every wave's; stage t-1 reads are done
      fetch_step();
      // the next stage is the row's next one, or the first stage of the next row
      k0_next = -1;
      if (t + 1 < 2 * cur.cnt) {
        if ((t & 1) == 0) {
          k0_next = stage_first_key(cur, J_cur, 1);
        } else {
          J_cur = J_pre;
          J_pre = ((t >> 1) + 2 < cur.cnt) ? cur.list[(t >> 1) + 2] : -1;
          k0_next = stage_first_key(cur, J_cur, 0);
        }
        if (k0_next >= 0) issue(cur, k0_next, buf ^ 1);
      } else {
        fetch_finish();
        if (nxt.valid) {
          k0_next = stage_first_key(nxt, nxt.J0, 0);
          if (k0_next >= 0) issue(nxt, k0_next, buf ^ 1);
        }
      }
      buf ^= 1;
      if (k0 < 0) continue;

    const int kq = k0 - q0;             // key offset relative to the query block start
    const bool diag = kq >= 0;          // diagonal block: keys after the query are masked
    f32x16 sacc[2];
    auto qk_block = [&](int b2) {
      sacc[b2] = f32x16{};
      const int r = b2 * 32 + lr;
      bf16x8 kf[KS];            // all K fragments in flight before the first MFMA
#pragma unroll
      for (int k = 0; k < KS; ++k)
        kf[k] = *reinterpret_cast<const bf16x8 *>(ks + r * S::RB + swz_k<D>(2 * k + lh, r) * 16);
#pragma unroll
      for (int k = 0; k < KS; ++k)
        sacc[b2] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[k], qf[k], sacc[b2], 0, 0, 0);
      // scheduling request: the KS LDS reads first, then the KS MFMAs
      __builtin_amdgcn_sched_group_barrier(0x100, KS, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, KS, 0);
    };
    auto mask_max = [&](int b2) -> float {
      if (diag) {
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int key = kq + b2 * 32 + 8 * (v >> 2) + 4 * lh + (v & 3);
          if (key > qrow) sacc[b2][v] = -INFINITY;
        }
      }
      float mt = -INFINITY;
#pragma unroll
      for (int v = 0; v < 16; ++v) mt = fmaxf(mt, sacc[b2][v]);
      return wave_pair_max(mt);
    };
    // Move the reference max when some row of the wave sees a new maximum (rare after the
    // first blocks), rescaling O and the row sums.  Returns whether it moved.
    auto update_max = [&](float mt) -> bool {
      const float m_new = fmaxf(m_ref, mt);
      if (__ballot(m_new > m_ref)) {
        const float alpha = __builtin_amdgcn_exp2f((m_ref - m_new) * c);
        const float a2 = (m_ref == m_new) ? 1.f : alpha;
        l_run *= a2;
#pragma unroll
        for (int i = 0; i < DB; ++i) oacc[i] *= a2;
        m_ref = m_new;
        return true;
      }
      return false;
    };
    auto weights0 = [&](float (&p0)[16]) {
      const float mc = (m_ref == -INFINITY) ? 0.f : m_ref * c;
#pragma unroll
      for (int v = 0; v < 16; ++v) p0[v] = __builtin_amdgcn_exp2f(fmaf(sacc[0][v], c, -mc));
    };
    // sub-block 0 scores and running max
    qk_block(0);
    update_max(mask_max(0));
    // sub-block 1 scores on MFMA while sub-block 0's weights are computed on VALU
    qk_block(1);
    // last stage of the row: the next row's Q fragments replace this row's (their last use
    // was the MFMAs just issued) and load while this stage finishes
    if (t + 1 == n_stages && nxt.valid) {
      load_q(nxt, qf);
      q_ready = true;
    }
    float p0[16];
    weights0(p0);
    // keep these exponentials here, beside sub-block 1's MFMAs (the compiler would
    // otherwise sink them past the rescale branch below, next to their use)
    asm volatile("" : "+v"(p0[0]), "+v"(p0[1]), "+v"(p0[2]), "+v"(p0[3]), "+v"(p0[4]),
                 "+v"(p0[5]), "+v"(p0[6]), "+v"(p0[7]), "+v"(p0[8]), "+v"(p0[9]),
                 "+v"(p0[10]), "+v"(p0[11]), "+v"(p0[12]), "+v"(p0[13]), "+v"(p0[14]),
                 "+v"(p0[15]));
    // sub-block 1 max; if the reference moved, sub-block 0's weights are recomputed
    if (update_max(mask_max(1))) weights0(p0);
    bf16x8 pf0[2];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      pf0[0][e] = (__bf16)p0[e];
      pf0[1][e] = (__bf16)p0[8 + e];
      l_run += p0[e] + p0[8 + e];
    }

    // ---- O^T += V^T P^T, 16 keys per step; V^T fragments by transposing loads
    uint32_t va[DB];
#pragma unroll
    for (int db = 0; db < DB; ++db)
      va[db] = lds_base + ((buf ^ 1) * 2 + 1) * S::BYTES + vaddr_rel[db];
    auto pv_step = [&](const bf16x8 &pf, s16x4 (&vlo)[DB], s16x4 (&vhi)[DB]) {
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        const s16x8 vv = __builtin_shufflevector(vlo[db], vhi[db], 0, 1, 2, 3, 4, 5, 6, 7);
        oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, vv), pf,
                                                           oacc[db], 0, 0, 0);
      }
    };
    {
      s16x4 vlo[DB], vhi[DB];
      v_frags<DB, 0 * 16 * S::RB, 0 * 16 * S::RB + 8 * S::RB>(va, vlo, vhi);
      pv_step(pf0[0], vlo, vhi);
      v_frags<DB, 1 * 16 * S::RB, 1 * 16 * S::RB + 8 * S::RB>(va, vlo, vhi);
      pv_step(pf0[1], vlo, vhi);
    }
    // sub-block 1 weights (VALU) overlap the PV MFMAs of sub-block 0
    bf16x8 pf1[2];
    {
      const float mc = (m_ref == -INFINITY) ? 0.f : m_ref * c;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const float p = __builtin_amdgcn_exp2f(fmaf(sacc[1][v], c, -mc));
        pf1[v >> 3][v & 7] = (__bf16)p;
        l_run += p;
      }
    }
    {
      s16x4 vlo[DB], vhi[DB];
      v_frags<DB, 2 * 16 * S::RB, 2 * 16 * S::RB + 8 * S::RB>(va, vlo, vhi);
      pv_step(pf1[0], vlo, vhi);
      v_frags<DB, 3 * 16 * S::RB, 3 * 16 * S::RB + 8 * S::RB>(va, vlo, vhi);
      pv_step(pf1[1], vlo, vhi);
    }
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
    if (!nxt.valid) break;
    cur = nxt;
    nxt.valid = 0;
    fs = 0;
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

// Fallback dispatch order (query block descending, then sequence ascending), used when a
// group has too many rows for the in-LDS sort; entry = (s << 20) | I, same for every group.
__global__ void build_row_order(SeqTable st, int hkv, int32_t *row_order, int32_t *queue) {
  const int nb_total = st.nb_off[st.n_seq];
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
    for (int g = 0; g < hkv; ++g) row_order[(int64_t)g * nb_total + pos] = (s << 20) | lo;
  }
}

constexpr int kSortMax = 8192;   // rows per KV group sorted in LDS

// Longest-processing-time-first order of one KV group's rows: cost = blocks listed for
// the row summed over the group's query heads; ties by query block descending.
__global__ __launch_bounds__(1024) void build_row_order_lpt(SeqTable st, const int32_t *kb_cnt,
                                                            int hq, int hkv,
                                                            int32_t *row_order,
                                                            int32_t *queue) {
  __shared__ unsigned long long key[kSortMax];
  const int g = blockIdx.x;
  const int G = hq / hkv;
  const int nb_total = st.nb_off[st.n_seq];
  if (g == 0 && threadIdx.x < 8) queue[threadIdx.x] = 0;
  int np = 1;
  while (np < nb_total) np <<= 1;
  for (int r = threadIdx.x; r < np; r += blockDim.x) {
    unsigned long long kv = 0ull;               // padding sorts last
    if (r < nb_total) {
      int s = 0;
      while (s + 1 < st.n_seq && st.nb_off[s + 1] <= r) ++s;
      const int I = r - st.nb_off[s];
      unsigned cost = 0;
      for (int k = 0; k < G; ++k) cost += (unsigned)kb_cnt[(int64_t)(g * G + k) * nb_total + r];
      kv = ((unsigned long long)(cost + 1) << 40) | ((unsigned long long)I << 20) |
           (unsigned long long)(0xFFFFF - s);
    }
    key[r] = kv;
  }
  __syncthreads();
  // bitonic sort, descending
  for (int size = 2; size <= np; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int i = threadIdx.x; i < np; i += blockDim.x) {
        const int j = i ^ stride;
        if (j > i) {
          const bool desc = (i & size) == 0;
          const unsigned long long a = key[i], b = key[j];
          if (desc ? (a < b) : (a > b)) {
            key[i] = b;
            key[j] = a;
          }
        }
      }
      __syncthreads();
    }
  }
  for (int r = threadIdx.x; r < nb_total; r += blockDim.x) {
    const unsigned long long kv = key[r];
    const int I = (int)((kv >> 20) & 0xFFFFF);
    const int s = 0xFFFFF - (int)(kv & 0xFFFFF);
    row_order[(int64_t)g * nb_total + r] = (s << 20) | I;
  }
}

}  // namespace

hipError_t launch_sparse_attn(const AttnArgs &a, hipStream_t stream) {
  if (a.nb_total <= kSortMax)
    hipLaunchKernelGGL(build_row_order_lpt, dim3(a.hkv), dim3(1024), 0, stream, a.st, a.kb_cnt,
                       a.hq, a.hkv, a.row_order, a.queue);
  else
    hipLaunchKernelGGL(build_row_order, dim3((a.nb_total + 255) / 256), dim3(256), 0, stream,
                       a.st, a.hkv, a.row_order, a.queue);
  // Persistent grid: about two resident workgroups per CU, a multiple of 8G so that every
  // block stays on one XCD's share of KV groups and the G heads of a row run together.
  static int cus = 0;
  if (cus == 0) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        cus <= 0)
      cus = 256;
  }
  const int G = a.hq / a.hkv;
  const int unit = 8 * G;
  const int total = ((a.nb_total * a.hkv + 7) / 8) * unit;
  int blocks = max(unit, (2 * cus / unit) * unit);
  blocks = min(blocks, total);
  if (a.d == 128)
    hipLaunchKernelGGL(sparse_fa_fwd<128>, dim3(blocks), dim3(kThreads), 0, stream, a);
  else
    hipLaunchKernelGGL(sparse_fa_fwd<64>, dim3(blocks), dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace fp
