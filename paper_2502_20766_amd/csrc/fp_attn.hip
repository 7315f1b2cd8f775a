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
//   * online softmax in the log2 domain (exp2 with log2(e) folded into the scale);
//   * O^T += V^T P^T on the same MFMA: P^T is already in B-operand layout (the key order
//     inside each 16-key step is permuted identically on both operands), and O^T keeps
//     one query row per lane, so the rescale by exp2(m_old - m_new) is per lane.
// Workgroups are ordered by query block descending (longest rows first), the G query
// heads that share a KV head are adjacent in dispatch order and on the same XCD.
#include "fp_internal.h"

namespace fp {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

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

// 16-byte chunk swizzle of the K tile row `key` (D/8 chunks per row)
template <int D>
__device__ __forceinline__ int k_swz(int chunk, int key) {
  if constexpr (D == 128) return chunk ^ (key & 15);
  else return chunk ^ ((key >> 1) & 7);
}

// 8-byte unit swizzle of the transposed V tile row `d` (32 units of 4 keys per row)
__device__ __forceinline__ int v_swz(int unit, int d) { return unit ^ (((d >> 2) ^ d) & 31); }

template <int D>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
void sparse_fa_fwd(AttnArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t Ks[BN * D];
  __shared__ __attribute__((aligned(16))) uint16_t Vt[D * BN];

  const int G = a.hq / a.hkv;
  const int bid = blockIdx.x;
  const int wg = (bid / (8 * G)) * 8 + (bid % 8);
  const int kk = (bid / 8) % G;
  const int groups = a.nb_total * a.hkv;
  if (wg >= groups) return;
  const int pos = wg / a.hkv;
  const int g = wg % a.hkv;
  const int h = g * G + kk;

  // row position `pos` in query-block-descending order -> (s, I), tabulated per call
  const int packed = a.row_order[pos];
  const int s = packed >> 20;
  const int I = packed & 0xFFFFF;
  const int tok0 = a.st.cu[s];
  const int n = a.st.cu[s + 1] - tok0;
  const int q0 = I * BM;

  const int tid = threadIdx.x;
  const int w = tid >> 6;
  const int lane = tid & 63;
  const int lr = lane & 31;
  const int lh = lane >> 5;

  const int cnt = min(a.kb_cnt[(int64_t)h * a.nb_total + a.st.nb_off[s] + I], I + 1);
  const int32_t *list = a.kb_idx + (int64_t)h * a.tri_total + a.st.tri_off[s] +
                        (int64_t)I * (I + 1) / 2;

  // Q^T fragments: lane owns query row q0 + 32w + lr, d = 16k + 8lh .. +8
  constexpr int KS = D / 16;
  bf16x8 qf[KS];
  const int qrow = 32 * w + lr;
  if (q0 + qrow < n) {
    const uint16_t *qp = a.q + ((int64_t)(tok0 + q0 + qrow) * a.hq + h) * D + 8 * lh;
#pragma unroll
    for (int k = 0; k < KS; ++k) qf[k] = *reinterpret_cast<const bf16x8 *>(qp + 16 * k);
  } else {
#pragma unroll
    for (int k = 0; k < KS; ++k) qf[k] = bf16x8{};
  }

  constexpr int DB = D / 32;
  f32x16 oacc[DB];
#pragma unroll
  for (int i = 0; i < DB; ++i) oacc[i] = f32x16{};
  float m_run = -INFINITY;
  float l_run = 0.f;

  const int64_t kv_row = (int64_t)a.hkv * D;  // elements between consecutive tokens
  const uint16_t *kbase = a.k + (int64_t)tok0 * kv_row + (int64_t)g * D;
  const uint16_t *vbase = a.v + (int64_t)tok0 * kv_row + (int64_t)g * D;

  for (int t = 0; t < cnt; ++t) {
    const int J = list[t];
    if (J < 0 || J > I) continue;
    const int k0 = J * BN;
    const int kvalid = min(BN, n - k0);

    __syncthreads();
    // ---- K tile -> LDS (row-major, swizzled 16-byte chunks)
    constexpr int KCH = D / 8;
#pragma unroll
    for (int it = 0; it < BN * KCH / kThreads; ++it) {
      const int c = it * kThreads + tid;
      const int key = c / KCH;
      const int ch = c % KCH;
      // rows past the sequence end read the last valid row and are zeroed (no branch)
      uint4 val = *reinterpret_cast<const uint4 *>(
          kbase + (int64_t)(k0 + min(key, kvalid - 1)) * kv_row + ch * 8);
      if (key >= kvalid) val = make_uint4(0, 0, 0, 0);
      *reinterpret_cast<uint4 *>(Ks + key * D + k_swz<D>(ch, key) * 8) = val;
    }
    // ---- V tile -> LDS transposed: each thread moves a 4-key x 4-d block
    constexpr int DQ = D / 4;
#pragma unroll
    for (int it = 0; it < BN * DQ / 4 / kThreads; ++it) {
      const int u = it * kThreads + tid;
      const int dq = u % DQ;
      const int kq = u / DQ;
      uint2 r[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int key = 4 * kq + e;
        r[e] = *reinterpret_cast<const uint2 *>(
            vbase + (int64_t)(k0 + min(key, kvalid - 1)) * kv_row + 4 * dq);
        if (key >= kvalid) r[e] = make_uint2(0, 0);
      }
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const uint32_t sh = (c & 1) ? 16u : 0u;
        const uint32_t w0 = ((c < 2 ? r[0].x : r[0].y) >> sh) & 0xFFFFu;
        const uint32_t w1 = ((c < 2 ? r[1].x : r[1].y) >> sh) & 0xFFFFu;
        const uint32_t w2 = ((c < 2 ? r[2].x : r[2].y) >> sh) & 0xFFFFu;
        const uint32_t w3 = ((c < 2 ? r[3].x : r[3].y) >> sh) & 0xFFFFu;
        const int d = 4 * dq + c;
        *reinterpret_cast<uint2 *>(Vt + d * BN + v_swz(kq, d) * 4) =
            make_uint2(w0 | (w1 << 16), w2 | (w3 << 16));
      }
    }
    __syncthreads();

    // ---- two halves of 64 keys: S^T = K Q^T, online softmax, O^T += V^T P^T
    const bool diag = (J == I);
#pragma unroll
    for (int hf = 0; hf < 2; ++hf) {
      f32x16 sacc[2];
#pragma unroll
      for (int b2 = 0; b2 < 2; ++b2) {
        sacc[b2] = f32x16{};
        const int key = (2 * hf + b2) * 32 + lr;
#pragma unroll
        for (int k = 0; k < KS; ++k) {
          const bf16x8 kf =
              *reinterpret_cast<const bf16x8 *>(Ks + key * D + k_swz<D>(2 * k + lh, key) * 8);
          sacc[b2] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[k], sacc[b2], 0, 0, 0);
        }
      }
      float mt = -INFINITY;
#pragma unroll
      for (int b2 = 0; b2 < 2; ++b2) {
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          float x = sacc[b2][v] * a.scale_log2;
          if (diag) {
            const int key = (2 * hf + b2) * 32 + 8 * (v >> 2) + 4 * lh + (v & 3);
            if (key > qrow) x = -INFINITY;
          }
          sacc[b2][v] = x;
          mt = fmaxf(mt, x);
        }
      }
      mt = wave_pair_max(mt);
      const float m_new = fmaxf(m_run, mt);
      const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_use);
      m_run = m_new;
      float lsum = 0.f;
#pragma unroll
      for (int b2 = 0; b2 < 2; ++b2) {
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const float p = __builtin_amdgcn_exp2f(sacc[b2][v] - m_use);
          sacc[b2][v] = p;
          lsum += p;
        }
      }
      l_run = l_run * alpha + lsum;
#pragma unroll
      for (int i = 0; i < DB; ++i) oacc[i] *= alpha;

#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const int b2 = ks >> 1;
        const int half = ks & 1;
        bf16x8 pf;
#pragma unroll
        for (int e = 0; e < 8; ++e) pf[e] = (__bf16)sacc[b2][8 * half + e];
        const int unit0 = ((2 * hf + b2) * 32 + 16 * half) / 4 + lh;
#pragma unroll
        for (int db = 0; db < DB; ++db) {
          const int d = db * 32 + lr;
          const bf16x4 v0 =
              *reinterpret_cast<const bf16x4 *>(Vt + d * BN + v_swz(unit0, d) * 4);
          const bf16x4 v1 =
              *reinterpret_cast<const bf16x4 *>(Vt + d * BN + v_swz(unit0 + 2, d) * 4);
          const bf16x8 vf = __builtin_shufflevector(v0, v1, 0, 1, 2, 3, 4, 5, 6, 7);
          oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf, oacc[db], 0, 0, 0);
        }
      }
    }
  }

  // ---- normalise and store: lane holds query row qrow, d = 32db + 8(v/4) + 4lh + v%4
  const float l_tot = wave_pair_sum(l_run);
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  if (q0 + qrow < n) {
    uint16_t *op = a.o + ((int64_t)(tok0 + q0 + qrow) * a.hq + h) * D;
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

// Tabulate the dispatch order of query-block rows: query block descending, then
// sequence ascending; entry = (s << 20) | I.
__global__ void build_row_order(SeqTable st, int32_t *row_order) {
  const int nb_total = st.nb_off[st.n_seq];
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
    row_order[pos] = (s << 20) | lo;
  }
}

}  // namespace

hipError_t launch_sparse_attn(const AttnArgs &a, hipStream_t stream) {
  hipLaunchKernelGGL(build_row_order, dim3((a.nb_total + 255) / 256), dim3(256), 0, stream, a.st,
                     a.row_order);
  const int G = a.hq / a.hkv;
  const int groups = a.nb_total * a.hkv;
  const int blocks = ((groups + 7) / 8) * 8 * G;
  if (a.d == 128)
    hipLaunchKernelGGL(sparse_fa_fwd<128>, dim3(blocks), dim3(kThreads), 0, stream, a);
  else
    hipLaunchKernelGGL(sparse_fa_fwd<64>, dim3(blocks), dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace fp
