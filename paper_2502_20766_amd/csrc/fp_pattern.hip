// Sparse pattern search (Algorithm 2) and the query-aware block estimate (Algorithm 4,
// first steps) for gfx950.
//
// pattern_parts + pattern_decide: per (sequence, query head)
//   a_bar = softmax(scale * avgpool(Q_hat) . avgpool(K)^T)       over all key blocks
//   a_hat = block sums of the vertical line scores a_v            (= sumpool of A_hat / b')
//   D_JS  = sqrt((KL(a_bar || m) + KL(a_hat || m)) / 2), m = (a_bar + a_hat) / 2, natural log
//   pattern = query-aware iff D_JS < tau (or the forced pattern).
// The divergence is accumulated in double with a fixed reduction tree.
//
// qa_logits / qa_softmax: for query-aware heads only,
//   A_bar[I, J] = softmax over J <= I of scale * Q_bar_I . K_bar_J
// stored as the flattened causal entries (row-major, I(I+1)/2 + J), in fp32 with the
// pooled vectors kept in fp32 (pooled means rounded to bf16 would move the selection).
#include "fp_internal.h"

namespace fp {
namespace {

constexpr int kThreads = 256;

__device__ __forceinline__ int seq_of_block(const SeqTable &st, int blk) {
  int s = 0;
  while (s + 1 < st.n_seq && st.nb_off[s + 1] <= blk) ++s;
  return s;
}

template <typename T>
__device__ __forceinline__ T block_sum(T v, T *scratch) {
  const int tid = threadIdx.x;
  scratch[tid] = v;
  __syncthreads();
  for (int off = kThreads / 2; off > 0; off >>= 1) {
    if (tid < off) scratch[tid] = scratch[tid] + scratch[tid + off];
    __syncthreads();
  }
  const T r = scratch[0];
  __syncthreads();
  return r;
}

__device__ __forceinline__ float block_max(float v, float *scratch) {
  const int tid = threadIdx.x;
  scratch[tid] = v;
  __syncthreads();
  for (int off = kThreads / 2; off > 0; off >>= 1) {
    if (tid < off) scratch[tid] = fmaxf(scratch[tid], scratch[tid + off]);
    __syncthreads();
  }
  const float r = scratch[0];
  __syncthreads();
  return r;
}

// ---------------------------------------------------------------- Algorithm 2

// Key blocks of one (sequence, head) are split over kPatSlices workgroups for the logits
// and the block sums, which dominate the work; one workgroup per (sequence, head) then
// reduces them.
constexpr int kPatSlices = 16;

// pattern_parts: grid (n_seq * kPatSlices, Hq).  Each workgroup pools Q_hat into q_bar,
// then for its key blocks J writes the logit scale * q_bar . K_bar_J (fp32) and
// a_hat[J] = sum of a_v over the block's tokens (double, token order).
template <int D>
__global__ __launch_bounds__(kThreads) void pattern_parts(SelectArgs a) {
  constexpr int CH = D / 8;                 // 16-byte chunks of a query row
  constexpr int PH = kThreads / CH;         // row phases of the Q_hat pooling
  __shared__ __attribute__((aligned(16))) float qbar[D];
  __shared__ float qpart[PH][D];
  const int s = blockIdx.x / kPatSlices, slice = blockIdx.x % kPatSlices;
  const int h = blockIdx.y, tid = threadIdx.x;
  const int tok0 = a.st.cu[s];
  const int n = a.st.cu[s + 1] - tok0;
  const int bp = min(a.block, n);
  const int nb = a.st.nb_off[s + 1] - a.st.nb_off[s];
  const int per = (nb + kPatSlices - 1) / kPatSlices;
  const int J0 = slice * per, J1 = min(nb, J0 + per);
  if (J0 >= J1) return;
  const int G = a.hq / a.hkv;
  const int g = h / G;

  // avgpool(Q_hat): thread (phase ph, chunk ch) sums rows ph, ph + PH, ... of its 8
  // dimensions; the phases are then added in order
  {
    const int ch = tid % CH, ph = tid / CH;
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    const uint16_t *qp = a.q + ((int64_t)(tok0 + n - bp) * a.hq + h) * D + ch * 8;
#pragma unroll 4
    for (int r = ph; r < bp; r += PH) {
      const uint4 v = *reinterpret_cast<const uint4 *>(qp + (int64_t)r * a.hq * D);
      const uint32_t wv[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        acc[2 * i] += __uint_as_float(wv[i] << 16);
        acc[2 * i + 1] += __uint_as_float(wv[i] & 0xFFFF0000u);
      }
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) qpart[ph][ch * 8 + i] = acc[i];
  }
  __syncthreads();
  if (tid < D) {
    float acc = 0.f;
    for (int ph = 0; ph < PH; ++ph) acc += qpart[ph][tid];
    qbar[tid] = acc / (float)bp;
  }
  __syncthreads();
  const float *av = a.a_v + (int64_t)h * a.total_tokens + tok0;
  for (int J = J0 + tid; J < J1; J += kThreads) {
    // logit: the pooled key read as 16-byte vectors
    const float4 *kb =
        reinterpret_cast<const float4 *>(a.kbar + ((int64_t)(a.st.nb_off[s] + J) * a.hkv + g) * D);
    float4 kv[D / 4];
#pragma unroll
    for (int i = 0; i < D / 4; ++i) kv[i] = kb[i];
    const float4 *q4 = reinterpret_cast<const float4 *>(qbar);
    float dot = 0.f;
#pragma unroll
    for (int i = 0; i < D / 4; ++i) {
      const float4 qv = q4[i];
      dot = fmaf(qv.x, kv[i].x, dot);
      dot = fmaf(qv.y, kv[i].y, dot);
      dot = fmaf(qv.z, kv[i].z, dot);
      dot = fmaf(qv.w, kv[i].w, dot);
    }
    a.pat_logit[(int64_t)h * a.nb_total + a.st.nb_off[s] + J] = dot * a.scale;
    // a_hat[J]: the block's line scores in token order
    double ph = 0.0;
    const int j0 = J * a.block, j1 = min(j0 + a.block, n);
    const float *ap = av + j0;
    int j = 0;
    if ((reinterpret_cast<uintptr_t>(ap) & 15) == 0) {
      // 16-byte loads, eight in flight; the sum stays in token order
      for (; j + 32 <= j1 - j0; j += 32) {
        float4 v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = reinterpret_cast<const float4 *>(ap + j)[u];
#pragma unroll
        for (int u = 0; u < 8; ++u)
          ph = (((ph + (double)v[u].x) + (double)v[u].y) + (double)v[u].z) + (double)v[u].w;
      }
    }
    for (; j < j1 - j0; ++j) ph += (double)ap[j];
    a.pat_ahat[(int64_t)h * a.nb_total + a.st.nb_off[s] + J] = ph;
  }
}

// pattern_decide: grid (n_seq, Hq).  a_bar = softmax of the logits, D_JS against a_hat
// (double, fixed reduction trees), pattern.
__global__ __launch_bounds__(kThreads) void pattern_decide(SelectArgs a) {
  extern __shared__ float dyn[];            // [max_nb] logits
  __shared__ float fscr[kThreads];
  __shared__ double dscr[kThreads];
  const int s = blockIdx.x, h = blockIdx.y, tid = threadIdx.x;
  const int nb = a.st.nb_off[s + 1] - a.st.nb_off[s];
  const float *lg = a.pat_logit + (int64_t)h * a.nb_total + a.st.nb_off[s];
  const double *ah = a.pat_ahat + (int64_t)h * a.nb_total + a.st.nb_off[s];
  float mx = -INFINITY;
  for (int J = tid; J < nb; J += kThreads) {
    const float x = lg[J];
    dyn[J] = x;
    mx = fmaxf(mx, x);
  }
  mx = block_max(mx, fscr);
  double se = 0.0;
  for (int J = tid; J < nb; J += kThreads) se += (double)expf(dyn[J] - mx);
  se = block_sum(se, dscr);
  // JSD terms, double precision
  double jsd = 0.0;
  for (int J = tid; J < nb; J += kThreads) {
    const double pb = (double)expf(dyn[J] - mx) / se;              // a_bar[J]
    const double ph = ah[J];                                        // a_hat[J]
    const double m = 0.5 * (pb + ph);
    if (pb > 0.0) jsd += 0.5 * pb * log(pb / m);
    if (ph > 0.0) jsd += 0.5 * ph * log(ph / m);
  }
  jsd = block_sum(jsd, dscr);
  if (tid == 0) {
    const float djs = (float)sqrt(jsd > 0.0 ? jsd : 0.0);
    int pat = (djs < a.tau) ? FP_PATTERN_QUERY_AWARE : FP_PATTERN_VERTICAL_SLASH;
    if (a.force_pattern == 0 || a.force_pattern == 1) pat = a.force_pattern;
    a.js[s * a.hq + h] = djs;
    a.pattern[s * a.hq + h] = (uint8_t)pat;
  }
}

// ---------------------------------------------------------------- Algorithm 4 estimate

constexpr int QT = 128;  // rows and columns of A_bar per workgroup tile
constexpr int kLogitThreads = 1024;   // 16 waves, one 32x32 block each

// Tile (TI, TJ), TJ <= TI, of the logits scale * Q_bar_I . K_bar_J written into the
// flattened causal layout.  Grid x enumerates the causal tile pairs of all sequences.
// The tile's 128 Q_bar rows and 128 K_bar rows are staged in LDS with coalesced 16-byte
// loads; each wave then computes one 32x32 block with the fp32 MFMA (products and sums
// in fp32, as the vector code would): lane (l % 32, l / 32) supplies Q_bar row l % 32 and
// K_bar row l % 32 over dimensions [l / 32 * D / 2, +D / 2), so the reduction runs over the
// same dimensions for both operands.
template <int D>
__global__ __launch_bounds__(kLogitThreads) void qa_logits(SelectArgs a) {
  typedef float f32x16 __attribute__((ext_vector_type(16)));
  constexpr int P = D + 4;               // LDS row pitch in floats (16-byte rows, no conflicts)
  __shared__ __attribute__((aligned(16))) float Qs[QT * P];
  __shared__ __attribute__((aligned(16))) float Ks[QT * P];
  const int h = blockIdx.y;
  // locate sequence and tile pair
  int t = blockIdx.x, s = 0, nt = 0;
  for (; s < a.st.n_seq; ++s) {
    const int nb = a.st.nb_off[s + 1] - a.st.nb_off[s];
    nt = (nb + QT - 1) / QT;
    const int pairs = nt * (nt + 1) / 2;
    if (t < pairs) break;
    t -= pairs;
  }
  if (s >= a.st.n_seq) return;
  if (a.pattern[s * a.hq + h] != FP_PATTERN_QUERY_AWARE) return;
  int TI = (int)((sqrtf(8.f * (float)t + 1.f) - 1.f) * 0.5f);
  while ((TI + 1) * (TI + 2) / 2 <= t) ++TI;
  while (TI * (TI + 1) / 2 > t) --TI;
  const int TJ = t - TI * (TI + 1) / 2;
  const int nb = a.st.nb_off[s + 1] - a.st.nb_off[s];
  const int G = a.hq / a.hkv;
  const int g = h / G;
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, lr = lane & 31, lh = lane >> 5;
  // stage the rows (rows past the sequence's last block are clamped; their logits are not
  // written)
  // (every load is issued before the first store, so the loads overlap)
  constexpr int NST = QT * (D / 4) / kLogitThreads;
  static_assert(NST * kLogitThreads == QT * (D / 4), "staging covers the tile exactly");
  float4 qv4[NST], kv4[NST];
#pragma unroll
  for (int u = 0; u < NST; ++u) {
    const int i = tid + u * kLogitThreads;
    const int row = i / (D / 4), c = i % (D / 4);
    const int I = min(TI * QT + row, nb - 1), J = min(TJ * QT + row, nb - 1);
    qv4[u] = reinterpret_cast<const float4 *>(
        a.qbar + ((int64_t)(a.st.nb_off[s] + I) * a.hq + h) * D)[c];
    kv4[u] = reinterpret_cast<const float4 *>(
        a.kbar + ((int64_t)(a.st.nb_off[s] + J) * a.hkv + g) * D)[c];
  }
#pragma unroll
  for (int u = 0; u < NST; ++u) {
    const int i = tid + u * kLogitThreads;
    const int row = i / (D / 4), c = i % (D / 4);
    *reinterpret_cast<float4 *>(Qs + row * P + 4 * c) = qv4[u];
    *reinterpret_cast<float4 *>(Ks + row * P + 4 * c) = kv4[u];
  }
  __syncthreads();
  const int i0 = 32 * (w >> 2), j0 = 32 * (w & 3);          // block within the tile
  const int I0 = TI * QT + i0, J0 = TJ * QT + j0;
  if (J0 > I0 + 31 || I0 >= nb) return;      // block above the diagonal or past the end
  const float *qa = Qs + (i0 + lr) * P + lh * (D / 2);
  const float *kb = Ks + (j0 + lr) * P + lh * (D / 2);
  f32x16 acc = {};
#pragma unroll
  for (int c = 0; c < D / 2; c += 4) {
    const float4 qv = *reinterpret_cast<const float4 *>(qa + c);
    const float4 kv = *reinterpret_cast<const float4 *>(kb + c);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(qv.x, kv.x, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(qv.y, kv.y, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(qv.z, kv.z, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(qv.w, kv.w, acc, 0, 0, 0);
  }
  // lane holds column J0 + lr of rows I0 + 8 (v / 4) + 4 lh + v % 4
  float *flat = a.flat + (int64_t)h * a.tri_total + a.st.tri_off[s];
  const int J = J0 + lr;
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const int I = I0 + 8 * (v >> 2) + 4 * lh + (v & 3);
    if (I < nb && J <= I) flat[(int64_t)I * (I + 1) / 2 + J] = acc[v] * a.scale;
  }
}

// Row softmax over J <= I of the flattened logits, one wave per row (in place).
constexpr int kRowRegs = 16;   // rows up to 1024 blocks are held in registers
__global__ __launch_bounds__(kThreads) void qa_softmax(SelectArgs a) {
  const int h = blockIdx.y;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= a.nb_total) return;
  const int s = seq_of_block(a.st, row);
  if (a.pattern[s * a.hq + h] != FP_PATTERN_QUERY_AWARE) return;
  const int I = row - a.st.nb_off[s];
  float *x = a.flat + (int64_t)h * a.tri_total + a.st.tri_off[s] + (int64_t)I * (I + 1) / 2;
  if (I < 64 * kRowRegs) {
    // the row fits in registers: one read, one write (same operations in the same order as
    // the streaming form below)
    float xv[kRowRegs];
    float mx = -INFINITY;
#pragma unroll
    for (int u = 0; u < kRowRegs; ++u) {
      const int J = lane + 64 * u;
      xv[u] = J <= I ? x[J] : -INFINITY;
      mx = fmaxf(mx, xv[u]);
    }
    for (int off = 32; off > 0; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
    float se = 0.f;
#pragma unroll
    for (int u = 0; u < kRowRegs; ++u)
      if (lane + 64 * u <= I) {
        xv[u] = expf(xv[u] - mx);
        se += xv[u];
      }
    for (int off = 32; off > 0; off >>= 1) se += __shfl_xor(se, off);
    const float inv = 1.f / se;
#pragma unroll
    for (int u = 0; u < kRowRegs; ++u)
      if (lane + 64 * u <= I) x[lane + 64 * u] = xv[u] * inv;
    return;
  }
  float mx = -INFINITY;
  for (int J = lane; J <= I; J += 64) mx = fmaxf(mx, x[J]);
  for (int off = 32; off > 0; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
  float se = 0.f;
  for (int J = lane; J <= I; J += 64) se += expf(x[J] - mx);
  for (int off = 32; off > 0; off >>= 1) se += __shfl_xor(se, off);
  const float inv = 1.f / se;
  for (int J = lane; J <= I; J += 64) x[J] = expf(x[J] - mx) * inv;
}

}  // namespace

hipError_t launch_pattern_search(const SelectArgs &a, hipStream_t stream) {
  const dim3 parts(a.st.n_seq * kPatSlices, a.hq);
  if (a.d == 128)
    hipLaunchKernelGGL(pattern_parts<128>, parts, dim3(kThreads), 0, stream, a);
  else
    hipLaunchKernelGGL(pattern_parts<64>, parts, dim3(kThreads), 0, stream, a);
  const size_t dyn = (size_t)a.st.max_nb * sizeof(float);
  hipLaunchKernelGGL(pattern_decide, dim3(a.st.n_seq, a.hq), dim3(kThreads), dyn, stream, a);
  return hipGetLastError();
}

hipError_t launch_qa_estimate(const SelectArgs &a, hipStream_t stream) {
  int pairs = 0;
  for (int s = 0; s < a.st.n_seq; ++s) {
    const int nb = a.st.nb_off[s + 1] - a.st.nb_off[s];
    const int nt = (nb + QT - 1) / QT;
    pairs += nt * (nt + 1) / 2;
  }
  if (a.d == 128)
    hipLaunchKernelGGL(qa_logits<128>, dim3(pairs, a.hq), dim3(kLogitThreads), 0, stream, a);
  else
    hipLaunchKernelGGL(qa_logits<64>, dim3(pairs, a.hq), dim3(kLogitThreads), 0, stream, a);
  hipLaunchKernelGGL(qa_softmax, dim3((a.nb_total + 3) / 4, a.hq), dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace fp
