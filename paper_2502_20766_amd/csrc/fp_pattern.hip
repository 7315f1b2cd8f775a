// Sparse pattern search (Algorithm 2) and the query-aware block estimate (Algorithm 4,
// first steps) for gfx950.
//
// pattern_search: per (sequence, query head)
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

template <int D>
__global__ __launch_bounds__(kThreads) void pattern_search(SelectArgs a) {
  extern __shared__ float dyn[];            // [max_nb] logits
  __shared__ float qbar[D];
  __shared__ float fscr[kThreads];
  __shared__ double dscr[kThreads];
  const int s = blockIdx.x, h = blockIdx.y, tid = threadIdx.x;
  const int tok0 = a.st.cu[s];
  const int n = a.st.cu[s + 1] - tok0;
  const int bp = min(a.block, n);
  const int nb = a.st.nb_off[s + 1] - a.st.nb_off[s];
  const int G = a.hq / a.hkv;
  const int g = h / G;

  // avgpool(Q_hat): mean of the last b' query rows
  if (tid < D) {
    float acc = 0.f;
    const uint16_t *qp = a.q + ((int64_t)(tok0 + n - bp) * a.hq + h) * D + tid;
    for (int r = 0; r < bp; ++r) acc += __uint_as_float((uint32_t)qp[(int64_t)r * a.hq * D] << 16);
    qbar[tid] = acc / (float)bp;
  }
  __syncthreads();
  // logits over key blocks
  float mx = -INFINITY;
  for (int J = tid; J < nb; J += kThreads) {
    const float *kb = a.kbar + ((int64_t)(a.st.nb_off[s] + J) * a.hkv + g) * D;
    float dot = 0.f;
#pragma unroll 8
    for (int d = 0; d < D; ++d) dot = fmaf(qbar[d], kb[d], dot);
    const float x = dot * a.scale;
    dyn[J] = x;
    mx = fmaxf(mx, x);
  }
  mx = block_max(mx, fscr);
  double se = 0.0;
  for (int J = tid; J < nb; J += kThreads) se += (double)expf(dyn[J] - mx);
  se = block_sum(se, dscr);
  // JSD terms, double precision
  double jsd = 0.0;
  const float *av = a.a_v + (int64_t)h * a.total_tokens + tok0;
  for (int J = tid; J < nb; J += kThreads) {
    const double pb = (double)expf(dyn[J] - mx) / se;              // a_bar[J]
    double ph = 0.0;                                                // a_hat[J]
    const int j1 = min((J + 1) * a.block, n);
    for (int j = J * a.block; j < j1; ++j) ph += (double)av[j];
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

constexpr int QT = 64;   // rows and columns of A_bar per workgroup tile

// Tile (TI, TJ), TJ <= TI, of the logits scale * Q_bar_I . K_bar_J written into the
// flattened causal layout.  Grid x enumerates the causal tile pairs of all sequences.
template <int D>
__global__ __launch_bounds__(kThreads) void qa_logits(SelectArgs a) {
  constexpr int DC = 64;                 // d staged per step
  __shared__ float Qs[QT][DC + 1];
  __shared__ float Ks[QT][DC + 1];
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
  const int tid = threadIdx.x;
  const int ti = tid / 16, tj = tid % 16;
  float acc[4][4] = {};
  for (int d0 = 0; d0 < D; d0 += DC) {
    __syncthreads();
    for (int i = tid; i < QT * DC; i += kThreads) {
      const int row = i / DC, d = d0 + i % DC;
      const int I = TI * QT + row, J = TJ * QT + row;
      Qs[row][i % DC] = I < nb ? a.qbar[((int64_t)(a.st.nb_off[s] + I) * a.hq + h) * D + d] : 0.f;
      Ks[row][i % DC] = J < nb ? a.kbar[((int64_t)(a.st.nb_off[s] + J) * a.hkv + g) * D + d] : 0.f;
    }
    __syncthreads();
    for (int d = 0; d < DC; ++d) {
      float qv[4], kv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        qv[i] = Qs[ti + 16 * i][d];
        kv[i] = Ks[tj + 16 * i][d];
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(qv[i], kv[j], acc[i][j]);
    }
  }
  float *flat = a.flat + (int64_t)h * a.tri_total + a.st.tri_off[s];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int I = TI * QT + ti + 16 * i;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int J = TJ * QT + tj + 16 * j;
      if (I < nb && J <= I) flat[(int64_t)I * (I + 1) / 2 + J] = acc[i][j] * a.scale;
    }
  }
}

// Row softmax over J <= I of the flattened logits, one wave per row (in place).
__global__ __launch_bounds__(kThreads) void qa_softmax(SelectArgs a) {
  const int h = blockIdx.y;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= a.nb_total) return;
  const int s = seq_of_block(a.st, row);
  if (a.pattern[s * a.hq + h] != FP_PATTERN_QUERY_AWARE) return;
  const int I = row - a.st.nb_off[s];
  float *x = a.flat + (int64_t)h * a.tri_total + a.st.tri_off[s] + (int64_t)I * (I + 1) / 2;
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
  const size_t dyn = (size_t)a.st.max_nb * sizeof(float);
  if (a.d == 128)
    hipLaunchKernelGGL(pattern_search<128>, dim3(a.st.n_seq, a.hq), dim3(kThreads), dyn, stream, a);
  else
    hipLaunchKernelGGL(pattern_search<64>, dim3(a.st.n_seq, a.hq), dim3(kThreads), dyn, stream, a);
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
    hipLaunchKernelGGL(qa_logits<128>, dim3(pairs, a.hq), dim3(kThreads), 0, stream, a);
  else
    hipLaunchKernelGGL(qa_logits<64>, dim3(pairs, a.hq), dim3(kThreads), 0, stream, a);
  hipLaunchKernelGGL(qa_softmax, dim3((a.nb_total + 3) / 4, a.hq), dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace fp
