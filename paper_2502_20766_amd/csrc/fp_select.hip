// Cumulative-attention index selection and conversion to key-block lists, for gfx950.
//
// Selection (Algorithms 3 and 4, "minimum computational budget"): for a score vector a,
// order the units by (score desc, id asc) and keep the shortest prefix whose normalised
// mass reaches gamma -- the greedy optimum of the objective equation (Appendix B).  The
// set is found without sorting: a three-digit radix select over the fp32 bit patterns
// (monotone for non-negative floats) finds the threshold key t* such that
//     mass(keys > t*) < gamma * total <= mass(keys >= t*),
// then takes the c lowest-id units with key == t* that are still needed.  Masses are
// accumulated as 2^-48 fixed-point integers, so every sum is exact and independent of
// atomic order: the selected set is bit-reproducible.  Normalisation by the explicit
// total is folded into the threshold (prefix >= gamma * total).
//
// Conversion: vertical-slash heads extend selected lines to the whole matrix (Section 3,
// vertical-slash head) at key-block granularity.  A vertical line j marks key block
// floor(j/b) for every query block at or below it; a slash line o = Delta*b + t marks the
// block diagonal Delta in every query block whose rows reach an offset-t key in it
// (t < rows of the query block), and the diagonal Delta+1 when t > 0.  Query-aware heads
// mark their selected (I, J) units.  Every row then keeps key blocks 0 and I and is
// topped up to min(m, I+1) blocks (query-aware: highest pooled score first, then lowest
// J; vertical-slash: nearest the diagonal first) -- the guards of Section 4.1.  With a
// maximum budget M, rows above M blocks keep 0, I and their other blocks in that same
// order (appendix "maximum budget limit").  Query-aware heads may instead select per query
// block (appendix "flatten ablation"); those rows, and capped query-aware rows, are
// finished by qa_rows.  With block-pooled lines the vertical-slash units are key blocks
// and offset blocks of lines (pool_lines), and a selected unit marks the tiles of all its
// lines.
#include "fp_internal.h"
#include "fp_sort.h"

namespace fp {

hipError_t launch_rep_scores(const SelectArgs &a, hipStream_t stream);
hipError_t launch_pattern_search(const SelectArgs &a, hipStream_t stream);
hipError_t launch_pool_q_query_aware(const SelectArgs &a, hipStream_t stream);
hipError_t launch_qa_estimate(const SelectArgs &a, hipStream_t stream);

namespace {

constexpr int kMaxNb = 8192;
constexpr int kSlice = 4096;          // units per histogram workgroup
constexpr double kFxScale = 281474976710656.0;   // 2^48

__device__ __forceinline__ unsigned long long to_fx(float x) {
  return x > 0.f ? (unsigned long long)((double)x * kFxScale) : 0ull;
}

struct Problem {
  const float *scores;
  int n;
  bool active;
};

__device__ __forceinline__ Problem problem_of(const SelectArgs &a, int p) {
  const int kind = p & 1;
  const int sh = p >> 1;
  const int s = sh / a.hq, h = sh % a.hq;
  const int pat = a.pattern[s * a.hq + h];
  const int tok0 = a.st.cu[s];
  const int n = a.st.cu[s + 1] - tok0;
  Problem pr{nullptr, 0, false};
  if (pat == FP_PATTERN_VERTICAL_SLASH && a.vs_granularity == 1) {
    pr.scores = (kind == 0 ? a.av_blk : a.as_blk) + (int64_t)h * a.nb_total + a.st.nb_off[s];
    pr.n = a.st.nb_off[s + 1] - a.st.nb_off[s];
    pr.active = true;
  } else if (pat == FP_PATTERN_VERTICAL_SLASH) {
    pr.scores = (kind == 0 ? a.a_v : a.a_s) + (int64_t)h * a.total_tokens + tok0;
    pr.n = n;
    pr.active = true;
  } else if (pat == FP_PATTERN_QUERY_AWARE && kind == 0 && a.qa_mode == 0) {
    const int nb = a.st.nb_off[s + 1] - a.st.nb_off[s];
    pr.scores = a.flat + (int64_t)h * a.tri_total + a.st.tri_off[s];
    pr.n = nb * (nb + 1) / 2;
    pr.active = true;
  }
  return pr;
}

// Inclusive scan, in thread order over the workgroup, of a (fixed-point mass, count) pair
// per thread, and the workgroup totals: a scan inside each wave through lane shuffles, then
// the NW wave totals through `wm`/`wc` (one barrier; the caller separates reuses of them
// by another).  Integer additions: the result does not depend on their order.
template <int NW>
__device__ __forceinline__ void block_incl_scan(unsigned long long &m, uint32_t &c,
                                                unsigned long long *wm, uint32_t *wc,
                                                unsigned long long &tot_m, uint32_t &tot_c) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const unsigned long long vm = __shfl_up(m, off);
    const uint32_t vc = __shfl_up(c, off);
    if (lane >= off) {
      m += vm;
      c += vc;
    }
  }
  if (lane == 63) {
    wm[w] = m;
    wc[w] = c;
  }
  __syncthreads();
  unsigned long long before_m = 0ull;
  uint32_t before_c = 0u;
  tot_m = 0ull;
  tot_c = 0u;
#pragma unroll
  for (int k = 0; k < NW; ++k) {
    const unsigned long long x = wm[k];
    const uint32_t y = wc[k];
    if (k < w) {
      before_m += x;
      before_c += y;
    }
    tot_m += x;
    tot_c += y;
  }
  m += before_m;
  c += before_c;
}

__device__ __forceinline__ bool is_selected(const SelState &S, float x, int id) {
  const uint32_t key = __float_as_uint(x);
  return key > S.key || (key == S.key && id <= S.idcut);
}

__global__ void sel_init(SelectArgs a) {
  const int p = blockIdx.x;
  for (int b = threadIdx.x; b < kHistBuckets; b += blockDim.x) {
    a.hist_cnt[(int64_t)p * kHistBuckets + b] = 0u;
    a.hist_mass[(int64_t)p * kHistBuckets + b] = 0ull;
  }
  if ((p & 1) == 0) {                     // clear the line marks of this (sequence, head)
    const int sh = p >> 1, s = sh / a.hq, h = sh % a.hq;
    const int nb = a.st.nb_off[s + 1] - a.st.nb_off[s];
    uint32_t *mk = reinterpret_cast<uint32_t *>(a.vs_marks) +
                   (int64_t)h * a.nb_total + a.st.nb_off[s];
    for (int i = threadIdx.x; i < nb; i += blockDim.x) mk[i] = 0u;
  }
  if (threadIdx.x == 0) {
    const Problem pr = problem_of(a, p);
    SelState S = {};
    S.mode = pr.active ? 0 : 2;
    S.n = pr.n;
    S.idcut = -1;
    a.sel[p] = S;
  }
}

template <int PASS>
__global__ __launch_bounds__(256) void sel_hist(SelectArgs a) {
  __shared__ uint32_t cnt[kHistBuckets];
  __shared__ unsigned long long mass[kHistBuckets];
  const int p = blockIdx.y;
  const SelState S = a.sel[p];
  if (S.mode != 0) return;
  const int start = blockIdx.x * kSlice;
  if (start >= S.n) return;
  const Problem pr = problem_of(a, p);
  for (int b = threadIdx.x; b < kHistBuckets; b += blockDim.x) {
    cnt[b] = 0u;
    mass[b] = 0ull;
  }
  __syncthreads();
  constexpr int shift = PASS == 0 ? 21 : (PASS == 1 ? 10 : 0);
  constexpr uint32_t dmask = PASS == 2 ? 1023u : 2047u;
  const int end = min(start + kSlice, S.n);
  const int nt = blockDim.x;
  // four scores per thread are loaded before their histogram updates
  for (int base = start + threadIdx.x; base < end; base += 4 * nt) {
    float xs[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int i = base + u * nt;
      xs[u] = i < end ? pr.scores[i] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      if (base + u * nt >= end) break;
      const float x = xs[u];
      const uint32_t key = __float_as_uint(x);
      bool match = true;
      if (PASS == 1) match = (key >> 21) == (S.prefix >> 21);
      if (PASS == 2) match = (key >> 10) == (S.prefix >> 10);
      if (match) {
        const uint32_t dg = (key >> shift) & dmask;
        atomicAdd(&cnt[dg], 1u);
        atomicAdd(&mass[dg], to_fx(x));
      }
    }
  }
  __syncthreads();
  for (int b = threadIdx.x; b < kHistBuckets; b += blockDim.x) {
    if (cnt[b]) {
      atomicAdd(&a.hist_cnt[(int64_t)p * kHistBuckets + b], cnt[b]);
      atomicAdd(&a.hist_mass[(int64_t)p * kHistBuckets + b], mass[b]);
    }
  }
}

// Find the digit whose bucket carries the cumulative mass across the threshold.  Thread t
// owns buckets [2048 - 8(t+1), 2048 - 8t), so thread order is descending key order.
template <int PASS>
__global__ __launch_bounds__(256) void sel_scan(SelectArgs a) {
  __shared__ unsigned long long wmass[4];
  __shared__ uint32_t wcnt[4];
  const int p = blockIdx.x, tid = threadIdx.x;
  SelState S = a.sel[p];
  if (S.mode != 0) return;
  unsigned long long *hm = a.hist_mass + (int64_t)p * kHistBuckets;
  uint32_t *hc = a.hist_cnt + (int64_t)p * kHistBuckets;
  const int top = kHistBuckets - 8 * tid;   // exclusive upper bucket
  unsigned long long bm[8];
  uint32_t bc[8];
  unsigned long long lm = 0;
  uint32_t lc = 0;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    bm[i] = hm[top - 1 - i];
    bc[i] = hc[top - 1 - i];
    lm += bm[i];
    lc += bc[i];
  }
  unsigned long long im = lm, s_total;
  uint32_t ic = lc, s_count;
  block_incl_scan<4>(im, ic, wmass, wcnt, s_total, s_count);
  const unsigned long long excl_m = im - lm;
  const uint32_t excl_c = ic - lc;
  if (PASS == 0) {
    const unsigned long long total = s_total;
    S.total = total;
    if (total == 0ull) {
      S.mode = 1;
    } else {
      double t = ceil((double)a.gamma * (double)total);
      unsigned long long thr = (unsigned long long)t;
      if (thr < 1ull) thr = 1ull;
      if (thr > total) S.mode = 1;    // never reached: take every unit
      S.thr = thr;
    }
    if (S.mode == 1) {
      S.key = 0u;
      S.idcut = 0x7FFFFFFF;
      S.k = S.n;
    }
  }
  __syncthreads();
  // all threads zero their buckets for the next pass once everyone has read them
  for (int i = 0; i < 8; ++i) {
    hm[top - 1 - i] = 0ull;
    hc[top - 1 - i] = 0u;
  }
  if (S.mode == 1) {
    if (tid == 0) a.sel[p] = S;
    return;
  }
  constexpr int shift = PASS == 0 ? 21 : (PASS == 1 ? 10 : 0);
  unsigned long long run = S.mass_above + excl_m;
  uint32_t runc = S.cnt_above + excl_c;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    if (run < S.thr && run + bm[i] >= S.thr) {
      const uint32_t digit = (uint32_t)(top - 1 - i);
      S.prefix |= digit << shift;
      S.mass_above = run;
      S.cnt_above = runc;
      if (PASS == 2) {
        S.key = S.prefix;
        S.n_eq = bc[i];
        const unsigned long long f = bm[i] / bc[i];   // equal keys carry equal mass
        const unsigned long long need = (S.thr - run + f - 1) / f;
        S.need_eq = (uint32_t)need;
        S.k = (int32_t)(runc + need);
        S.idcut = (need >= bc[i]) ? 0x7FFFFFFF : -1;
      }
      a.sel[p] = S;
    }
    run += bm[i];
    runc += bc[i];
  }
}

// Lowest-id tie break: find the id of the need_eq-th unit (in id order) whose key equals
// the threshold key.  Only runs when some but not all of those units are taken.
__global__ __launch_bounds__(1024) void sel_tie(SelectArgs a) {
  __shared__ uint32_t wcount[16];
  __shared__ int found;
  const int p = blockIdx.x;
  SelState S = a.sel[p];
  if (S.mode != 0 || S.idcut != -1) return;
  const Problem pr = problem_of(a, p);
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
  uint32_t running = 0;
  if (tid == 0) found = -1;
  __syncthreads();
  for (int base = 0; base < S.n; base += 1024) {
    const int i = base + tid;
    const bool f = i < S.n && __float_as_uint(pr.scores[i]) == S.key;
    const unsigned long long bal = __ballot(f);
    if (lane == 0) wcount[w] = (uint32_t)__popcll(bal);
    __syncthreads();
    uint32_t before = 0, chunk = 0;
    for (int k = 0; k < 16; ++k) {
      if (k < w) before += wcount[k];
      chunk += wcount[k];
    }
    const uint32_t rank = running + before + (uint32_t)__popcll(bal & __lanemask_lt());
    if (f && rank + 1 == S.need_eq) found = i;
    __syncthreads();
    if (found >= 0) break;
    running += chunk;
    __syncthreads();
  }
  if (tid == 0) {
    S.idcut = found;
    a.sel[p] = S;
  }
}

// Short problems: every selection problem of the call in one 1024-thread workgroup, the
// three radix passes through an LDS histogram and the lowest-id tie break in the same
// launch -- one launch instead of the seven above, the same threshold key, counts and
// tie cut (every sum is an exact integer, so the result does not depend on the path).
constexpr int kSmallUnits = 16384;    // largest problem (units) taken by sel_small

__global__ __launch_bounds__(1024) void sel_small(SelectArgs a) {
  __shared__ uint32_t cnt[kHistBuckets];
  __shared__ unsigned long long mass[kHistBuckets];
  __shared__ unsigned long long wmass[16];
  __shared__ uint32_t wcnt[16];
  __shared__ SelState sS;
  __shared__ uint32_t wcount[16];
  __shared__ int found;
  const int p = blockIdx.x, tid = threadIdx.x;
  SelState S = a.sel[p];
  if (S.mode != 0) return;                // the same decision in every thread
  const Problem pr = problem_of(a, p);
  const int top = kHistBuckets - 2 * tid; // thread t owns buckets [top - 2, top): thread
                                          // order is descending key order
#pragma unroll 1
  for (int pass = 0; pass < 3; ++pass) {
    const int shift = pass == 0 ? 21 : (pass == 1 ? 10 : 0);
    const uint32_t dmask = pass == 2 ? 1023u : 2047u;
    for (int b = tid; b < kHistBuckets; b += 1024) {
      cnt[b] = 0u;
      mass[b] = 0ull;
    }
    if (tid == 0) sS = S;
    __syncthreads();
    for (int i = tid; i < S.n; i += 1024) {
      const float x = pr.scores[i];
      const uint32_t key = __float_as_uint(x);
      const bool match = pass == 0 || (pass == 1 && (key >> 21) == (S.prefix >> 21)) ||
                         (pass == 2 && (key >> 10) == (S.prefix >> 10));
      if (match) {
        const uint32_t dg = (key >> shift) & dmask;
        atomicAdd(&cnt[dg], 1u);
        atomicAdd(&mass[dg], to_fx(x));
      }
    }
    __syncthreads();
    unsigned long long bm[2];
    uint32_t bc[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      bm[i] = mass[top - 1 - i];
      bc[i] = cnt[top - 1 - i];
    }
    const unsigned long long lm = bm[0] + bm[1];
    const uint32_t lc = bc[0] + bc[1];
    unsigned long long im = lm, total_m;
    uint32_t ic = lc, total_c;
    block_incl_scan<16>(im, ic, wmass, wcnt, total_m, total_c);
    const unsigned long long excl_m = im - lm;
    const uint32_t excl_c = ic - lc;
    if (pass == 0) {
      const unsigned long long total = total_m;
      S.total = total;
      if (total == 0ull) {
        S.mode = 1;
      } else {
        double t = ceil((double)a.gamma * (double)total);
        unsigned long long thr = (unsigned long long)t;
        if (thr < 1ull) thr = 1ull;
        if (thr > total) S.mode = 1;      // never reached: take every unit
        S.thr = thr;
      }
      if (S.mode == 1) {                  // the same in every thread
        S.key = 0u;
        S.idcut = 0x7FFFFFFF;
        S.k = S.n;
        if (tid == 0) a.sel[p] = S;
        return;
      }
      if (tid == 0) sS = S;
      __syncthreads();
    }
    unsigned long long run = S.mass_above + excl_m;
    uint32_t runc = S.cnt_above + excl_c;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      if (run < S.thr && run + bm[i] >= S.thr) {   // exactly one bucket of all threads
        SelState T = S;
        const uint32_t digit = (uint32_t)(top - 1 - i);
        T.prefix |= digit << shift;
        T.mass_above = run;
        T.cnt_above = runc;
        if (pass == 2) {
          T.key = T.prefix;
          T.n_eq = bc[i];
          const unsigned long long f = bm[i] / bc[i];   // equal keys carry equal mass
          const unsigned long long need = (T.thr - run + f - 1) / f;
          T.need_eq = (uint32_t)need;
          T.k = (int32_t)(runc + need);
          T.idcut = (need >= bc[i]) ? 0x7FFFFFFF : -1;
        }
        sS = T;
      }
      run += bm[i];
      runc += bc[i];
    }
    __syncthreads();
    S = sS;
    __syncthreads();                      // every thread has read sS before it is reused
  }
  // lowest-id tie break (as sel_tie), when some but not all units of the key are taken
  if (S.idcut == -1) {
    const int w = tid >> 6, lane = tid & 63;
    uint32_t running = 0;
    if (tid == 0) found = -1;
    __syncthreads();
    for (int base = 0; base < S.n; base += 1024) {
      const int i = base + tid;
      const bool f = i < S.n && __float_as_uint(pr.scores[i]) == S.key;
      const unsigned long long bal = __ballot(f);
      if (lane == 0) wcount[w] = (uint32_t)__popcll(bal);
      __syncthreads();
      uint32_t before = 0, chunk = 0;
      for (int k = 0; k < 16; ++k) {
        if (k < w) before += wcount[k];
        chunk += wcount[k];
      }
      const uint32_t rank = running + before + (uint32_t)__popcll(bal & __lanemask_lt());
      if (f && rank + 1 == S.need_eq) found = i;
      __syncthreads();
      if (found >= 0) break;
      running += chunk;
      __syncthreads();
    }
    S.idcut = found;
  }
  if (tid == 0) a.sel[p] = S;
}

// ---------------------------------------------------------------- conversion to lists

// Vertical-slash heads: mark, per key block / block diagonal, what the selected lines
// reach (vertical j: column floor(j/b); slash o = D*b + t: diagonal D in full query blocks,
// diagonal D in the partial last query block when t < its rows, diagonal D+1 when t > 0).
// One workgroup per (sequence, head, slice of kMarkSlice lines); the stores only ever
// write 1, so their order does not matter.
constexpr int kMarkSlice = 8192;

__global__ __launch_bounds__(256) void vs_marks(SelectArgs a) {
  const int s = blockIdx.x / a.hq, h = blockIdx.x % a.hq;
  if (a.pattern[s * a.hq + h] != FP_PATTERN_VERTICAL_SLASH) return;
  const int tok0 = a.st.cu[s];
  const int n = a.st.cu[s + 1] - tok0;
  const int b = a.block;
  const int nb = a.st.nb_off[s + 1] - a.st.nb_off[s];
  const int last_rows = n - (nb - 1) * b;
  const int p0 = (s * a.hq + h) * 2;
  const SelState S0 = a.sel[p0];
  const SelState S1 = a.sel[p0 + 1];
  uint8_t *mk = a.vs_marks + 4 * ((int64_t)h * a.nb_total + a.st.nb_off[s]);
  if (a.vs_granularity == 1) {
    // a selected unit selects all its lines: key block J is a column; offset block D
    // holds o = D*b (t = 0: diagonal D in every row) and, when it has more than one
    // offset, o = D*b + t with t > 0 (diagonal D + 1)
    const int u = blockIdx.y * blockDim.x + threadIdx.x;
    if (u >= nb) return;
    const float *avb = a.av_blk + (int64_t)h * a.nb_total + a.st.nb_off[s];
    const float *asb = a.as_blk + (int64_t)h * a.nb_total + a.st.nb_off[s];
    if (is_selected(S0, avb[u], u)) mk[4 * u + 0] = 1;
    if (is_selected(S1, asb[u], u)) {
      mk[4 * u + 1] = 1;
      mk[4 * u + 2] = 1;
      if (n - u * b > 1 && u + 1 < nb) mk[4 * (u + 1) + 3] = 1;
    }
    return;
  }
  const float *av = a.a_v + (int64_t)h * a.total_tokens + tok0;
  const float *as = a.a_s + (int64_t)h * a.total_tokens + tok0;
  const int j0 = blockIdx.y * kMarkSlice;
  const int j1 = min(j0 + kMarkSlice, n);
  // four scores per thread are loaded before any mark is stored (a byte store may alias
  // the scores, so the compiler would otherwise wait for each load in turn)
  const int nt = blockDim.x;
  for (int base = j0 + threadIdx.x; base < j1; base += 4 * nt) {
    float xv[4], xs[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int j = base + u * nt;
      xv[u] = j < j1 ? av[j] : 0.f;
      xs[u] = j < j1 ? as[j] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int j = base + u * nt;
      if (j >= j1) break;
      if (is_selected(S0, xv[u], j)) mk[4 * (j / b) + 0] = 1;
      if (is_selected(S1, xs[u], j)) {
        const int dl = j / b, t = j % b;
        mk[4 * dl + 1] = 1;
        if (t < last_rows) mk[4 * dl + 2] = 1;
        if (t > 0 && dl + 1 < nb) mk[4 * (dl + 1) + 3] = 1;
      }
    }
  }
}

// Lists of one (sequence, head): grid (sequence * head, row slice); wave w of slice r
// converts rows I = 16 r + w + 16 R k.
__global__ __launch_bounds__(1024) void convert_tiles(SelectArgs a) {
  __shared__ uint8_t colsel[kMaxNb];
  __shared__ uint8_t d0[kMaxNb];
  __shared__ uint8_t d0p[kMaxNb];
  __shared__ uint8_t d1[kMaxNb + 1];
  __shared__ int added[16][FP_MAX_MIN_BUDGET];
  const int s = blockIdx.x / a.hq, h = blockIdx.x % a.hq;
  const int slice = blockIdx.y, n_slices = gridDim.y;
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
  const int tok0 = a.st.cu[s];
  const int n = a.st.cu[s + 1] - tok0;
  const int b = a.block;
  const int nb = a.st.nb_off[s + 1] - a.st.nb_off[s];
  const int pat = a.pattern[s * a.hq + h];
  const bool vs = pat == FP_PATTERN_VERTICAL_SLASH;
  const int p0 = (s * a.hq + h) * 2;
  const SelState S0 = a.sel[p0];
  const SelState S1 = a.sel[p0 + 1];
  const float *flat = a.flat + (int64_t)h * a.tri_total + a.st.tri_off[s];
  (void)tok0;
  (void)n;
  if (slice * 16 >= nb) return;                 // no row of this (sequence, head) here

  if (vs) {
    const uint32_t *mk = reinterpret_cast<const uint32_t *>(a.vs_marks) +
                         (int64_t)h * a.nb_total + a.st.nb_off[s];
    for (int i = tid; i < nb; i += blockDim.x) {
      const uint32_t m4 = mk[i];
      colsel[i] = m4 & 0xFF;
      d0[i] = (m4 >> 8) & 0xFF;
      d0p[i] = (m4 >> 16) & 0xFF;
      d1[i] = m4 >> 24;
    }
    if (tid == 0) d1[nb] = 0;
    __syncthreads();
  }
  if (tid == 0 && slice == 0) {
    // per-query-block selection accumulates its K over the rows (qa_rows, launched next)
    a.units[(s * a.hq + h) * 2 + 0] = (!vs && a.qa_mode == 1) ? 0 : S0.k;
    a.units[(s * a.hq + h) * 2 + 1] = vs ? S1.k : 0;
  }
  if (!vs && (a.qa_mode == 1 || a.max_budget > 0)) return;   // rows written by qa_rows
  const int last_rows = n - (nb - 1) * b;            // rows of the last query block

  const int m = a.min_budget;
  for (int I = slice * 16 + w; I < nb; I += 16 * n_slices) {
    const bool row_full = (I < nb - 1) || (last_rows == b);
    const int64_t tri_row = (int64_t)I * (I + 1) / 2;
    auto sel = [&](int J) -> bool {
      if (J == 0 || J == I) return true;
      if (vs) {
        const int dl = I - J;
        return colsel[J] || (row_full ? d0[dl] : d0p[dl]) || d1[dl];
      }
      return is_selected(S0, flat[tri_row + J], (int)(tri_row + J));
    };
    // selected count, only as far as the minimum budget needs it (exact whenever it stays
    // below the target, which is the only case that uses it)
    const int target = min(m, I + 1);
    int count = 0;
    for (int J0 = 0; J0 <= I && count < target; J0 += 64) {
      const int J = J0 + lane;
      count += __popcll(__ballot(J <= I && sel(J)));
    }
    int jmin = I;          // vertical-slash top-up: every unselected J in [jmin, I)
    int n_added = 0;       // query-aware top-up: added[w][0..n_added)
    if (count < target) {
      int need = target - count;
      if (vs) {
        for (int top = I - 1; top >= 0 && need > 0; top -= 64) {
          const int J = top - lane;
          const bool un = J >= 0 && !sel(J);
          const unsigned long long bal = __ballot(un);
          const int c = __popcll(bal);
          if (c >= need) {
            const int rank = __popcll(bal & __lanemask_lt());
            const unsigned long long pick = __ballot(un && rank == need - 1);
            jmin = top - (__ffsll((long long)pick) - 1);
            need = 0;
          } else {
            need -= c;
            jmin = top - 63;
          }
        }
      } else {
        for (; n_added < need; ++n_added) {
          float best = -1.f;
          int bj = 0x7FFFFFFF;
          // four 64-block chunks per step, their scores loaded before the first is tested
          for (int J0 = 0; J0 <= I; J0 += 256) {
            float xs[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
              const int J = J0 + 64 * u + lane;
              xs[u] = J <= I ? flat[tri_row + J] : 0.f;
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) {
              const int J = J0 + 64 * u + lane;
              if (J > I || J == 0 || J == I || is_selected(S0, xs[u], (int)(tri_row + J)))
                continue;
              bool taken = false;
              for (int q = 0; q < n_added; ++q) taken |= (added[w][q] == J);
              if (taken) continue;
              const float x = xs[u];
              if (x > best || (x == best && J < bj)) { best = x; bj = J; }
            }
          }
          for (int off = 32; off > 0; off >>= 1) {
            const float ob = __shfl_xor(best, off);
            const int oj = __shfl_xor(bj, off);
            if (ob > best || (ob == best && oj < bj)) { best = ob; bj = oj; }
          }
          if (lane == 0) added[w][n_added] = bj;
          __builtin_amdgcn_wave_barrier();
          __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
        }
      }
    }
    auto kept = [&](int J) -> bool {
      bool f = sel(J) || (J >= jmin && J < I);
      for (int q = 0; q < n_added; ++q) f |= (added[w][q] == J);
      return f;
    };
    // maximum budget (vertical-slash rows; query-aware rows are capped in qa_rows): keep
    // blocks 0 and I and the nearest-to-diagonal others, i.e. every kept J >= jcap
    int jcap = 0;
    if (vs && a.max_budget > 0 && I > 0) {
      int total = 0;
      for (int J0 = 0; J0 <= I; J0 += 64) {
        const int J = J0 + lane;
        total += __popcll(__ballot(J <= I && kept(J)));
      }
      if (total > a.max_budget) {
        int need = a.max_budget - 2;               // others to keep, nearest I first
        jcap = I;                                    // need == 0: no other block
        for (int top = I - 1; top >= 1 && need > 0; top -= 64) {
          const int J = top - lane;
          const bool f = J >= 1 && kept(J);
          const unsigned long long bal = __ballot(f);
          const int c = __popcll(bal);
          if (c >= need) {
            const int rank = __popcll(bal & __lanemask_lt());
            const unsigned long long pick = __ballot(f && rank == need - 1);
            jcap = top - (__ffsll((long long)pick) - 1);
            need = 0;
          } else {
            need -= c;
          }
        }
      }
    }
    int32_t *out = a.kb_idx + (int64_t)h * a.tri_total + a.st.tri_off[s] + tri_row;
    int running = 0;
    // four 64-block chunks per step; a query-aware row's scores of all four are loaded
    // before the first is tested
    for (int J0 = 0; J0 <= I; J0 += 256) {
      float xs[4] = {0.f, 0.f, 0.f, 0.f};
      if (!vs) {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int J = J0 + 64 * u + lane;
          if (J <= I) xs[u] = flat[tri_row + J];
        }
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int J = J0 + 64 * u + lane;
        bool f = false;
        if (J <= I) {
          bool k = (J == 0 || J == I) ? true
                   : vs               ? sel(J)
                                      : is_selected(S0, xs[u], (int)(tri_row + J));
          k = k || (J >= jmin && J < I);
          for (int q = 0; q < n_added; ++q) k |= (added[w][q] == J);
          f = k && (J == 0 || J == I || J >= jcap);
        }
        const unsigned long long bal = __ballot(f);
        if (f) out[running + __popcll(bal & __lanemask_lt())] = J;
        running += __popcll(bal);
      }
    }
    if (lane == 0) a.kb_cnt[(int64_t)h * a.nb_total + a.st.nb_off[s] + I] = running;
  }
}

// Block-pooled lines: a_v summed over each key block and a_s over each offset block, one
// wave per (query head, block); vertical-slash heads only.
__global__ __launch_bounds__(256) void pool_lines(SelectArgs a) {
  const int h = blockIdx.y;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= a.nb_total) return;
  int s = 0;
  while (s + 1 < a.st.n_seq && a.st.nb_off[s + 1] <= row) ++s;
  if (a.pattern[s * a.hq + h] != FP_PATTERN_VERTICAL_SLASH) return;
  const int u = row - a.st.nb_off[s];
  const int tok0 = a.st.cu[s];
  const int n = a.st.cu[s + 1] - tok0;
  const int lo = u * a.block, hi = min(lo + a.block, n);
  const float *av = a.a_v + (int64_t)h * a.total_tokens + tok0;
  const float *as = a.a_s + (int64_t)h * a.total_tokens + tok0;
  float sv = 0.f, ss = 0.f;
  for (int j = lo + lane; j < hi; j += 64) {
    sv += av[j];
    ss += as[j];
  }
  for (int off = 32; off > 0; off >>= 1) {
    sv += __shfl_xor(sv, off);
    ss += __shfl_xor(ss, off);
  }
  if (lane == 0) {
    a.av_blk[(int64_t)h * a.nb_total + row] = sv;
    a.as_blk[(int64_t)h * a.nb_total + row] = ss;
  }
}

// Query-aware rows when the selection is per query block (qa_mode 1) or rows are capped
// (max_budget > 0).  One workgroup per (query head, query block I): the row's pooled scores
// A_bar[I, J], J <= I, are sorted by (score desc, J asc).  The gamma-selected units of the
// row are then a prefix of that order in both modes (flattened: the head's radix
// threshold; per query block: the shortest prefix whose exact fixed-point mass reaches
// ceil(gamma * row total)).  Blocks 0 and I are always kept; the other blocks are taken
// along the same order: the selected prefix, raised to min(m, I+1) blocks in total by the
// top-up and lowered to max_budget by the cap.
constexpr int kRowWavesMax = 8;

struct RowShared {
  unsigned long long wsum[kRowWavesMax];
  uint32_t wcnt[kRowWavesMax];
  int pos0, posI, kcut;
};

template <typename T>
__device__ __forceinline__ T wave_incl_scan(T v, int lane) {
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const T u = __shfl_up(v, off);
    if (lane >= off) v += u;
  }
  return v;
}

// One row of NT*E >= I+1 sort slots (E a power of two).
template <int NT, int E>
__device__ void qa_row(const SelectArgs &a, unsigned long long *lds, uint8_t *keep,
                       RowShared &sh, int s, int h, int I, int row) {
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int len = I + 1;
  const int64_t tri_row = (int64_t)I * (I + 1) / 2;
  const float *x = a.flat + (int64_t)h * a.tri_total + a.st.tri_off[s] + tri_row;
  unsigned long long k[E];                           // (~score bits) << 32 | J
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int i = tid * E + e;
    k[e] = i < len ? ((unsigned long long)(~__float_as_uint(x[i])) << 32) | (uint32_t)i
                   : ~0ull;
  }
  if (tid == 0) sh.kcut = len;
  bitonic_sort<NT, E, 2>(k, lds, tid);
  auto score_of = [](unsigned long long key) { return __uint_as_float(~(uint32_t)(key >> 32)); };
  auto id_of = [](unsigned long long key) { return (int)(key & 0xFFFFFFFFu); };
  // positions of the forced blocks 0 and I in the order
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int p = tid * E + e;
    if (p < len) {
      const int J = id_of(k[e]);
      if (J == 0) sh.pos0 = p;
      if (J == I) sh.posI = p;
    }
  }
  int K;                                             // gamma-selected units of the row
  if (a.qa_mode == 1) {
    auto mass_at = [&](int e) {
      return tid * E + e < len ? to_fx(score_of(k[e])) : 0ull;
    };
    unsigned long long mine = 0ull;
#pragma unroll
    for (int e = 0; e < E; ++e) mine += mass_at(e);
    const unsigned long long incl = wave_incl_scan(mine, lane);
    if (lane == 63) sh.wsum[w] = incl;
    __syncthreads();
    unsigned long long run = incl - mine, total = 0ull;
#pragma unroll
    for (int q = 0; q < NT / 64; ++q) {
      if (q < w) run += sh.wsum[q];
      total += sh.wsum[q];
    }
    unsigned long long thr = (unsigned long long)ceil((double)a.gamma * (double)total);
    if (thr < 1ull) thr = 1ull;
    if (total > 0ull && thr <= total) {
      int cut = len;
#pragma unroll
      for (int e = 0; e < E; ++e) {
        run += mass_at(e);
        if (cut == len && run >= thr) cut = tid * E + e + 1;
      }
      if (cut < len) atomicMin(&sh.kcut, cut);
    }
    __syncthreads();
    K = sh.kcut;
    if (tid == 0) atomicAdd(&a.units[(s * a.hq + h) * 2], K);
  } else {
    const SelState S0 = a.sel[(s * a.hq + h) * 2];
    int c = 0;
#pragma unroll
    for (int e = 0; e < E; ++e)
      if (tid * E + e < len)
        c += is_selected(S0, score_of(k[e]), (int)(tri_row + id_of(k[e])));
    c = (int)__reduce_add_sync(~0ull, (unsigned)c);
    if (lane == 0) sh.wcnt[w] = (uint32_t)c;
    __syncthreads();
    K = 0;
#pragma unroll
    for (int q = 0; q < NT / 64; ++q) K += (int)sh.wcnt[q];
  }
  const int pos0 = sh.pos0, posI = sh.posI;
  const int f = I == 0 ? 1 : 2;                       // forced blocks
  const int in_f = (pos0 < K) + (I > 0 && posI < K);
  int k_final = K - in_f;                             // other blocks, along the order
  k_final = max(k_final, min(a.min_budget, len) - f);
  if (a.max_budget > 0) k_final = min(k_final, a.max_budget - f);
  // every J <= I sits at exactly one position p < len, so this writes all of keep[0..I]
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int p = tid * E + e;
    if (p < len) {
      const int J = id_of(k[e]);
      const int rank = p - (pos0 < p) - (I > 0 && posI < p);   // position among the others
      keep[J] = (J == 0 || J == I || rank < k_final) ? 1 : 0;
    }
  }
  __syncthreads();
  // ascending compaction: thread t owns blocks t*E .. t*E+E-1
  uint32_t bits = 0u;
  int cnt = 0;
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int J = tid * E + e;
    if (J < len && keep[J]) {
      bits |= 1u << e;
      ++cnt;
    }
  }
  const int incl = wave_incl_scan(cnt, lane);
  if (lane == 63) sh.wcnt[w] = (uint32_t)incl;
  __syncthreads();
  int base = incl - cnt, total = 0;
#pragma unroll
  for (int q = 0; q < NT / 64; ++q) {
    if (q < w) base += (int)sh.wcnt[q];
    total += (int)sh.wcnt[q];
  }
  int32_t *out = a.kb_idx + (int64_t)h * a.tri_total + a.st.tri_off[s] + tri_row;
#pragma unroll
  for (int e = 0; e < E; ++e)
    if ((bits >> e) & 1u) out[base++] = tid * E + e;
  if (tid == 0) a.kb_cnt[(int64_t)h * a.nb_total + row] = total;
}

// NT threads per row, EMAX = sort slots per thread for the longest row (NT*EMAX >= max_nb).
template <int NT, int EMAX>
__global__ __launch_bounds__(NT) void qa_rows(SelectArgs a) {
  // dynamic LDS: NT*EMAX sort keys, then NT*EMAX keep flags
  extern __shared__ __attribute__((aligned(16))) unsigned char dyn[];
  unsigned long long *lds = reinterpret_cast<unsigned long long *>(dyn);
  uint8_t *keep = dyn + (size_t)NT * EMAX * sizeof(unsigned long long);
  __shared__ RowShared sh;
  const int h = blockIdx.y;
  const int row = blockIdx.x;
  int s = 0;
  while (s + 1 < a.st.n_seq && a.st.nb_off[s + 1] <= row) ++s;
  if (a.pattern[s * a.hq + h] != FP_PATTERN_QUERY_AWARE) return;
  const int I = row - a.st.nb_off[s];
  if (I < NT) {
    qa_row<NT, 1>(a, lds, keep, sh, s, h, I, row);
  } else if (I < 2 * NT) {
    if constexpr (EMAX >= 2) qa_row<NT, 2>(a, lds, keep, sh, s, h, I, row);
  } else if (I < 4 * NT) {
    if constexpr (EMAX >= 4) qa_row<NT, 4>(a, lds, keep, sh, s, h, I, row);
  } else if (I < 8 * NT) {
    if constexpr (EMAX >= 8) qa_row<NT, 8>(a, lds, keep, sh, s, h, I, row);
  } else {
    if constexpr (EMAX >= 16) qa_row<NT, 16>(a, lds, keep, sh, s, h, I, row);
  }
}

// gamma >= 1: every causal key block, no search (full attention).
__global__ __launch_bounds__(256) void dense_lists(SelectArgs a) {
  const int h = blockIdx.y;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= a.nb_total) return;
  int s = 0;
  while (s + 1 < a.st.n_seq && a.st.nb_off[s + 1] <= row) ++s;
  const int I = row - a.st.nb_off[s];
  int32_t *out = a.kb_idx + (int64_t)h * a.tri_total + a.st.tri_off[s] + (int64_t)I * (I + 1) / 2;
  for (int J = lane; J <= I; J += 64) out[J] = J;
  if (lane == 0) a.kb_cnt[(int64_t)h * a.nb_total + row] = I + 1;
  if (I == 0 && lane == 0) {
    const int nb = a.st.nb_off[s + 1] - a.st.nb_off[s];
    a.pattern[s * a.hq + h] = FP_PATTERN_DENSE;
    a.js[s * a.hq + h] = -1.f;
    a.units[(s * a.hq + h) * 2 + 0] = nb * (nb + 1) / 2;
    a.units[(s * a.hq + h) * 2 + 1] = 0;
  }
}

}  // namespace

template <int NT, int EMAX>
hipError_t launch_qa_rows_e(const SelectArgs &a, hipStream_t stream) {
  const size_t dyn = (size_t)NT * EMAX * (sizeof(unsigned long long) + 1);
  if (dyn > 65536) {          // rows above 4096 blocks: allow the larger LDS allocation
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(qa_rows<NT, EMAX>),
                                             hipFuncAttributeMaxDynamicSharedMemorySize,
                                             (int)dyn);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL((qa_rows<NT, EMAX>), dim3(a.nb_total, a.hq), dim3(NT), dyn, stream, a);
  return hipGetLastError();
}

hipError_t launch_qa_rows(const SelectArgs &a, hipStream_t stream) {
  // row I holds I+1 <= max_nb keys in NT*E slots; at most 16 slots per thread keeps the
  // keys in registers, so the longest rows take 512 threads
  if (a.st.max_nb <= 256) return launch_qa_rows_e<256, 1>(a, stream);
  if (a.st.max_nb <= 512) return launch_qa_rows_e<256, 2>(a, stream);
  if (a.st.max_nb <= 1024) return launch_qa_rows_e<256, 4>(a, stream);
  if (a.st.max_nb <= 2048) return launch_qa_rows_e<256, 8>(a, stream);
  if (a.st.max_nb <= 4096) return launch_qa_rows_e<256, 16>(a, stream);
  if (a.st.max_nb <= 8192) return launch_qa_rows_e<512, 16>(a, stream);
  return hipErrorInvalidValue;
}

hipError_t launch_dense_lists(const SelectArgs &a, hipStream_t stream) {
  hipLaunchKernelGGL(dense_lists, dim3((a.nb_total + 3) / 4, a.hq), dim3(256), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_select_pipeline(const SelectArgs &a, hipStream_t stream) {
  hipError_t e;
  if ((e = launch_rep_scores(a, stream)) != hipSuccess) return e;
  if ((e = launch_pattern_search(a, stream)) != hipSuccess) return e;
  if ((e = launch_pool_q_query_aware(a, stream)) != hipSuccess) return e;
  if ((e = launch_qa_estimate(a, stream)) != hipSuccess) return e;
  const int problems = a.st.n_seq * a.hq * 2;
  int max_units = 0;
  for (int s = 0; s < a.st.n_seq; ++s) {
    const int n = a.st.cu[s + 1] - a.st.cu[s];
    const int nb = a.st.nb_off[s + 1] - a.st.nb_off[s];
    max_units = max(max_units, max(n, nb * (nb + 1) / 2));
  }
  const int slices = (max_units + kSlice - 1) / kSlice;
  if (a.vs_granularity == 1)
    hipLaunchKernelGGL(pool_lines, dim3((a.nb_total + 3) / 4, a.hq), dim3(256), 0, stream, a);
  hipLaunchKernelGGL(sel_init, dim3(problems), dim3(256), 0, stream, a);
  if (max_units <= kSmallUnits) {
    hipLaunchKernelGGL(sel_small, dim3(problems), dim3(1024), 0, stream, a);
  } else {
    hipLaunchKernelGGL(sel_hist<0>, dim3(slices, problems), dim3(256), 0, stream, a);
    hipLaunchKernelGGL(sel_scan<0>, dim3(problems), dim3(256), 0, stream, a);
    hipLaunchKernelGGL(sel_hist<1>, dim3(slices, problems), dim3(256), 0, stream, a);
    hipLaunchKernelGGL(sel_scan<1>, dim3(problems), dim3(256), 0, stream, a);
    hipLaunchKernelGGL(sel_hist<2>, dim3(slices, problems), dim3(256), 0, stream, a);
    hipLaunchKernelGGL(sel_scan<2>, dim3(problems), dim3(256), 0, stream, a);
    hipLaunchKernelGGL(sel_tie, dim3(problems), dim3(1024), 0, stream, a);
  }
  {
    int max_n = 0;
    for (int s = 0; s < a.st.n_seq; ++s) max_n = max(max_n, a.st.cu[s + 1] - a.st.cu[s]);
    const int mark_slices = a.vs_granularity == 1 ? (a.st.max_nb + 255) / 256
                                                  : (max_n + kMarkSlice - 1) / kMarkSlice;
    hipLaunchKernelGGL(vs_marks, dim3(a.st.n_seq * a.hq, mark_slices), dim3(256), 0, stream, a);
    // row slices: about two workgroups per CU over all (sequence, head) pairs, and at
    // most four rows per wave on the longest sequence (packed batches mix lengths, and
    // the workgroups of short sequences end early)
    const int pairs = a.st.n_seq * a.hq;
    int slices = max((512 + pairs - 1) / pairs, (a.st.max_nb + 63) / 64);
    slices = max(1, min(slices, (a.st.max_nb + 15) / 16));
    hipLaunchKernelGGL(convert_tiles, dim3(pairs, slices), dim3(1024), 0, stream, a);
  }
  if (a.qa_mode == 1 || a.max_budget > 0) {
    if ((e = hipGetLastError()) != hipSuccess) return e;
    return launch_qa_rows(a, stream);
  }
  return hipGetLastError();
}

}  // namespace fp
