// Bitonic sort of 64-bit keys held in registers across a workgroup (device code only;
// included by the HIP sources).
#pragma once
#include <hip/hip_runtime.h>

namespace fp {

// One side of a compare-exchange: the partner's key v if (v < u) == take_min, else the own
// key u -- min(u, v) when take_min, max(u, v) otherwise (equal keys: either is the value).
// One 64-bit compare and two selects per key.
__device__ __forceinline__ unsigned long long key_keep(unsigned long long u,
                                                       unsigned long long v, bool take_min) {
  return ((v < u) == take_min) ? v : u;
}

// The value of lane l ^ LX (LX < 64): DPP moves inside quads and rows, a swizzle inside
// 32-lane groups, a permute across the halves.
template <int LX>
__device__ __forceinline__ unsigned lane_xor32(unsigned x) {
  if constexpr (LX == 1) return (unsigned)__builtin_amdgcn_mov_dpp((int)x, 0xB1, 0xF, 0xF, false);
  else if constexpr (LX == 2) return (unsigned)__builtin_amdgcn_mov_dpp((int)x, 0x4E, 0xF, 0xF, false);
  else if constexpr (LX == 8) return (unsigned)__builtin_amdgcn_mov_dpp((int)x, 0x128, 0xF, 0xF, false);
  else if constexpr (LX == 4 || LX == 16) return (unsigned)__builtin_amdgcn_ds_swizzle((int)x, 0x1F | (LX << 10));
  else return (unsigned)__shfl_xor((int)x, LX);
}
template <int LX>
__device__ __forceinline__ unsigned long long lane_xor(unsigned long long x) {
  const unsigned lo = lane_xor32<LX>((unsigned)x), hi = lane_xor32<LX>((unsigned)(x >> 32));
  return ((unsigned long long)hi << 32) | lo;
}

// One compare-exchange stage (SIZE, STRIDE) of an ascending bitonic sort of NT*E keys,
// thread t holding positions t*E .. t*E+E-1 in k[].  Strides below E pair keys of one
// thread, strides below 64*E pair lanes of one wave, wider strides go through `lds`
// (NT*E keys, used as scratch).
template <int NT, int E, int SIZE, int STRIDE>
__device__ __forceinline__ void bitonic_stage(unsigned long long (&k)[E],
                                              unsigned long long *lds, int tid) {
  if constexpr (STRIDE < E) {
#pragma unroll
    for (int e = 0; e < E; ++e) {
      if ((e & STRIDE) == 0) {
        const int f = e | STRIDE;
        const bool up = ((tid * E + e) & SIZE) == 0;
        const unsigned long long u = k[e], v = k[f];
        const bool sw = (v < u) == up;     // out of order for this half (equal: no matter)
        k[e] = sw ? v : u;
        k[f] = sw ? u : v;
      }
    }
  } else if constexpr (STRIDE < 64 * E) {
    constexpr int LX = STRIDE / E;
    const bool take_min = ((tid & LX) == 0) == (((tid * E) & SIZE) == 0);
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const unsigned long long v = lane_xor<LX>(k[e]);
      k[e] = key_keep(k[e], v, take_min);
    }
  } else {
    // Position tid * E + e pairs with (tid ^ TX) * E + e.  The exchange is stored
    // element-major (key e of thread t at e * NT + t), so that the lanes of a wave touch
    // consecutive words (thread-major order would put adjacent lanes E words apart, all in
    // the same few LDS banks).
    constexpr int TX = STRIDE / E;
    __syncthreads();                 // the previous LDS stage's reads are done
#pragma unroll
    for (int e = 0; e < E; ++e) lds[e * NT + tid] = k[e];
    __syncthreads();
    const bool take_min = (((tid * E) & STRIDE) == 0) == (((tid * E) & SIZE) == 0);
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const unsigned long long v = lds[e * NT + (tid ^ TX)];
      k[e] = key_keep(k[e], v, take_min);
    }
  }
  if constexpr (STRIDE > 1) bitonic_stage<NT, E, SIZE, STRIDE / 2>(k, lds, tid);
}

// Whole sort: k[] ascending over the workgroup in thread-major order on return.
template <int NT, int E, int SIZE = 2>
__device__ __forceinline__ void bitonic_sort(unsigned long long (&k)[E],
                                             unsigned long long *lds, int tid) {
  bitonic_stage<NT, E, SIZE, SIZE / 2>(k, lds, tid);
  if constexpr (SIZE < NT * E) bitonic_sort<NT, E, SIZE * 2>(k, lds, tid);
}

}  // namespace fp
