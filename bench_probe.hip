// Stage-mix probe for the attention kernel's roofline discussion (run by `bench.py --probe`).
//
// Runs the instruction mix of one sparse_fa_fwd<128, 128> stage -- per wave 16 K-fragment
// LDS reads and 16 MFMAs (S^T = K Q^T over 64 keys x 32 queries x d 128), the row max, 32
// exponentials with their scale FMAs, bf16 packing and row sums, then 16 V^T-fragment LDS
// reads and 16 MFMAs (O^T += V^T P^T) -- on a persistent grid of two 4-wave workgroups per
// CU (the kernel's occupancy), with none of the kernel's row logic, in seven modes:
//   mode 0  the mix alone (one LDS tile pair, no barrier, no copies);
//   mode 1  plus one workgroup barrier per stage;
//   mode 2  plus the stage copies: K and V^T tiles (16 KB each) copied global -> LDS with
//           buffer_load ... lds from an L2-resident 4 MB region, double-buffered, with the
//           kernel's wait + barrier per stage;
//   mode 3  the MFMAs and fragment reads only (no softmax work), no barrier, no copies;
//   mode 4  mode 0 with the P V product one stage behind: the previous stage's 16 PV MFMAs
//           issued one by one between this stage's exponentials (scheduling fences);
//   mode 5  mode 0 with the wave priority raised around its MFMA groups (s_setprio);
//   mode 6  the mix as a ping-pong of two 4-wave groups in one 8-wave workgroup per CU.
// Each mode reports the MFMA rate over its launches (hipEvents); the clock and the
// matrix-pipe busy fraction come from a counter pass over the same program (GRBM_GUI_ACTIVE,
// SQ_VALU_MFMA_BUSY_CYCLES).  Operands are hashed finite bf16 values
// (|v| in [0.5, 2)); results are summed into one output word per thread so that nothing is
// optimised away.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kThreads = 256;          // 4 waves
constexpr int kTile = 16384;           // bytes of one K (or V^T) stage tile: 64 keys x 128 d
constexpr int kSrcBytes = 4 << 20;     // copy source (L2-resident)

// bf16 pattern of index i: a hashed value of magnitude below 2, so that the MFMA operands
// toggle like real activations (the matrix pipes draw less power on constant operands).
__device__ __forceinline__ uint32_t hashed_bf16x2(uint32_t i) {
  uint32_t x = i * 0x9E3779B1u;
  x ^= x >> 15;
  x *= 0x85EBCA77u;
  x ^= x >> 13;
  // sign and low mantissa bits from the hash, exponent 126 or 127 (|v| in [0.5, 2))
  const uint32_t lo = (x & 0x807Fu) | (0x3F00u + ((x >> 8) & 0x80u));
  const uint32_t hi = ((x >> 16) & 0x807Fu) | (0x3F00u + ((x >> 24) & 0x80u));
  return lo | (hi << 16);
}

__global__ __launch_bounds__(256) void fill_source(uint32_t *src, int words) {
  for (int i = blockIdx.x * 256 + threadIdx.x; i < words; i += gridDim.x * 256)
    src[i] = hashed_bf16x2((uint32_t)i);
}

// grid: 2 workgroups per CU; every workgroup runs `stages` stages of the given mode.
// LDS: two stage buffers of [K tile | V^T tile] (64 KB).  Fragment addresses stay inside
// one tile: lane offset (0 .. 1008) + fragment offset (k * 1024 + 8192 * b2 <= 15360).
template <int MODE>
__global__ __launch_bounds__(kThreads) void stage_mix(int stages, const uint4 *src,
                                                      float *sink) {
  __shared__ __attribute__((aligned(1024))) uint8_t lds[4 * kTile];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  for (int i = tid; i < 4 * kTile / 4; i += kThreads)
    reinterpret_cast<uint32_t *>(lds)[i] = hashed_bf16x2(0x40000u + (uint32_t)i);
  __syncthreads();
  bf16x8 qf[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    uint32_t u[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) u[e] = hashed_bf16x2(0x80000u + 64u * (32u * k + 4u * e) + lane);
    qf[k] = __builtin_bit_cast(bf16x8, make_uint4(u[0], u[1], u[2], u[3]));
  }
  f32x16 oacc[4] = {};
  bf16x8 pprev[4] = {};
  float l_run = 0.f, m_ref = 0.f;
  const float c = 0.12751743f;          // 1/sqrt(128) * log2(e)
  const uint32_t lane_off = 16u * (uint32_t)lane;
  const __amdgpu_buffer_rsrc_t rsrc =
      __builtin_amdgcn_make_buffer_rsrc((void *)src, (short)0, kSrcBytes, 0x00020000);
  // every copy stays inside the source: src_wg + 7 * 2 * kTile + 2 * kTile <= kSrcBytes
  const uint32_t src_wg = (uint32_t)(blockIdx.x * 65536u) % (uint32_t)(kSrcBytes - 16 * kTile);
  __syncthreads();
  for (int t = 0; t < stages; ++t) {
    const int cur = (MODE == 2) ? (t & 1) : 0;
    if constexpr (MODE == 2) {
      // this wave's copies of stage t landed, every wave's too; then the copies of stage t+1
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      __builtin_amdgcn_s_barrier();
      uint8_t *dst = lds + (cur ^ 1) * 2 * kTile;
      const uint32_t so = src_wg + (uint32_t)(t & 7) * 2 * kTile;
#pragma unroll
      for (int i = 0; i < 4; ++i) {       // this wave's 4 KB of each tile
        const int slot = w * 4 + i;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(
            rsrc, (__attribute__((address_space(3))) void *)(dst + slot * 1024), 16,
            so + slot * 1024 + lane_off, 0, 0, 0);
        __builtin_amdgcn_raw_ptr_buffer_load_lds(
            rsrc, (__attribute__((address_space(3))) void *)(dst + kTile + slot * 1024), 16,
            so + kTile + slot * 1024 + lane_off, 0, 0, 0);
      }
    } else if constexpr (MODE == 1) {
      __builtin_amdgcn_s_barrier();
    }
    const uint8_t *kt = lds + cur * 2 * kTile;
    const uint8_t *vt = kt + kTile;
    // the fragment position moves with the stage so that no read is loop-invariant
    const uint32_t rot = 16u * (uint32_t)(t & 3);
    f32x16 sacc[2];
    if constexpr (MODE == 5) __builtin_amdgcn_s_setprio(1);
#pragma unroll
    for (int b2 = 0; b2 < 2; ++b2) {
      sacc[b2] = f32x16{};
      bf16x8 kf[8];
#pragma unroll
      for (int k = 0; k < 8; ++k)
        kf[k] = *reinterpret_cast<const bf16x8 *>(kt + ((lane_off ^ rot) + k * 1024 + b2 * 8192));
#pragma unroll
      for (int k = 0; k < 8; ++k)
        sacc[b2] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[k], qf[k], sacc[b2], 0, 0, 0);
    }
    if constexpr (MODE == 5) __builtin_amdgcn_s_setprio(0);
    bf16x8 pf[4];
    if constexpr (MODE == 4) {
      float mt = m_ref;
#pragma unroll
      for (int b2 = 0; b2 < 2; ++b2)
#pragma unroll
        for (int v = 0; v < 16; ++v) mt = fmaxf(mt, sacc[b2][v]);
      auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(mt), __float_as_uint(mt), false,
                                                false);
      m_ref = fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
      const float mc = m_ref * c;
      bf16x8 vf[2][4];
      auto rd = [&](int st, bf16x8 (&d)[4]) {
#pragma unroll
        for (int db = 0; db < 4; ++db)
          d[db] = *reinterpret_cast<const bf16x8 *>(vt + ((lane_off ^ rot) + db * 1024 + st * 4096));
      };
      rd(0, vf[0]);
#pragma unroll
      for (int st = 0; st < 4; ++st) {
        if (st + 1 < 4) rd(st + 1, vf[(st + 1) & 1]);
#pragma unroll
        for (int db = 0; db < 4; ++db) {
          oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[st & 1][db], pprev[st], oacc[db], 0, 0, 0);
#pragma unroll
          for (int v = 2 * db; v < 2 * db + 2; ++v)
            pf[st][v] = (__bf16)__builtin_amdgcn_exp2f(fmaf(sacc[st >> 1][8 * (st & 1) + v], c, -mc));
          __builtin_amdgcn_sched_barrier(0);
        }
      }
      const bf16x2 one = {(__bf16)1.0f, (__bf16)1.0f};
#pragma unroll
      for (int st = 0; st < 4; ++st)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const bf16x2 pair = {pf[st][2 * e], pf[st][2 * e + 1]};
          l_run = __builtin_amdgcn_fdot2_f32_bf16(pair, one, l_run, false);
        }
#pragma unroll
      for (int st = 0; st < 4; ++st) pprev[st] = pf[st];
      continue;                         // the product of this stage follows in the next one
    }
    if constexpr (MODE == 3) {
#pragma unroll
      for (int st = 0; st < 4; ++st)
#pragma unroll
        for (int v = 0; v < 8; ++v) pf[st][v] = (__bf16)sacc[st >> 1][8 * (st & 1) + v];
    } else {
      float mt = m_ref;
#pragma unroll
      for (int b2 = 0; b2 < 2; ++b2)
#pragma unroll
        for (int v = 0; v < 16; ++v) mt = fmaxf(mt, sacc[b2][v]);
      auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(mt), __float_as_uint(mt), false,
                                                false);
      m_ref = fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
      const float mc = m_ref * c;
#pragma unroll
      for (int st = 0; st < 4; ++st)
#pragma unroll
        for (int v = 0; v < 8; ++v)
          pf[st][v] =
              (__bf16)__builtin_amdgcn_exp2f(fmaf(sacc[st >> 1][8 * (st & 1) + v], c, -mc));
      const bf16x2 one = {(__bf16)1.0f, (__bf16)1.0f};
#pragma unroll
      for (int st = 0; st < 4; ++st)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const bf16x2 pair = {pf[st][2 * e], pf[st][2 * e + 1]};
          l_run = __builtin_amdgcn_fdot2_f32_bf16(pair, one, l_run, false);
        }
    }
    if constexpr (MODE == 5) __builtin_amdgcn_s_setprio(1);
#pragma unroll
    for (int st = 0; st < 4; ++st) {
      bf16x8 vf[4];
#pragma unroll
      for (int db = 0; db < 4; ++db)
        vf[db] = *reinterpret_cast<const bf16x8 *>(vt + ((lane_off ^ rot) + db * 1024 + st * 4096));
#pragma unroll
      for (int db = 0; db < 4; ++db)
        oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[db], pf[st], oacc[db], 0, 0, 0);
    }
    if constexpr (MODE == 5) __builtin_amdgcn_s_setprio(0);
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  float s = l_run + m_ref;
#pragma unroll
  for (int db = 0; db < 4; ++db)
#pragma unroll
    for (int i = 0; i < 16; ++i) s += oacc[db][i];
  sink[(size_t)blockIdx.x * kThreads + tid] = s;
}

// mode 6: one 8-wave workgroup per CU (the same two waves per SIMD); waves 0-3 and 4-7
// alternate an MFMA phase (the previous stage's P V, then this stage's Q K) and a VALU phase
// (the softmax of that stage), switched at workgroup barriers, so that the two waves of a
// SIMD are always in opposite phases.  LDS: one K tile and one V^T tile (32 KB).
__global__ __launch_bounds__(2 * kThreads) void ping_pong(int stages, float *sink) {
  __shared__ __attribute__((aligned(1024))) uint8_t lds[2 * kTile];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, grp = w >> 2;
  for (int i = tid; i < 2 * kTile / 4; i += 2 * kThreads)
    reinterpret_cast<uint32_t *>(lds)[i] = hashed_bf16x2(0x40000u + (uint32_t)i);
  __syncthreads();
  bf16x8 qf[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    uint32_t u[4];
#pragma unroll
    for (int e = 0; e < 4; ++e)
      u[e] = hashed_bf16x2(0x80000u + 64u * (32u * k + 4u * e) + lane + 4096u * w);
    qf[k] = __builtin_bit_cast(bf16x8, make_uint4(u[0], u[1], u[2], u[3]));
  }
  f32x16 oacc[4] = {};
  f32x16 sacc[2] = {};
  bf16x8 pf[4] = {};
  float l_run = 0.f, m_ref = 0.f;
  const float c = 0.12751743f;
  const uint32_t lane_off = 16u * (uint32_t)lane;
  const uint8_t *kt = lds, *vt = lds + kTile;
  auto mfma_phase = [&](int t) {
    const uint32_t rot = 16u * (uint32_t)(t & 3);
#pragma unroll
    for (int st = 0; st < 4; ++st) {
      bf16x8 vf[4];
#pragma unroll
      for (int db = 0; db < 4; ++db)
        vf[db] = *reinterpret_cast<const bf16x8 *>(vt + ((lane_off ^ rot) + db * 1024 + st * 4096));
#pragma unroll
      for (int db = 0; db < 4; ++db)
        oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[db], pf[st], oacc[db], 0, 0, 0);
    }
#pragma unroll
    for (int b2 = 0; b2 < 2; ++b2) {
      sacc[b2] = f32x16{};
      bf16x8 kf[8];
#pragma unroll
      for (int k = 0; k < 8; ++k)
        kf[k] = *reinterpret_cast<const bf16x8 *>(kt + ((lane_off ^ rot) + k * 1024 + b2 * 8192));
#pragma unroll
      for (int k = 0; k < 8; ++k)
        sacc[b2] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[k], qf[k], sacc[b2], 0, 0, 0);
    }
  };
  auto valu_phase = [&]() {
    float mt = m_ref;
#pragma unroll
    for (int b2 = 0; b2 < 2; ++b2)
#pragma unroll
      for (int v = 0; v < 16; ++v) mt = fmaxf(mt, sacc[b2][v]);
    auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(mt), __float_as_uint(mt), false,
                                              false);
    m_ref = fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
    const float mc = m_ref * c;
#pragma unroll
    for (int st = 0; st < 4; ++st)
#pragma unroll
      for (int v = 0; v < 8; ++v)
        pf[st][v] = (__bf16)__builtin_amdgcn_exp2f(fmaf(sacc[st >> 1][8 * (st & 1) + v], c, -mc));
    const bf16x2 one = {(__bf16)1.0f, (__bf16)1.0f};
#pragma unroll
    for (int st = 0; st < 4; ++st)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const bf16x2 pair = {pf[st][2 * e], pf[st][2 * e + 1]};
        l_run = __builtin_amdgcn_fdot2_f32_bf16(pair, one, l_run, false);
      }
  };
  for (int t = 0; t < stages; ++t) {
    if (grp == 0) mfma_phase(t);
    else valu_phase();
    __builtin_amdgcn_s_barrier();
    if (grp == 0) valu_phase();
    else mfma_phase(t);
    __builtin_amdgcn_s_barrier();
  }
  float s = l_run + m_ref;
#pragma unroll
  for (int db = 0; db < 4; ++db)
#pragma unroll
    for (int i = 0; i < 16; ++i) s += oacc[db][i];
  sink[(size_t)blockIdx.x * 2 * kThreads + tid] = s;
}

bool check(hipError_t e, const char *what) {
  if (e != hipSuccess) {
    fprintf(stderr, "%s: %s\n", what, hipGetErrorString(e));
    return false;
  }
  return true;
}

template <int MODE>
bool run_mode(int nblk, int stages, const uint4 *src, float *d_sink,
              const char *name, bool last) {
  hipEvent_t e0, e1;
  if (!check(hipEventCreate(&e0), "event") || !check(hipEventCreate(&e1), "event")) return false;
  hipLaunchKernelGGL(stage_mix<MODE>, dim3(nblk), dim3(kThreads), 0, 0, 16, src, d_sink);
  if (!check(hipDeviceSynchronize(), "warm-up launch")) return false;
  constexpr int kReps = 3;
  if (!check(hipEventRecord(e0, 0), "event")) return false;
  for (int r = 0; r < kReps; ++r)
    hipLaunchKernelGGL(stage_mix<MODE>, dim3(nblk), dim3(kThreads), 0, 0, stages, src, d_sink);
  if (!check(hipEventRecord(e1, 0), "event")) return false;
  if (!check(hipEventSynchronize(e1), "timed launches")) return false;
  float ms = 0.f;
  if (!check(hipEventElapsedTime(&ms, e0, e1), "event")) return false;
  ms /= kReps;
  const double flop = (double)nblk * 4 * 32 * 32768.0 * stages;
  printf("    {\"mode\": %d, \"what\": \"%s\", \"ms\": %.3f, \"tflops\": %.1f}%s\n", MODE,
         name, ms, flop / (ms * 1e-3) / 1e12, last ? "" : ",");
  return check(hipEventDestroy(e0), "event") && check(hipEventDestroy(e1), "event");
}

bool run_ping_pong(int cus, int stages, float *d_sink) {
  hipEvent_t e0, e1;
  if (!check(hipEventCreate(&e0), "event") || !check(hipEventCreate(&e1), "event")) return false;
  hipLaunchKernelGGL(ping_pong, dim3(cus), dim3(2 * kThreads), 0, 0, 16, d_sink);
  if (!check(hipDeviceSynchronize(), "warm-up launch")) return false;
  constexpr int kReps = 3;
  if (!check(hipEventRecord(e0, 0), "event")) return false;
  for (int r = 0; r < kReps; ++r)
    hipLaunchKernelGGL(ping_pong, dim3(cus), dim3(2 * kThreads), 0, 0, stages, d_sink);
  if (!check(hipEventRecord(e1, 0), "event")) return false;
  if (!check(hipEventSynchronize(e1), "timed launches")) return false;
  float ms = 0.f;
  if (!check(hipEventElapsedTime(&ms, e0, e1), "event")) return false;
  ms /= kReps;
  const double flop = (double)cus * 8 * 32 * 32768.0 * stages;
  printf("    {\"mode\": 6, \"what\": \"ping-pong of two 4-wave groups\", \"ms\": %.3f, "
         "\"tflops\": %.1f}\n", ms, flop / (ms * 1e-3) / 1e12);
  return check(hipEventDestroy(e0), "event") && check(hipEventDestroy(e1), "event");
}

}  // namespace

int main(int argc, char **argv) {
  int cus = 0;
  if (!check(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, 0), "device"))
    return 1;
  const int nblk = 2 * cus;               // two 4-wave workgroups per CU, all resident
  const int stages = argc > 1 ? atoi(argv[1]) : 50000;
  if (stages < 1 || stages > 1000000) {
    fprintf(stderr, "stages out of range\n");
    return 1;
  }
  uint4 *src = nullptr;
  float *d_sink = nullptr;
  if (!check(hipMalloc(&src, kSrcBytes), "alloc") ||
      !check(hipMalloc(&d_sink, (size_t)nblk * kThreads * 4), "alloc"))
    return 1;
  hipLaunchKernelGGL(fill_source, dim3(1024), dim3(256), 0, 0, (uint32_t *)src, kSrcBytes / 4);
  if (!check(hipDeviceSynchronize(), "fill")) return 1;
  printf("{\"probe\": \"sparse_fa_fwd<128, 128> stage mix\", \"workgroups\": %d, "
         "\"stages_per_workgroup\": %d, \"modes\": [\n", nblk, stages);
  bool ok = run_mode<0>(nblk, stages, src, d_sink, "stage mix alone", false) &&
            run_mode<1>(nblk, stages, src, d_sink, "+ barrier per stage", false) &&
            run_mode<2>(nblk, stages, src, d_sink, "+ K/V stage copies, wait, barrier",
                        false) &&
            run_mode<3>(nblk, stages, src, d_sink, "MFMAs and fragment reads only", false) &&
            run_mode<4>(nblk, stages, src, d_sink, "PV of previous stage between exps", false) &&
            run_mode<5>(nblk, stages, src, d_sink, "mix with setprio around MFMAs", false) &&
            run_ping_pong(cus, stages, d_sink);
  printf("]}\n");
  ok = check(hipFree(src), "free") && check(hipFree(d_sink), "free") && ok;
  return ok ? 0 : 1;
}
