// fp_sparse_attn_noalloc: the attention entry point for callers that cannot allocate device
// memory (code under graph capture, serving loops, harnesses that forbid hipMalloc).  Its
// workspace -- the work order, the queue counters and the V^T tiles of fp_sparse_attn -- is a
// fixed device array of FP_NOALLOC_SCRATCH_BYTES defined in this file, one copy per GPU, held
// from module load to process end.  Calls on one GPU share that array.
#include <mutex>

#include "fp_internal.h"

namespace fp {
namespace {

constexpr int kMaxDevices = 64;

// The scratch array.  In host code `scratch` names a host-side stand-in, not device memory:
// only the address returned by hipGetSymbolAddress for the current device is passed on.
__device__ __align__(256) unsigned char scratch[FP_NOALLOC_SCRATCH_BYTES];

std::mutex g_mu;
void *g_ptr[kMaxDevices];

}  // namespace

// Device address of the current device's scratch array, looked up once per device (with
// that device current) and kept.  No allocation.
hipError_t noalloc_scratch(void **out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_mu);
  if (g_ptr[dev] == nullptr) {
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    g_ptr[dev] = p;
  }
  *out = g_ptr[dev];
  return hipSuccess;
}

}  // namespace fp
