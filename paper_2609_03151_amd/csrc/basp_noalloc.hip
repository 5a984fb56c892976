// basp_noalloc.hip -- the device scratch buffer behind basp_attn_bwd_noalloc.
//
// The backward needs device memory beyond its inputs and outputs: the
// per-row (LSE, D) pairs and, for long sequences, the per-chunk partial sums
// of dK and dV.  basp_attn_bwd takes that workspace from the caller; callers
// that cannot allocate (code under stream capture, allocation-free serving
// loops) use this fixed file-scope array instead.  Each GPU the library runs
// on holds its own copy of the array, from the first call on that GPU until
// the process ends.  In host code the array's name only stands for the
// symbol: its device address, per device, comes from hipGetSymbolAddress with
// that device current, and only that address is handed to kernels.
#include <hip/hip_runtime.h>

#include <mutex>

#include "../../include/basp.h"
#include "basp_internal.hpp"

static __device__ __align__(256) unsigned char scratch[BASP_NOALLOC_SCRATCH_BYTES];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_mu;
void *g_scratch[kMaxDevices];  // device address of `scratch`, per device
}  // namespace

namespace basp {

hipError_t noalloc_scratch(hipStream_t stream, void **ptr) {
  int dev = 0;
  hipError_t e = stream ? hipStreamGetDevice(stream, &dev) : hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_scratch[dev]) {
    int cur = 0;
    if ((e = hipGetDevice(&cur)) != hipSuccess) return e;
    if (cur != dev && (e = hipSetDevice(dev)) != hipSuccess) return e;
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (cur != dev) {
      const hipError_t e2 = hipSetDevice(cur);
      if (e == hipSuccess) e = e2;
    }
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch[dev] = p;
  }
  *ptr = g_scratch[dev];
  return hipSuccess;
}

}  // namespace basp
