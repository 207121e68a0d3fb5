// The static device scratch of the allocation-free entry point (csg_ag_gemm_noalloc).
//
// `scratch` is a file-scope device array: every device the library runs on holds its own
// copy at its own address. Host code never passes the array's name to a kernel or a
// copy (in host code the name is a host-side stand-in); it looks up each device's
// address once, with that device current, and uses that address everywhere.
#include <hip/hip_runtime.h>

#include <mutex>

#include "noalloc.hpp"

namespace csg {
namespace {

static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_ptr[kMaxDevices] = {};

}  // namespace

hipError_t noalloc_scratch(int device, void** ptr) {
  if (device < 0 || device >= kMaxDevices || !ptr) return hipErrorInvalidValue;
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_ptr[device]) {
    int cur = -1;
    hipError_t e = hipGetDevice(&cur);
    if (e != hipSuccess) return e;
    if (cur != device) return hipErrorInvalidDevice;  // the caller makes the device current
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_ptr[device] = p;
  }
  *ptr = g_ptr[device];
  return hipSuccess;
}

}  // namespace csg
