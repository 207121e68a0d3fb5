// The library's static device scratch, used by the allocation-free entry point
// (csg_ag_gemm_noalloc) for its tables and per-call state.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>

namespace csg {

// Size of the scratch array every device holds (from the library's load until the
// process ends).
constexpr size_t kNoAllocScratchBytes = size_t{2} << 20;

// Device address of `device`'s copy of the scratch array: looked up once per device
// (hipGetSymbolAddress with that device current; the caller makes it current) and
// kept. Thread-safe.
hipError_t noalloc_scratch(int device, void** ptr);

}  // namespace csg
