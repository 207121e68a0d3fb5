// Two small kernels that serve measurement and stream ordering, outside the GEMM:
//
//   chunk_join   waits (bounded) until the completion values of a list of copies read
//                0, so work queued behind it on its stream follows those copies on the
//                device (csg_plan_join);
//   mfma_peak    every SIMD of every CU issues independent v_mfma_f32_32x32x16_bf16
//                back to back on register operands: the bf16 matrix rate the chip
//                sustains under that load, and the shader clock it runs at
//                (csg_measure_mfma_peak).
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include "kernels.hpp"

namespace csg {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef unsigned short u16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kJoinThreads = 256;

// Thread t polls values t, t + 256, ..., each about every 20 ns for at most
// timeout_ticks (100 MHz wall clock); a value still not 0 then sets *timed_out and
// the thread moves on. A completion value sits in memory that a load reaches with
// over a microsecond of latency, so the threads' loads overlap instead of queueing
// behind one another. No barrier: every thread ends on its own, and so the kernel.
__global__ __launch_bounds__(kJoinThreads) void chunk_join(const int64_t* const* values, int32_t n,
                                                           uint64_t timeout_ticks, uint32_t* timed_out) {
  for (int32_t i = static_cast<int32_t>(threadIdx.x); i < n; i += kJoinThreads) {
    const int64_t* p = values[i];
    const uint64_t t0 = wall_clock64();
    while (__hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM) != 0) {
      if (wall_clock64() - t0 > timeout_ticks) {
        __hip_atomic_store(timed_out, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
        break;
      }
      __builtin_amdgcn_s_sleep(1);
    }
  }
}

hipError_t launch_join(const int64_t* const* values, int32_t n, uint64_t timeout_ticks, uint32_t* timed_out,
                       hipStream_t stream) {
  hipLaunchKernelGGL(chunk_join, dim3(1), dim3(kJoinThreads), 0, stream, values, n, timeout_ticks, timed_out);
  return hipGetLastError();
}

// A bf16 value of magnitude 2^-7 .. 2^-5 with a pseudo-random sign and mantissa, from a
// 32-bit hash: operands that toggle like N(0, 0.02) data, not constants.
__device__ __forceinline__ unsigned short hashed_bf16(uint32_t x) {
  x ^= x >> 16;
  x *= 0x7feb352dU;
  x ^= x >> 15;
  x *= 0x846ca68bU;
  x ^= x >> 16;
  const uint32_t sign = (x >> 31) & 1u;
  const uint32_t expo = 120u + ((x >> 7) % 3u);  // biased exponent: 2^-7 .. 2^-5
  return static_cast<unsigned short>((sign << 15) | (expo << 7) | (x & 0x7fu));
}

// 4 waves per workgroup, one workgroup per CU: one wave per SIMD. Each wave keeps 8
// independent accumulators, so an MFMA never waits for the previous one's result.
// Wave 0 of workgroup 0 records the shader cycles and the wall-clock ticks of its loop.
constexpr int kPeakAcc = 8;
__global__ __launch_bounds__(256) void mfma_peak(int32_t iters, float* sink, uint64_t* clocks) {
  const uint32_t tid = blockIdx.x * blockDim.x + threadIdx.x;
  u16x8 ra, rb;
  for (int e = 0; e < 8; ++e) {
    ra[e] = hashed_bf16(tid * 16u + e);
    rb[e] = hashed_bf16(tid * 16u + 8u + e + 0x9e3779b9u);
  }
  const bf16x8 a = __builtin_bit_cast(bf16x8, ra), b = __builtin_bit_cast(bf16x8, rb);
  f32x16 acc[kPeakAcc];
  for (int i = 0; i < kPeakAcc; ++i) acc[i] = f32x16{};
  const uint64_t c0 = clock64(), w0 = wall_clock64();
  for (int32_t it = 0; it < iters; ++it) {
#pragma unroll
    for (int i = 0; i < kPeakAcc; ++i) acc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[i], 0, 0, 0);
  }
  const uint64_t c1 = clock64(), w1 = wall_clock64();
  float s = 0.0f;
  for (int i = 0; i < kPeakAcc; ++i)
    for (int e = 0; e < 16; ++e) s += acc[i][e];
  if (s == 12345.678f) sink[tid] = s;  // keeps the products live; never true in practice
  if (tid == 0) {
    clocks[0] = c1 - c0;
    clocks[1] = w1 - w0;
  }
}

hipError_t launch_mfma_peak(int32_t grid, int32_t iters, float* sink, uint64_t* clocks, hipStream_t stream,
                            hipEvent_t start, hipEvent_t stop) {
  hipExtLaunchKernelGGL(mfma_peak, dim3(grid), dim3(256), 0, stream, start, stop, 0, iters, sink, clocks);
  return hipGetLastError();
}

// Flops of one mfma_peak launch.
double mfma_peak_flops(int32_t grid, int32_t iters) {
  return 2.0 * 32 * 32 * 16 * 4.0 * kPeakAcc * static_cast<double>(grid) * static_cast<double>(iters);
}

}  // namespace csg
