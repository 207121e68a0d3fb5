// Interface between the host runtime and the ring-attention kernel.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "kernels.hpp"

namespace csg {

constexpr int kAttnHeadDim = 128;  // head dimension the kernel is built for
constexpr int kAttnBlockQ = 128;   // query rows per work unit
constexpr int kAttnBlockKV = 64;   // key rows per inner step (chunks are multiples of it)

struct AttnArgs {
  const uint16_t* Q;          // [Sq][H][D] bf16
  const uint16_t* K;          // [S][Hkv][D] bf16, the landing buffer
  const uint16_t* V;          // [S][Hkv][D] bf16, the landing buffer
  uint16_t* O;                // [Sq][H][D] bf16
  float* LSE;                 // [H][Sq] natural-log log-sum-exp of the scaled scores
  int32_t Sq, H, Hkv;
  int32_t n_units;            // work units: ceil(Sq / kAttnBlockQ) * H
  int32_t n_chunks;
  const int32_t* arrival;     // [n_chunks]: chunk id at each arrival position
  const int32_t* chunk_rows;  // [2 * n_chunks] by chunk id: key row begin, end
  const int64_t* const* ready;  // per chunk id: 0 once its keys and values have landed
  uint32_t* counters;         // per chunk id: units done reading it
  uint32_t* out_flags;        // per chunk id: the call number once every unit has read it
  uint32_t* ticket;           // [kXcdLists] work-unit tickets, one per die's range of units
  DeviceDiag* diag;
  uint64_t timeout_ticks;
  uint32_t epoch;
  float scale_log2;           // softmax scale times log2(e)
  // the next call's state set, cleared by workgroup 0 at the start (null: not here)
  uint32_t* next_ticket;
  uint32_t* next_counters;
  DeviceDiag* next_diag;
};

int32_t attn_threads();
hipError_t launch_ring_attn(const AttnArgs& args, int32_t grid, hipStream_t stream, hipEvent_t start, hipEvent_t stop);
// Co-resident workgroups of the attention kernel on `device`.
hipError_t attn_grid(int device, int32_t* grid);

}  // namespace csg
