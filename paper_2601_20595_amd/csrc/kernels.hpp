// Interface between the host runtime and the HIP kernels of the chunk-scheduled GEMM.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace csg {

// Written by the kernel when a bounded flag wait gives up; read back by csg_plan_check.
struct DeviceDiag {
  uint32_t timed_out;
  int32_t chunk;
  int32_t tile;
  uint32_t observed;
  uint32_t epoch;
  uint32_t abort;     // set once any workgroup gave up; the others stop taking tiles
  uint32_t units_done;  // work units executed, summed over workgroups as they exit
  uint32_t pad;
};

// One entry of the execution-ordered tile list.
// One work unit of the execution list: a tile, or one K-slice of a tile split along K.
struct TileDesc {
  int32_t row_begin;  // first output row (global)
  int32_t row_end;    // one past the last valid output row
  int32_t n_tile;     // tile index along N
  int32_t group;      // expert index (grouped GEMM), else 0
  int32_t kt_begin;   // first K step (units of the tile's BK)
  int32_t kt_end;     // one past the last K step
  int32_t slot;       // split tiles: workspace index of the tile's first slice (its slices are
                      // consecutive); -1 if not split
  int32_t slice;      // split tiles: slice index | (number of slices << 16)
};

// One slab of a chunk moved by the kernel's copy workgroups: bytes [off, off + bytes)
// of the copy source, written to the same offsets of the destination.
struct CopyItem {
  int64_t off;
  int32_t bytes;  // a multiple of 4
  int32_t rpos;   // position of the chunk among the remote chunks (arrival / emission order)
};

// Per-call state of the copy workgroups, set by the prologue.
struct CopyState {
  uint64_t t0;  // wall clock (100 MHz) when the call's prologue ran; release times count from it
};

struct GemmArgs {
  const void* A;             // rows of A (AG: landing buffer; grouped: routed X), K contiguous
  const void* B;             // N x K, or E x N x K
  void* C;                   // M x N
  int64_t M, N, K;
  int64_t b_group_stride;    // elements between consecutive experts' weights
  const TileDesc* tiles;     // [n_tiles] in execution order
  const int32_t* list_ptr;   // [n_tiles + 1]: per execution position, its chunks
  const int32_t* list_ids;   // consumer: remote chunks to wait for; producer: chunks written
  const int32_t* raster;     // [n_tiles] raster id per execution position (diagnostics)
  const int64_t* const* ready;  // per chunk, the value a copy engine brings to 0: consumers,
                                // once the chunk has landed; producer, once the previous call's
                                // copy out of the chunk has completed (local chunks: a 0)
  uint32_t* counters;        // per chunk: producer: tiles written; consumers: units done reading it
  const int32_t* need;       // per chunk: the count at which the chunk is complete
  uint32_t* out_flags;       // per chunk, host-visible memory, set to epoch when complete:
                             // producer: output rows written; consumers: rows read
  uint32_t* ticket;          // [kXcdLists] tickets, one per tile sub-list
  const int32_t* list_begin; // [kXcdLists + 1]: sub-list x is positions [list_begin[x], list_begin[x+1])
  DeviceDiag* diag;
  float* ws;                 // split-K partial sums: [slice buffer][BM * BN] fp32, thread-major
  uint32_t* slot_count;      // split-K: finished slices per tile (by raster id)
  uint64_t timeout_ticks;    // bound of one flag wait, in 100 MHz wall-clock ticks
  uint32_t epoch;            // call number: the value the producer's emitted flags take
  int32_t n_tiles;
  int32_t n_chunks;
  int32_t dynamic_ticket;
  // Static dispatch: positions tail_begin .. n_tiles - 1 (the units of the tiles on the
  // critical path, which end the list) are taken in order from ticket[0] by whichever
  // workgroup is free first, instead of by a fixed workgroup. 0: every position static.
  int32_t tail_begin;
  // Consumers: 1 if a cache line of A may hold rows of two chunks (a chunk boundary
  // or the buffer start not on a 128-byte line), so a line cached while one chunk was
  // ready could hold stale rows of the next; then a workgroup drops its caches when
  // it first sees a chunk ready. With line-aligned chunks no line of a chunk is read
  // before its flag, and lines cached by earlier work are dropped at kernel launch.
  int32_t acquire_fresh;
  // Consumers: tiles along N (> 0: a workgroup that sees a chunk land first warms its
  // share, 1 / n_tiles_n, of the tile's A rows; 0: off).
  int32_t n_tiles_n;
  // 1: a workgroup whose die's sub-list is exhausted takes entries of other dies'
  // lists. 0: every entry runs on its own die. The slices of a split tile exchange
  // partial sums through memory either way (written through, read past the caches),
  // so they may run on any die and need no L2 maintenance.
  int32_t steal;
  // Optional (nullptr = off): per execution position, kTraceWords words written by
  // the workgroup that ran it: wall-clock ticks (100 MHz) when it took the position,
  // when its waits were over, when it finished, (die << 32 | workgroup id), and the
  // shader-clock counter when its waits were over and when it finished.
  uint64_t* trace;
  // Chunk moves done by the kernel itself (Section 5.2, load/store realizations)
  // instead of the copy engines; all zero / null when the engines move the chunks.
  // Copy workgroups: workgroups 0 .. copy_wgs - 1 move the copy items (in arrival
  // order, item i by workgroup i mod copy_wgs), then join the tile list.
  const CopyItem* copy_items;
  int32_t n_copy_items;      // 0: no copy workgroups in this launch
  int32_t copy_wgs;
  const unsigned char* copy_src;
  unsigned char* copy_dst;
  const int32_t* copy_chunk;     // per remote position: chunk id
  const int32_t* copy_parts;     // per remote position: its copy items
  uint32_t* copy_done;           // per remote position: items finished (cleared by the prologue)
  int64_t* copy_ready;           // per chunk: ready word, set to 0 once the chunk's last item is done
  CopyState* copy_state;
  const uint64_t* release_ticks; // per remote position: earliest start after t0, 100 MHz ticks (null: none)
  // Producer: output rows of a chunk that is sent are also stored here (same layout
  // as C) by the tile epilogue; null when the copy engines send them.
  void* C2;
  const int32_t* chunk_sent;     // per chunk: 1 if it is sent (producer with C2)
  // GEMM + all-reduce (producer kernels built with the reduction): a tile of the own
  // shard adds the other ranks' partial sums of its rows to its accumulators before
  // storing, once they have landed.
  const unsigned char* partials;        // [n_peers][own_rows][N], C's element type
  const int64_t* const* partial_ready;  // [n_peers * (own_rows / own_chunk_rows)]: 0 once landed
  int64_t own_row0;                     // first row of the own shard
  int64_t own_rows;
  int32_t n_peers;
  int32_t own_chunk_rows;
  int32_t own_shard;                    // shard index of the own shard (diagnostics)
  // Per-call state comes in two sets, by call parity. The kernel of one call clears the
  // set the next call uses (workgroup 0, at its start: the call before, which used that
  // set, has finished), so a call whose predecessor ran such a kernel needs no prologue
  // kernel. Null when the next call's prologue clears it instead.
  uint32_t* next_ticket;
  uint32_t* next_counters;
  uint32_t* next_slot_count;
  DeviceDiag* next_diag;
  int32_t next_n_slots;
};

// Everything the per-call prologue resets.
struct PrologueArgs {
  uint32_t* counters;
  int32_t n_chunks;
  uint32_t epoch;
  uint32_t* ticket;
  DeviceDiag* diag;
  uint32_t* slot_count;   // split-K slot counts (null: none)
  int32_t n_slots;
  int64_t* ready_words;   // kernel-moved chunks: per chunk ready word, set to ready_value (null: none)
  int64_t ready_value;    // 1 = not landed yet, 0 = ready
  uint32_t* copy_done;    // per remote position, cleared
  int32_t n_remote;
  CopyState* copy_state;  // its t0 set to the prologue's wall clock
};

constexpr int kTraceWords = 6;

enum class InType : int32_t { BF16 = 0, F32 = 1 };

// The tile list is split into one sub-list per XCD (accelerator complex die, each
// with its own L2); a workgroup takes tiles from the sub-list of the die it runs on
// and steals from the others once its own is exhausted.
constexpr int kXcdLists = 8;

struct KernelKey {
  InType in;
  bool out_bf16;
  bool producer;
  int32_t bm, bn, bk;
  bool reduce = false;  // producer with the all-reduce's fused reduction
};

// Kernel variants compiled into this library; false if `key` has none.
bool kernel_supported(const KernelKey& key);
// Largest chunk count the per-workgroup ready cache holds.
int32_t kernel_max_chunks();
// Persistent grid size: co-resident workgroups on the device.
hipError_t kernel_grid(const KernelKey& key, int device, int32_t* grid);
// start/stop (may be null) receive the kernel's own start and end timestamps
hipError_t launch_chunk_gemm(const KernelKey& key, const GemmArgs& args, int32_t grid, hipStream_t stream,
                             hipEvent_t start, hipEvent_t stop);

// One thread waits until each of the n values reads 0 (the completion values of
// copies), at most timeout_ticks (100 MHz) per value; *timed_out is set to 1 if one did
// not. Work queued behind it on `stream` then follows those copies.
hipError_t launch_join(const int64_t* const* values, int32_t n, uint64_t timeout_ticks, uint32_t* timed_out,
                       hipStream_t stream);
// MFMA microbenchmark: `grid` workgroups of 4 waves, each wave `iters` rounds of 8
// independent bf16 32x32x16 MFMAs. clocks[0] = shader cycles, clocks[1] = 100 MHz
// ticks of workgroup 0's loop. start/stop receive the dispatch's timestamps.
hipError_t launch_mfma_peak(int32_t grid, int32_t iters, float* sink, uint64_t* clocks, hipStream_t stream,
                            hipEvent_t start, hipEvent_t stop);
double mfma_peak_flops(int32_t grid, int32_t iters);

// Per-call set-up on the compute stream: clears the per-chunk counters, the
// tickets, the split-K slot counts, the diagnostics and the copy workgroups' state,
// and sets the ready words of kernel-moved chunks.
hipError_t launch_prologue(const PrologueArgs& args, hipStream_t stream);

}  // namespace csg
