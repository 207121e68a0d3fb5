// Device execution tables of a chunk-scheduled GEMM, built on the host from the
// chunk-ordered tile list: the work units in execution order (one sub-list per die),
// each unit's chunk list, and the chunk copy items of the kernel copy backend. Plans
// upload them to memory they own; the allocation-free entry point writes them into the
// library's static scratch.
#pragma once

#include <cstdint>
#include <vector>

#include "kernels.hpp"
#include "planner.hpp"

namespace csg {

struct ExecOptions {
  bool consumer = true;     // AG / grouped (units wait for remote chunks) vs producer (units signal chunks)
  int64_t K = 0;
  int64_t in_bytes = 2;     // bytes per element of A
  int32_t bk = 64;
  int32_t split_k = 1;      // K-slices of every tile
  int32_t tail_split = 0;   // K-slices of the tiles on the critical path (0/1: none)
  int32_t tail_chunks = 0;  // ... those reading one of the last (consumers) / first (producer) chunks
  int32_t tail_taper = 0;   // 1: the tail split tapers from tail_split (the last / first chunk) to 1
  int32_t tile_dispatch = 0;  // 2: one plain list (dealt statically, die-major), else per-die sub-lists
  int32_t grid = 0;         // persistent workgroups (round-robin over the dies)
  int32_t tail_wave = 0;    // > 1: K-slices (at most) for each die's last partial wave of tiles
};

struct ExecTables {
  std::vector<TileDesc> units;       // execution order
  std::vector<int32_t> list_ptr;     // [units + 1]
  std::vector<int32_t> list_ids;     // consumers: remote chunks a unit waits for; producer: chunks it writes
  std::vector<int32_t> raster;       // raster id per unit
  std::vector<int32_t> need;         // per chunk: units reading it (consumers) / tiles writing it (producer)
  std::vector<int32_t> list_begin;   // [kXcdLists + 1]: die x runs units [list_begin[x], list_begin[x + 1])
  int32_t ws_slices = 0;             // partial-sum buffers of split tiles
  int32_t tail_begin = 0;            // static dispatch, consumers: first unit of the trailing
                                     // critical tiles, dealt from a shared ticket (0: none)
  bool lines_aligned = true;         // every chunk of A starts on a 128-byte line
};

// Execution tables of a tile map. A tile goes to die (row-tile index mod kXcdLists),
// so tiles sharing A rows share an L2; every sub-list keeps the chunk order.
void build_exec_tables(const Schedule& s, const TileMap& m, const ExecOptions& o, ExecTables* out);

// Copy items of the kernel copy backend: every chunk of `moved` (chunk ids, in the
// order the copy workgroups move them) cut into slabs of at most `slab` bytes of
// rows of `row_bytes`; parts[i] = the items of moved[i].
void build_copy_items(const Schedule& s, const std::vector<int32_t>& moved, int64_t row_bytes, int64_t slab,
                      std::vector<CopyItem>* items, std::vector<int32_t>* parts);

}  // namespace csg
