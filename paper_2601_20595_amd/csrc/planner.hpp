// Host planner: chunk schedules, the chunk-tile dependence map and the
// chunk-ordered tile list. Pure C++ (no HIP), so it runs on any host.
//
// Schedules follow the paper's communication-schedule abstraction (Section 5.1):
// chunks are logical row blocks moved as units; one rank's schedule is an
// ordered list of chunk operations, instantiated from parameterised templates.
// The map follows Section 5.2 (dependency parsing): a tile depends on the chunks
// its rows read (consumer ops) or write (producer op); the tile list follows the
// tile-scheduler swizzle: chunks in communication order, and inside a chunk the
// local kernel's raster order or a band-by-band column order.
#pragma once

#include <cstdint>
#include <string>
#include <vector>

namespace csg {

struct ChunkDesc {
  int64_t row_begin;
  int64_t row_end;
  int32_t src_rank;
  int32_t group;
  int32_t is_local;
};

struct Schedule {
  std::vector<ChunkDesc> chunks;  // in row order
  std::vector<int32_t> order;     // arrival / emission order (chunk ids)
  int64_t total_rows = 0;
};

enum class OrderKind : int32_t { Ring = 0, Swizzle1D = 1, Permutation = 2, RsRing = 3 };

// Returns "" on success, else a description of the violated rule.
std::string validate_schedule(const std::vector<ChunkDesc>& chunks, const std::vector<int32_t>& order);

std::string make_uniform_schedule(int32_t world, int32_t rank, int64_t shard_rows, int32_t chunks_per_shard,
                                  OrderKind kind, const int32_t* remote_perm, Schedule* out);

std::string make_grouped_schedule(int32_t world, int32_t rank, int32_t n_groups, const int64_t* counts,
                                  Schedule* out);

// One row of output tiles: rows [row_begin, row_end) of group `group`.
struct RowTile {
  int64_t row_begin;
  int64_t row_end;
  int32_t group;
};

struct TileMap {
  int32_t n_tiles_n = 0;
  std::vector<RowTile> row_tiles;
  // D(t) per raster tile id and its inverse T(c); both lists ascending.
  std::vector<int32_t> tile_ptr, tile_chunks;
  std::vector<int32_t> chunk_ptr, chunk_tiles;
  std::vector<int32_t> order;  // raster ids in execution order
  int32_t n_tiles() const { return static_cast<int32_t>(tile_ptr.size()) - 1; }
};

// producer = true selects the emission key (earliest chunk written), false the
// arrival key (latest chunk read). group_rows empty = one group spanning M.
// Inside a key, intra_order 0 keeps the raster order; 1 cuts the key's row tiles
// (ascending) into bands of group_m and visits each band column by column
// (Section 5.2, intra-chunk swizzle): order = (key, band, n, m).
std::string build_tile_map(const Schedule& s, int64_t M, int64_t N, int32_t bm, int32_t bn, bool producer,
                           const std::vector<int64_t>& group_rows, TileMap* out, int32_t intra_order = 0,
                           int32_t group_m = 8);

}  // namespace csg
