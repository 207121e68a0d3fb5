// Host planner (see planner.hpp).
#include "planner.hpp"

#include <algorithm>
#include <numeric>
#include <tuple>
#include <utility>

namespace csg {

std::string validate_schedule(const std::vector<ChunkDesc>& chunks, const std::vector<int32_t>& order) {
  if (chunks.empty()) return "schedule has no chunks";
  if (order.size() != chunks.size()) return "order length differs from the number of chunks";
  int64_t pos = 0;
  for (size_t i = 0; i < chunks.size(); ++i) {
    const ChunkDesc& c = chunks[i];
    if (c.row_begin != pos) return "chunk " + std::to_string(i) + " leaves a gap or overlaps its predecessor";
    if (c.row_end <= c.row_begin) return "chunk " + std::to_string(i) + " is empty";
    if (c.group < 0) return "chunk " + std::to_string(i) + " has a negative group";
    pos = c.row_end;
  }
  std::vector<char> seen(chunks.size(), 0);
  for (int32_t o : order) {
    if (o < 0 || static_cast<size_t>(o) >= chunks.size() || seen[o]) return "order is not a permutation of the chunk ids";
    seen[o] = 1;
  }
  return "";
}

static void append_shard(std::vector<int32_t>& order, int32_t s, int32_t Q) {
  for (int32_t q = 0; q < Q; ++q) order.push_back(s * Q + q);
}

std::string make_uniform_schedule(int32_t world, int32_t rank, int64_t shard_rows, int32_t chunks_per_shard,
                                  OrderKind kind, const int32_t* remote_perm, Schedule* out) {
  if (world < 1 || rank < 0 || rank >= world) return "rank must lie in [0, world)";
  if (shard_rows < 1 || chunks_per_shard < 1) return "shard rows and chunks per shard must be positive";
  if (shard_rows % chunks_per_shard) return "shard rows must be divisible by chunks per shard";
  if (static_cast<int64_t>(world) * chunks_per_shard > (1 << 20)) return "too many chunks";
  const int32_t Q = chunks_per_shard;
  const int64_t h = shard_rows / Q;
  Schedule s;
  for (int32_t r = 0; r < world; ++r)
    for (int32_t q = 0; q < Q; ++q) {
      const int64_t b = r * shard_rows + q * h;
      s.chunks.push_back({b, b + h, r, 0, r == rank ? 1 : 0});
    }
  switch (kind) {
    case OrderKind::Ring:  // the local shard is present; at ring step t the shard of rank r - t lands
      append_shard(s.order, rank, Q);
      for (int32_t t = 1; t < world; ++t) append_shard(s.order, ((rank - t) % world + world) % world, Q);
      break;
    case OrderKind::Swizzle1D:  // pull peer (i + r) mod W for i = 1 .. W-1 (self skipped)
      append_shard(s.order, rank, Q);
      for (int32_t i = 1; i < world; ++i) append_shard(s.order, (i + rank) % world, Q);
      break;
    case OrderKind::RsRing:  // emit shard (r + 1 + t) mod W; own shard last
      for (int32_t t = 0; t < world; ++t) append_shard(s.order, (rank + 1 + t) % world, Q);
      break;
    case OrderKind::Permutation: {
      if (!remote_perm && world > 1) return "a permutation order needs remote_perm";
      append_shard(s.order, rank, Q);
      std::vector<int32_t> remote;
      for (int32_t r = 0; r < world; ++r)
        if (r != rank) append_shard(remote, r, Q);
      std::vector<char> seen(remote.size(), 0);
      for (size_t i = 0; i < remote.size(); ++i) {
        const int32_t p = remote_perm[i];
        if (p < 0 || static_cast<size_t>(p) >= remote.size() || seen[p]) return "remote_perm is not a permutation";
        seen[p] = 1;
        s.order.push_back(remote[p]);
      }
      break;
    }
    default:
      return "unknown order kind";
  }
  s.total_rows = world * shard_rows;
  std::string err = validate_schedule(s.chunks, s.order);
  if (!err.empty()) return err;
  *out = std::move(s);
  return "";
}

std::string make_grouped_schedule(int32_t world, int32_t rank, int32_t n_groups, const int64_t* counts,
                                  Schedule* out) {
  if (world < 1 || rank < 0 || rank >= world || n_groups < 1) return "bad world, rank or group count";
  if (!counts) return "counts is NULL";
  Schedule s;
  std::vector<int32_t> seg(static_cast<size_t>(world) * n_groups, -1);  // (src, group) -> chunk id
  int64_t row = 0;
  for (int32_t e = 0; e < n_groups; ++e)
    for (int32_t r = 0; r < world; ++r) {
      const int64_t n = counts[static_cast<size_t>(r) * n_groups + e];
      if (n < 0) return "negative count";
      if (n == 0) continue;
      seg[static_cast<size_t>(r) * n_groups + e] = static_cast<int32_t>(s.chunks.size());
      s.chunks.push_back({row, row + n, r, e, r == rank ? 1 : 0});
      row += n;
    }
  if (s.chunks.empty()) return "all counts are zero";
  for (int32_t t = 0; t < world; ++t) {
    const int32_t r = ((rank - t) % world + world) % world;
    for (int32_t e = 0; e < n_groups; ++e) {
      const int32_t id = seg[static_cast<size_t>(r) * n_groups + e];
      if (id >= 0) s.order.push_back(id);
    }
  }
  s.total_rows = row;
  std::string err = validate_schedule(s.chunks, s.order);
  if (!err.empty()) return err;
  *out = std::move(s);
  return "";
}

std::string build_tile_map(const Schedule& s, int64_t M, int64_t N, int32_t bm, int32_t bn, bool producer,
                           const std::vector<int64_t>& group_rows, TileMap* out, int32_t intra_order,
                           int32_t group_m) {
  if (M < 1 || N < 1 || bm < 1 || bn < 1) return "shape and tile sizes must be positive";
  if (intra_order < 0 || intra_order > 1 || group_m < 1) return "unknown intra-chunk order";
  if (s.total_rows != M) return "the schedule's chunks do not cover exactly M rows";
  TileMap tm;
  const int64_t nN = (N + bn - 1) / bn;
  if (nN > (1 << 20)) return "too many tiles along N";
  tm.n_tiles_n = static_cast<int32_t>(nN);
  if (group_rows.empty()) {
    for (int64_t m = 0; m * bm < M; ++m) tm.row_tiles.push_back({m * bm, std::min((m + 1) * bm, M), 0});
  } else {
    int64_t off = 0;
    for (size_t e = 0; e < group_rows.size(); ++e) {
      const int64_t n = group_rows[e];
      if (n < 0) return "negative group rows";
      for (int64_t m = 0; m * bm < n; ++m)
        tm.row_tiles.push_back({off + m * bm, off + std::min((m + 1) * bm, n), static_cast<int32_t>(e)});
      off += n;
    }
    if (off != M) return "group rows do not sum to M";
    // every chunk must stay inside its group's rows
    std::vector<int64_t> goff(group_rows.size() + 1, 0);
    for (size_t e = 0; e < group_rows.size(); ++e) goff[e + 1] = goff[e] + group_rows[e];
    for (const ChunkDesc& c : s.chunks) {
      if (c.group < 0 || static_cast<size_t>(c.group) >= group_rows.size()) return "chunk group out of range";
      if (c.row_begin < goff[c.group] || c.row_end > goff[c.group + 1]) return "a chunk crosses its group's rows";
    }
  }
  const int64_t n_tiles = static_cast<int64_t>(tm.row_tiles.size()) * nN;
  if (n_tiles > (1 << 24)) return "too many tiles";
  const int32_t n_chunks = static_cast<int32_t>(s.chunks.size());
  std::vector<int32_t> pos(n_chunks);
  for (int32_t p = 0; p < n_chunks; ++p) pos[s.order[p]] = p;

  // chunks intersecting each row tile: chunks are sorted by row, so binary search the first
  std::vector<int64_t> starts(n_chunks);
  for (int32_t c = 0; c < n_chunks; ++c) starts[c] = s.chunks[c].row_begin;
  std::vector<std::vector<int32_t>> rowD(tm.row_tiles.size());
  for (size_t m = 0; m < tm.row_tiles.size(); ++m) {
    const RowTile& rt = tm.row_tiles[m];
    int32_t c = static_cast<int32_t>(std::upper_bound(starts.begin(), starts.end(), rt.row_begin) - starts.begin()) - 1;
    for (; c < n_chunks && s.chunks[c].row_begin < rt.row_end; ++c)
      if (s.chunks[c].row_end > rt.row_begin) rowD[m].push_back(c);
    if (rowD[m].empty()) return "a tile touches no chunk";
  }
  tm.tile_ptr.assign(n_tiles + 1, 0);
  for (int64_t t = 0; t < n_tiles; ++t) tm.tile_ptr[t + 1] = tm.tile_ptr[t] + static_cast<int32_t>(rowD[t / nN].size());
  tm.tile_chunks.reserve(tm.tile_ptr.back());
  std::vector<int32_t> need(n_chunks, 0);
  for (int64_t t = 0; t < n_tiles; ++t)
    for (int32_t c : rowD[t / nN]) {
      tm.tile_chunks.push_back(c);
      ++need[c];
    }
  tm.chunk_ptr.assign(n_chunks + 1, 0);
  for (int32_t c = 0; c < n_chunks; ++c) tm.chunk_ptr[c + 1] = tm.chunk_ptr[c] + need[c];
  tm.chunk_tiles.assign(tm.chunk_ptr.back(), 0);
  std::vector<int32_t> fill(tm.chunk_ptr.begin(), tm.chunk_ptr.end() - 1);
  for (int64_t t = 0; t < n_tiles; ++t)  // ascending t keeps each T(c) sorted
    for (int32_t c : rowD[t / nN]) tm.chunk_tiles[fill[c]++] = static_cast<int32_t>(t);

  std::vector<int32_t> rowkey(tm.row_tiles.size());
  for (size_t m = 0; m < tm.row_tiles.size(); ++m) {
    int32_t k = pos[rowD[m][0]];
    for (int32_t c : rowD[m]) k = producer ? std::min(k, pos[c]) : std::max(k, pos[c]);
    rowkey[m] = k;
  }
  tm.order.resize(n_tiles);
  std::iota(tm.order.begin(), tm.order.end(), 0);
  if (intra_order == 0) {
    std::stable_sort(tm.order.begin(), tm.order.end(),
                     [&](int32_t a, int32_t b) { return rowkey[a / nN] < rowkey[b / nN]; });
  } else {
    // band of a row tile: its rank among the row tiles of the same key (ascending), / group_m
    std::vector<int32_t> band(tm.row_tiles.size());
    std::vector<std::pair<int32_t, int32_t>> by_key(tm.row_tiles.size());
    for (size_t m = 0; m < by_key.size(); ++m) by_key[m] = {rowkey[m], static_cast<int32_t>(m)};
    std::sort(by_key.begin(), by_key.end());
    for (size_t i = 0, rank = 0; i < by_key.size(); ++i) {
      rank = (i > 0 && by_key[i].first == by_key[i - 1].first) ? rank + 1 : 0;
      band[by_key[i].second] = static_cast<int32_t>(rank) / group_m;
    }
    auto sort_key = [&](int32_t t) {
      const int32_t m = static_cast<int32_t>(t / nN), n = static_cast<int32_t>(t % nN);
      return std::make_tuple(rowkey[m], band[m], n, m);
    };
    std::sort(tm.order.begin(), tm.order.end(), [&](int32_t a, int32_t b) { return sort_key(a) < sort_key(b); });
  }
  *out = std::move(tm);
  return "";
}

}  // namespace csg
