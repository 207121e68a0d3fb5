// Device execution tables (see exec_tables.hpp).
#include "exec_tables.hpp"

#include <algorithm>

namespace csg {

void build_exec_tables(const Schedule& s, const TileMap& m, const ExecOptions& o, ExecTables* out) {
  const int32_t n_tiles = m.n_tiles();
  const int32_t nN = m.n_tiles_n;
  const int32_t n_chunks = static_cast<int32_t>(s.chunks.size());
  // execution list: the chunk-ordered tile list split into one sub-list per die, a
  // tile going to die (row-tile index mod dies) so that tiles sharing A rows share
  // an L2; each sub-list keeps the chunk order (static dispatch uses the plain list)
  std::vector<int32_t> exec_order;
  std::vector<int32_t> list_begin(kXcdLists + 1, 0);
  if (o.tile_dispatch == 2) {
    exec_order = m.order;
    list_begin.assign(kXcdLists + 1, n_tiles);
    list_begin[0] = 0;
  } else {
    for (int x = 0; x < kXcdLists; ++x) {
      list_begin[x] = static_cast<int32_t>(exec_order.size());
      for (int32_t t : m.order)
        if ((t / nN) % kXcdLists == x) exec_order.push_back(t);
    }
    list_begin[kXcdLists] = static_cast<int32_t>(exec_order.size());
  }
  // K-slices per tile: split_k for every tile; tail_split for the tiles on the
  // critical path of the overlap, i.e. those reading one of the tail_chunks
  // last-arriving chunks (consumers), or writing one of the tail_chunks first-emitted
  // chunks (producer)
  const int32_t KT = static_cast<int32_t>(o.K / o.bk);
  std::vector<int32_t> tile_split(n_tiles, std::max(1, o.split_k));
  std::vector<char> critical_tile(n_tiles, 0);
  if (o.tail_split > 1 && o.tail_chunks > 0) {
    std::vector<int32_t> pos(n_chunks);
    for (int32_t i = 0; i < n_chunks; ++i) pos[s.order[i]] = i;
    for (int32_t t = 0; t < n_tiles; ++t) {
      int32_t lo = n_chunks, hi = -1;
      for (int32_t q = m.tile_ptr[t]; q < m.tile_ptr[t + 1]; ++q) {
        lo = std::min(lo, pos[m.tile_chunks[q]]);
        hi = std::max(hi, pos[m.tile_chunks[q]]);
      }
      const bool critical = o.consumer ? hi >= n_chunks - o.tail_chunks : lo < o.tail_chunks;
      if (critical) {
        // tapered: the tiles of the j-th chunk from the end of the tail (j = 0: the last
        // to arrive, or the first to be emitted) get ceil(S / (1 + j (S - 1) / (C - 1)))
        // slices, S = tail_split, C = tail_chunks: S for the last chunk, 1 for the C-th;
        // a chunk landing d before the last leaves its tiles about d to finish in, and
        // the slice count falls roughly as 1 / d
        int32_t sp = o.tail_split;
        if (o.tail_taper && o.tail_chunks > 1) {
          const int64_t j = o.consumer ? n_chunks - 1 - hi : lo;
          const int64_t S = o.tail_split, Cn = o.tail_chunks;
          // ceil(S (C - 1) / (C - 1 + j (S - 1)))
          sp = static_cast<int32_t>((S * (Cn - 1) + (Cn - 1 + j * (S - 1)) - 1) / (Cn - 1 + j * (S - 1)));
        }
        tile_split[t] = std::max(tile_split[t], sp);
        critical_tile[t] = 1;
      }
    }
  }
  // Static dispatch, consumers: the critical tiles read the last-arriving chunks, so
  // they end the chunk-ordered list; the units from the first of that trailing run on
  // are dealt from a shared ticket.
  int32_t tail_tile = n_tiles;
  if (o.tile_dispatch == 2 && o.consumer && o.tail_split > 1 && o.tail_chunks > 0)
    while (tail_tile > 0 && critical_tile[exec_order[tail_tile - 1]]) --tail_tile;
  // Each die's last partial wave: with w workgroups on a die and L tiles in its list,
  // the last L mod w tiles would run with the rest of the die idle; split each of them
  // into up to w / (L mod w) K-slices (at most tail_wave) so that they fill the die.
  if (o.tail_wave > 1 && o.tile_dispatch != 2 && o.grid >= kXcdLists) {
    const int32_t w = o.grid / kXcdLists;
    for (int x = 0; x < kXcdLists; ++x) {
      const int32_t len = list_begin[x + 1] - list_begin[x];
      const int32_t rem = len % w;
      if (rem == 0) continue;
      const int32_t sp = std::min(o.tail_wave, w / rem);
      if (sp < 2) continue;
      for (int32_t i = list_begin[x + 1] - rem; i < list_begin[x + 1]; ++i)
        tile_split[exec_order[i]] = std::max(tile_split[exec_order[i]], sp);
    }
  }
  for (int32_t& sp : tile_split) sp = std::min(sp, KT);
  // work units: every tile, as tile_split[t] consecutive K-slices; the slices of a
  // split tile own consecutive partial-sum buffers of the workspace
  ExecTables r;
  r.list_ptr.assign(1, 0);
  std::vector<int32_t> unit_begin(kXcdLists + 1, 0);
  for (int32_t i = 0, x = 0; i < n_tiles; ++i) {
    while (x <= kXcdLists && list_begin[x] == i) unit_begin[x++] = static_cast<int32_t>(r.units.size());
    if (i == tail_tile) r.tail_begin = static_cast<int32_t>(r.units.size());
    const int32_t t = exec_order[i];
    const RowTile& rt = m.row_tiles[t / nN];
    const int32_t split = tile_split[t];
    for (int32_t sl = 0; sl < split; ++sl) {
      const int32_t k0 = static_cast<int32_t>(static_cast<int64_t>(KT) * sl / split);
      const int32_t k1 = static_cast<int32_t>(static_cast<int64_t>(KT) * (sl + 1) / split);
      r.units.push_back({static_cast<int32_t>(rt.row_begin), static_cast<int32_t>(rt.row_end), t % nN, rt.group, k0,
                         k1, split > 1 ? r.ws_slices : -1, sl | (split << 16)});
      r.raster.push_back(t);
      for (int32_t q = m.tile_ptr[t]; q < m.tile_ptr[t + 1]; ++q) {
        const int32_t c = m.tile_chunks[q];
        // consumers wait only for chunks that have to arrive; producers signal every chunk
        if (!o.consumer || !s.chunks[c].is_local) r.list_ids.push_back(c);
      }
      r.list_ptr.push_back(static_cast<int32_t>(r.list_ids.size()));
    }
    if (split > 1) r.ws_slices += split;
  }
  for (int x = 0; x <= kXcdLists; ++x)
    if (list_begin[x] == n_tiles) unit_begin[x] = static_cast<int32_t>(r.units.size());
  r.list_begin = unit_begin;
  for (const ChunkDesc& c : s.chunks)
    if ((c.row_begin * o.K * o.in_bytes) % 128 != 0) r.lines_aligned = false;
  // per chunk: tiles that write it (producer), or work units that read it (consumers:
  // the units of split tiles each read the chunk's rows for their K range)
  r.need.assign(n_chunks, 0);
  if (o.consumer)
    for (int32_t c : r.list_ids) ++r.need[c];
  else
    for (int32_t c = 0; c < n_chunks; ++c) r.need[c] = m.chunk_ptr[c + 1] - m.chunk_ptr[c];
  *out = std::move(r);
}

void build_copy_items(const Schedule& s, const std::vector<int32_t>& moved, int64_t row_bytes, int64_t slab,
                      std::vector<CopyItem>* items, std::vector<int32_t>* parts) {
  items->clear();
  parts->clear();
  for (size_t i = 0; i < moved.size(); ++i) {
    const ChunkDesc& ch = s.chunks[moved[i]];
    const int64_t off = ch.row_begin * row_bytes, bytes = (ch.row_end - ch.row_begin) * row_bytes;
    int32_t n = 0;
    for (int64_t b = 0; b < bytes; b += slab, ++n)
      items->push_back({off + b, static_cast<int32_t>(std::min<int64_t>(slab, bytes - b)), static_cast<int32_t>(i)});
    parts->push_back(n);
  }
}

}  // namespace csg
