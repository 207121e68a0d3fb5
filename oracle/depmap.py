"""Oracle: chunk-tile dependence map and the chunk-ordered tile list.

TEST INFRASTRUCTURE ONLY. Nothing in the product path may import this module.

Dependency parsing (Section 5.2): a tile depends on the chunks it reads (all-
gather, grouped) or writes (reduce-scatter), found from its tile index and the
chunk-to-row mapping; a tile that consumes a chunk waits for that chunk. The
tile-scheduler swizzle (Section 5.2, Figure tile_scheduler (c)) visits chunks in
the communication order and, inside a chunk, keeps the kernel's original
traversal (row-major raster over (m, n)) by default.

Definitions used here (written out plainly; no blocking or shortcuts):
  tile t = (m, n) covers output rows R(t) = [m*BM, min((m+1)*BM, M)) (grouped:
  rows of one group only) and raster id m*ceil(N/BN) + n;
  D(t) = ascending ids of chunks whose rows intersect R(t);
  T(c) = ascending raster ids of the tiles whose D contains c;  need(c) = |T(c)|;
  key(t) = max_{c in D(t)} pos(c) for consumers (all-gather, grouped),
           min_{c in D(t)} pos(c) for producers (reduce-scatter);
  order = tiles sorted by (key(t), raster id)                   [intra_order 0].

Intra-chunk swizzle (Section 5.2, tile-scheduler swizzling: inside a chunk, visit the
tiles in an order that keeps locality; Section 5.3: the tuner searches intra-tile
orders). Reading used here [intra_order 1, band height G = group_m]: the tiles sharing
one key form a group; the group's row tiles, ascending, are cut into bands of G
consecutive ones, and each band is visited column by column, so consecutive tiles
share B columns across the band's rows and A rows across the columns:
  band(t) = (number of the group's row tiles below t's row tile) // G,
  order = tiles sorted by (key(t), band(t), n, m).
G = 1 gives the raster order again; the chunk order (the key) is never changed.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import List, Sequence

import numpy as np

from .schedule import Chunk


@dataclass
class TileGrid:
    """Row tiles (one entry per m: global row range and group) times N tiles."""
    row_tiles: List[tuple]      # (row_begin, row_end, group)
    n_tiles_n: int

    @property
    def n_tiles(self) -> int:
        return len(self.row_tiles) * self.n_tiles_n


def cdiv(a: int, b: int) -> int:
    return -(-a // b)


def tile_grid(M: int, N: int, BM: int, BN: int, group_rows: Sequence[int] = None) -> TileGrid:
    if group_rows is None:
        rts = [(m * BM, min((m + 1) * BM, M), 0) for m in range(cdiv(M, BM))]
    else:
        rts = []
        off = 0
        for e, n_e in enumerate(group_rows):
            for m in range(cdiv(int(n_e), BM)):
                rts.append((off + m * BM, off + min((m + 1) * BM, int(n_e)), e))
            off += int(n_e)
    return TileGrid(rts, cdiv(N, BN))


@dataclass
class DepMap:
    tile_ptr: np.ndarray        # [n_tiles + 1]
    tile_chunks: np.ndarray     # [nnz]
    chunk_ptr: np.ndarray       # [n_chunks + 1]
    chunk_tiles: np.ndarray     # [nnz]
    need: np.ndarray            # [n_chunks]
    order: np.ndarray           # [n_tiles] raster ids in execution order
    keys: np.ndarray            # [n_tiles] key per raster id


def dep_map(chunks: Sequence[Chunk], order: Sequence[int], M: int, N: int, BM: int, BN: int,
            producer: bool = False, group_rows: Sequence[int] = None, intra_order: int = 0,
            group_m: int = 8) -> DepMap:
    grid = tile_grid(M, N, BM, BN, group_rows)
    nN = grid.n_tiles_n
    n_chunks = len(chunks)
    pos = [0] * n_chunks
    for p, c in enumerate(order):
        pos[int(c)] = p
    D = []
    for t in range(grid.n_tiles):
        rb, re, g = grid.row_tiles[t // nN]
        d = [cid for cid, c in enumerate(chunks)
             if c.row_begin < re and rb < c.row_end and (group_rows is None or c.group == g)]
        D.append(d)
    T = [[] for _ in range(n_chunks)]
    for t, d in enumerate(D):
        for cid in d:
            T[cid].append(t)
    tile_ptr = np.zeros(grid.n_tiles + 1, dtype=np.int32)
    for t, d in enumerate(D):
        tile_ptr[t + 1] = tile_ptr[t] + len(d)
    tile_chunks = np.array([cid for d in D for cid in d], dtype=np.int32)
    chunk_ptr = np.zeros(n_chunks + 1, dtype=np.int32)
    for c in range(n_chunks):
        chunk_ptr[c + 1] = chunk_ptr[c] + len(T[c])
    chunk_tiles = np.array([t for lst in T for t in lst], dtype=np.int32)
    need = np.array([len(lst) for lst in T], dtype=np.int32)
    keys = np.array([(min if producer else max)(pos[c] for c in d) for d in D], dtype=np.int64)
    if intra_order == 0:
        ord_ = np.array(sorted(range(grid.n_tiles), key=lambda t: (keys[t], t)), dtype=np.int32)
    elif intra_order == 1:
        # every tile of a row tile has the same D, hence the same key
        n_rows = len(grid.row_tiles)
        row_key = [int(keys[m * nN]) for m in range(n_rows)]
        band = []
        for m in range(n_rows):
            below = sum(1 for mm in range(m) if row_key[mm] == row_key[m])
            band.append(below // group_m)
        ord_ = np.array(sorted(range(grid.n_tiles),
                               key=lambda t: (keys[t], band[t // nN], t % nN, t // nN)), dtype=np.int32)
    else:
        raise ValueError("intra_order must be 0 or 1")
    return DepMap(tile_ptr, tile_chunks, chunk_ptr, chunk_tiles, need, ord_, keys)
