"""Oracle: one rank's communication schedule (chunk list + arrival/emission order).

TEST INFRASTRUCTURE ONLY. Nothing in the product path may import this module.

Follows the paper's communication-schedule abstraction (Section 5.1): a chunk is
a logical block moved as a unit; a rank's schedule is an ordered list of chunk
operations; manual schedules are parameterised algorithms (loops over ranks and
chunks) specialised to a world size and chunk configuration. On one rank of an
AllGather the chunk operations are pulls of the peers' row shards of A; on one
rank of a ReduceScatter they are pushes of row shards of C.

Chunk ids are in global row order: chunk ``c = s*Q + q`` of a uniform schedule
covers rows ``[s*S + q*h, s*S + (q+1)*h)`` with ``h = S/Q``.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import List, Sequence

import numpy as np


@dataclass(frozen=True)
class Chunk:
    row_begin: int
    row_end: int
    src_rank: int
    group: int
    is_local: bool

    @property
    def rows(self) -> int:
        return self.row_end - self.row_begin


class ScheduleError(ValueError):
    pass


def uniform_chunks(world: int, rank: int, shard_rows: int, chunks_per_shard: int) -> List[Chunk]:
    """Row shards of S rows per rank, each split into Q equal chunks (Section 5.1:
    chunk = logical block; Figure comm_schedule (c) ring AllGather over shards)."""
    if world < 1 or not (0 <= rank < world) or shard_rows < 1 or chunks_per_shard < 1:
        raise ScheduleError("bad uniform schedule parameters")
    if shard_rows % chunks_per_shard:
        raise ScheduleError("shard rows must be divisible by chunks per shard")
    h = shard_rows // chunks_per_shard
    out = []
    for s in range(world):
        for q in range(chunks_per_shard):
            b = s * shard_rows + q * h
            out.append(Chunk(b, b + h, s, 0, s == rank))
    return out


def _shard_ids(s: int, Q: int) -> List[int]:
    return [s * Q + q for q in range(Q)]


def order_ring(world: int, rank: int, Q: int) -> List[int]:
    """Ring AllGather as seen by the receiving rank (Figure comm_schedule (c)):
    the local shard is present first; at ring step t = 1..W-1 the shard of rank
    (rank - t) mod W arrives (each rank forwards what it received from its left
    neighbour). Chunks of a shard arrive in row order."""
    out = _shard_ids(rank, Q)
    for t in range(1, world):
        out += _shard_ids((rank - t) % world, Q)
    return out


def order_swizzle1d(world: int, rank: int, Q: int) -> List[int]:
    """1-D swizzled AllGather pull (the paper's schedule example): loop i over the
    mesh, peer = (i + rank) mod W, skip the rank itself, pull that peer's shard.
    The local shard is present first."""
    out = _shard_ids(rank, Q)
    for i in range(world):
        peer = (i + rank) % world
        if peer == rank:
            continue
        out += _shard_ids(peer, Q)
    return out


def order_rs_ring(world: int, rank: int, Q: int) -> List[int]:
    """ReduceScatter emission order on one rank: shards (rank + 1 + t) mod W for
    t = 0..W-1, so the rank's own shard (which it keeps and receives the
    reduction into) is produced last; chunks of a shard in row order."""
    out = []
    for t in range(world):
        out += _shard_ids((rank + 1 + t) % world, Q)
    return out


def order_permutation(chunks: Sequence[Chunk], remote_perm: Sequence[int]) -> List[int]:
    """Local chunks first (they are present when the call starts), then the remote
    chunks in a given random order: ``remote_perm`` permutes the ascending list
    of remote chunk ids."""
    local = [i for i, c in enumerate(chunks) if c.is_local]
    remote = [i for i, c in enumerate(chunks) if not c.is_local]
    perm = list(int(p) for p in remote_perm)
    if sorted(perm) != list(range(len(remote))):
        raise ScheduleError("remote_perm is not a permutation of the remote chunks")
    return local + [remote[p] for p in perm]


def uniform_schedule(world: int, rank: int, shard_rows: int, chunks_per_shard: int, kind: str,
                     remote_perm=None):
    chunks = uniform_chunks(world, rank, shard_rows, chunks_per_shard)
    Q = chunks_per_shard
    if kind == "ring":
        order = order_ring(world, rank, Q)
    elif kind == "swizzle1d":
        order = order_swizzle1d(world, rank, Q)
    elif kind == "rs_ring":
        order = order_rs_ring(world, rank, Q)
    elif kind == "permutation":
        order = order_permutation(chunks, remote_perm)
    else:
        raise ScheduleError(kind)
    validate(chunks, order, total_rows=world * shard_rows)
    return chunks, order


def grouped_schedule(world: int, rank: int, counts: np.ndarray):
    """All-to-all dispatch into a grouped GEMM, one rank's view. ``counts[s][e]`` is
    the number of routed rows source rank s sends to local expert e. The landing
    buffer is expert-major, then source-major; each non-empty (source, expert)
    segment is one chunk (chunk ids in row order), its group is the expert.
    Arrival: the rank's own segments first, then sources in ring order
    (rank-1, rank-2, ...), experts ascending within a source.
    Returns (chunks, order, group_rows)."""
    counts = np.asarray(counts, dtype=np.int64)
    W, E = counts.shape
    if W != world or not (0 <= rank < world) or (counts < 0).any():
        raise ScheduleError("bad grouped schedule parameters")
    chunks = []
    seg_id = {}
    row = 0
    for e in range(E):
        for s in range(W):
            n = int(counts[s, e])
            if n == 0:
                continue
            seg_id[(s, e)] = len(chunks)
            chunks.append(Chunk(row, row + n, s, e, s == rank))
            row += n
    group_rows = counts.sum(axis=0)
    order = []
    for t in range(W):
        s = (rank - t) % W
        for e in range(E):
            if (s, e) in seg_id:
                order.append(seg_id[(s, e)])
    validate_grouped(chunks, order, group_rows)
    return chunks, order, [int(x) for x in group_rows]


def validate(chunks: Sequence[Chunk], order: Sequence[int], total_rows: int) -> None:
    """Chunks must tile [0, total_rows) in row order, be non-empty, and ``order``
    must be a permutation of the chunk ids."""
    if len(chunks) == 0 or total_rows <= 0:
        raise ScheduleError("empty schedule")
    pos = 0
    for c in chunks:
        if c.row_begin != pos or c.row_end <= c.row_begin:
            raise ScheduleError("chunks must be non-empty and tile the rows in order")
        pos = c.row_end
    if pos != total_rows:
        raise ScheduleError("chunks do not cover the rows")
    if sorted(int(o) for o in order) != list(range(len(chunks))):
        raise ScheduleError("order is not a permutation")


def validate_grouped(chunks: Sequence[Chunk], order: Sequence[int], group_rows: Sequence[int]) -> None:
    total = int(sum(group_rows))
    validate(chunks, order, total)
    off = np.concatenate([[0], np.cumsum(group_rows)])
    for c in chunks:
        e = c.group
        if not (0 <= e < len(group_rows)) or c.row_begin < off[e] or c.row_end > off[e + 1]:
            raise ScheduleError("chunk crosses its group's rows")
