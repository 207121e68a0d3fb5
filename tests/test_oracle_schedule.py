"""Pins for the oracle's schedules and dependence map (CPU only).

The oracle is checked against hand-worked examples (tests/golden), closed forms
and an independent row-by-row construction, so that a wrong index, a swapped
min/max or an off-by-one fails here before the oracle judges the GPU path.
"""
import bisect
import json
import os

import numpy as np
import pytest

import oracle
from oracle.schedule import Chunk, ScheduleError, validate

GOLDEN = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "hand_examples.json")))


@pytest.mark.parametrize("ex", GOLDEN["schedules"], ids=lambda e: e["name"])
def test_schedule_hand_examples(ex):
    chunks, order = oracle.uniform_schedule(ex["world"], ex["rank"], ex["Q"] * 16, ex["Q"], ex["kind"],
                                            ex.get("remote_perm"))
    assert order == ex["order"]


@pytest.mark.parametrize("W", [1, 2, 3, 8])
@pytest.mark.parametrize("Q", [1, 4])
def test_schedule_invariants(W, Q):
    for r in range(W):
        for kind in ("ring", "swizzle1d", "rs_ring"):
            chunks, order = oracle.uniform_schedule(W, r, Q * 8, Q, kind)
            assert sorted(order) == list(range(W * Q))
            shard_seq = [chunks[c].src_rank for c in order][::Q]
            # each shard's chunks are contiguous in the order and in row order
            for i in range(W):
                ids = order[i * Q:(i + 1) * Q]
                assert ids == list(range(shard_seq[i] * Q, shard_seq[i] * Q + Q))
            if kind in ("ring", "swizzle1d"):
                assert shard_seq[0] == r                       # local shard first
            else:
                assert shard_seq[-1] == r                      # own shard last
            if kind == "ring":
                assert shard_seq == [(r - t) % W for t in range(W)]
            if kind == "swizzle1d":
                assert shard_seq == [(r + t) % W for t in range(W)]
        for c in chunks:
            assert c.is_local == (c.src_rank == r)


def test_permutation_order_locals_first():
    chunks = oracle.uniform_chunks(4, 2, 64, 4)
    rng = np.random.default_rng(5)
    perm = rng.permutation(12)
    order = oracle.order_permutation(chunks, perm)
    assert order[:4] == [8, 9, 10, 11]
    remote = [i for i in range(16) if not 8 <= i < 12]
    assert order[4:] == [remote[p] for p in perm]
    with pytest.raises(ScheduleError):
        oracle.order_permutation(chunks, [0, 1, 2])


def test_validation_errors():
    good = [Chunk(0, 4, 0, 0, True), Chunk(4, 8, 1, 0, False)]
    validate(good, [1, 0], 8)
    with pytest.raises(ScheduleError):
        validate([Chunk(0, 4, 0, 0, True), Chunk(5, 8, 1, 0, False)], [0, 1], 8)     # gap
    with pytest.raises(ScheduleError):
        validate([Chunk(0, 5, 0, 0, True), Chunk(4, 8, 1, 0, False)], [0, 1], 8)     # overlap
    with pytest.raises(ScheduleError):
        validate(good, [0, 0], 8)                                                   # not a permutation
    with pytest.raises(ScheduleError):
        validate([Chunk(0, 0, 0, 0, True), Chunk(0, 8, 1, 0, False)], [0, 1], 8)     # empty chunk
    with pytest.raises(ScheduleError):
        validate(good, [0, 1], 9)                                                   # short coverage
    with pytest.raises(ScheduleError):
        oracle.uniform_chunks(2, 0, 10, 3)                                          # S % Q != 0


def _chunks_of(ex):
    return oracle.uniform_schedule(ex["world"], ex["rank"], ex["S"], ex["Q"], ex["kind"], ex.get("remote_perm"))


@pytest.mark.parametrize("ex", GOLDEN["depmaps"], ids=lambda e: e["name"])
def test_depmap_hand_examples(ex):
    chunks, order = _chunks_of(ex)
    dm = oracle.dep_map(chunks, order, ex["M"], ex["N"], ex["BM"], ex["BN"], producer=ex["producer"])
    for k in ("tile_ptr", "tile_chunks", "chunk_ptr", "chunk_tiles"):
        assert getattr(dm, k).tolist() == ex[k], k
    assert dm.order.tolist() == ex["order"]


@pytest.mark.parametrize("ex", GOLDEN["grouped"], ids=lambda e: e["name"])
def test_grouped_hand_example(ex):
    chunks, order, group_rows = oracle.grouped_schedule(ex["world"], ex["rank"], np.array(ex["counts"]))
    assert [[c.row_begin, c.row_end, c.src_rank, c.group, int(c.is_local)] for c in chunks] == ex["chunks"]
    assert order == ex["order"]
    assert group_rows == ex["group_rows"]
    dm = oracle.dep_map(chunks, order, sum(group_rows), ex["N"], ex["BM"], ex["BN"], group_rows=group_rows)
    assert dm.tile_ptr.tolist() == ex["tile_ptr"]
    assert dm.tile_chunks.tolist() == ex["tile_chunks"]
    assert dm.order.tolist() == ex["tile_order"]


def _rowwise_D(chunks, M, N, BM, BN):
    """Independent construction: map every row of a tile to its chunk by bisection."""
    starts = [c.row_begin for c in chunks]
    nN = -(-N // BN)
    D = []
    for m in range(-(-M // BM)):
        s = sorted({bisect.bisect_right(starts, r) - 1 for r in range(m * BM, min((m + 1) * BM, M))})
        D += [s] * nN
    return D


@pytest.mark.parametrize("S,Q,BM,BN,N", [(128, 2, 32, 128, 256),    # BM | h
                                         (256, 2, 64, 96, 200),     # BM | h, ragged N
                                         (128, 4, 64, 64, 128),     # h | BM
                                         (128, 2, 96, 64, 130),     # straddling
                                         (96, 3, 80, 48, 100)])     # straddling, ragged M tail
def test_depmap_closed_forms_and_rowwise(S, Q, BM, BN, N):
    W = 3
    M = W * S
    chunks, order = oracle.uniform_schedule(W, 1, S, Q, "ring")
    dm = oracle.dep_map(chunks, order, M, N, BM, BN)
    nN = -(-N // BN)
    h = S // Q
    D = [dm.tile_chunks[dm.tile_ptr[t]:dm.tile_ptr[t + 1]].tolist() for t in range(len(dm.tile_ptr) - 1)]
    assert D == _rowwise_D(chunks, M, N, BM, BN)
    if h % BM == 0:
        for t, d in enumerate(D):
            assert d == [(t // nN) * BM // h]
        assert dm.need.tolist() == [(h // BM) * nN] * len(chunks)
    if BM % h == 0:
        for t, d in enumerate(D):
            m = t // nN
            assert d == list(range(m * BM // h, min((m + 1) * BM // h, len(chunks))))
    assert int(dm.need.sum()) == len(dm.tile_chunks) == int(dm.tile_ptr[-1])
    # T is the inverse of D
    for c in range(len(chunks)):
        tiles = dm.chunk_tiles[dm.chunk_ptr[c]:dm.chunk_ptr[c + 1]].tolist()
        assert tiles == [t for t, d in enumerate(D) if c in d]


@pytest.mark.parametrize("producer", [False, True])
def test_tile_order_properties(producer):
    W, S, Q = 4, 96, 3
    rng = np.random.default_rng(11)
    chunks = oracle.uniform_chunks(W, 2, S, Q)
    order = oracle.order_permutation(chunks, rng.permutation((W - 1) * Q))
    dm = oracle.dep_map(chunks, order, W * S, 70, 40, 32, producer=producer)
    n_tiles = len(dm.tile_ptr) - 1
    assert sorted(dm.order.tolist()) == list(range(n_tiles))
    pos = {c: p for p, c in enumerate(order)}
    keys = []
    for t in dm.order:
        d = dm.tile_chunks[dm.tile_ptr[t]:dm.tile_ptr[t + 1]]
        keys.append((min if producer else max)(pos[int(c)] for c in d))
    assert keys == sorted(keys)
    for i in range(1, n_tiles):
        if keys[i] == keys[i - 1]:
            assert dm.order[i] > dm.order[i - 1]


@pytest.mark.parametrize("ex", GOLDEN["intra_orders"], ids=lambda e: e["name"])
def test_intra_order_hand_examples(ex):
    chunks, order = _chunks_of(ex)
    dm = oracle.dep_map(chunks, order, ex["M"], ex["N"], ex["BM"], ex["BN"], producer=ex["producer"],
                        intra_order=ex["intra_order"], group_m=ex["group_m"])
    assert dm.order.tolist() == ex["order"]


@pytest.mark.parametrize("producer", [False, True])
@pytest.mark.parametrize("S,Q,BM,BN,N,G", [(128, 2, 32, 40, 160, 2),   # BM | h: bands inside a chunk
                                           (96, 3, 80, 48, 100, 3),     # straddling tiles, ragged tails
                                           (256, 1, 32, 64, 192, 3)])   # 8 row tiles per chunk, ragged band
def test_intra_order_keeps_the_chunk_order_and_the_map(producer, S, Q, BM, BN, N, G):
    W = 4
    rng = np.random.default_rng(12)
    chunks = oracle.uniform_chunks(W, 1, S, Q)
    order = oracle.order_permutation(chunks, rng.permutation((W - 1) * Q))
    base = oracle.dep_map(chunks, order, W * S, N, BM, BN, producer=producer)
    sw = oracle.dep_map(chunks, order, W * S, N, BM, BN, producer=producer, intra_order=1, group_m=G)
    for k in ("tile_ptr", "tile_chunks", "chunk_ptr", "chunk_tiles", "need", "keys"):
        assert getattr(sw, k).tolist() == getattr(base, k).tolist(), k
    assert sorted(sw.order.tolist()) == list(range(len(base.order)))
    assert [int(base.keys[t]) for t in sw.order] == [int(base.keys[t]) for t in base.order]
    # band height 1 is the raster order
    one = oracle.dep_map(chunks, order, W * S, N, BM, BN, producer=producer, intra_order=1, group_m=1)
    assert one.order.tolist() == base.order.tolist()


def test_intra_order_whole_chunk_band_is_column_major():
    """Closed form: with BM | h and G >= h / BM every chunk is one band, so its tiles are
    visited column by column: n outer, the chunk's row tiles inner."""
    W, S, Q, BM, BN, N = 3, 256, 2, 32, 64, 320
    chunks, order = oracle.uniform_schedule(W, 2, S, Q, "ring")
    nN = -(-N // BN)
    rows_per_chunk = (S // Q) // BM
    dm = oracle.dep_map(chunks, order, W * S, N, BM, BN, intra_order=1, group_m=rows_per_chunk)
    want = []
    for c in order:
        m0 = chunks[c].row_begin // BM
        want += [m * nN + n for n in range(nN) for m in range(m0, m0 + rows_per_chunk)]
    assert dm.order.tolist() == want
