"""GPU parity: the HIP path (called through the C ABI) against the CPU oracle.

Small cases span several tiles, chunks that straddle tiles, and ragged M / N
tails; they are compared element by element. The benchmark's full-size workloads
are compared on sampled output rows the oracle computes one by one, in the launch
configuration the benchmark times. Tolerances: max relative error (metric of
oracle.max_rel_error) <= 2e-2 with bf16, <= 1e-4 for fp32 end to end; integer-
valued inputs are compared bit for bit.
"""
import sys

import numpy as np
import pytest

import oracle
import paper_2601_20595_amd as csg
import seeded_inputs as si

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    from gpu_util import (DEV, assert_close, bf16_rne_of_f64, out_to_f64, run_ag, run_rs, sample_rows, streams,
                          to_dev, tol_for, empty_out, nan_fill_)


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _small_ag(W, r, S, Q, kind, N, K, dtype, out_dtype, dist="normal", rep=0, cfg_id=101):
    w = si.Workload(cfg_id, "small", "ag", M=W * S, N=N, K=K, dtype=dtype, out_dtype=out_dtype, dist=dist,
                    world=W, rank=r, shard_rows=S, chunks_per_shard=Q, order=kind)
    d = si.draw(w, rep=rep)
    perm = si.draw_permutation(cfg_id, rep, (W - 1) * Q) if kind == "permutation" else None
    chunks, order = oracle.uniform_schedule(W, r, S, Q, kind, perm)
    return w, d, perm, chunks, order


def test_device_is_gfx950():
    assert csg.csg_device_check(0).startswith("gfx950")


AG_SMALL = [
    # W, r, S, Q, kind, N, K, dtype, out
    (2, 0, 128, 2, "permutation", 256, 256, "f32", "f32"),      # the 256^3 fp32 workload itself
    (3, 1, 100, 2, "ring", 200, 96, "f32", "f32"),              # ragged M and N, straddling tiles
    (4, 0, 300, 2, "ring", 600, 512, "bf16", "bf16"),           # ragged M (1200) and N (600), h = 150
    (4, 3, 256, 4, "swizzle1d", 520, 320, "bf16", "bf16"),      # 4 chunks per 256-row tile
    (2, 1, 512, 1, "permutation", 256, 1024, "bf16", "f32"),    # bf16 in, fp32 out
]


@pytest.mark.parametrize("case", AG_SMALL, ids=lambda c: "W%d-r%d-S%d-Q%d-%s-N%d-K%d-%s-%s" % c)
@pytest.mark.parametrize("mode", ["overlap", "compute_only"])
def test_ag_small_parity(case, mode):
    W, r, S, Q, kind, N, K, dtype, out_dtype = case
    _say("ag small %s mode=%s" % (case, mode))
    w, d, perm, chunks, order = _small_ag(W, r, S, Q, kind, N, K, dtype, out_dtype)
    s = csg.Schedule.uniform(W, r, S, Q, kind, perm)
    plan = csg.Plan("ag", W * S, N, K, dtype, out_dtype, s, cfg={"timeout_ms": 1000})
    c, landing = run_ag(plan, chunks, d.A, d.B, out_dtype, mode=mode)
    G = out_to_f64(c, out_dtype)
    R = oracle.ag_gemm(d.A.device_array, d.B.device_array, chunks, order)
    assert_close(G, R, tol_for(out_dtype, dtype), "ag small")
    if mode == "overlap":
        # every remote chunk landed: landing == A
        assert torch.equal(landing.cpu(), to_dev(d.A.device_array).cpu())


@pytest.mark.parametrize("out_dtype", ["f32", "bf16"])
def test_integer_inputs_bit_exact(out_dtype):
    W, r, S, Q, N, K = 4, 2, 192, 3, 384, 640
    _say("integer bit-exact out=%s" % out_dtype)
    w, d, perm, chunks, order = _small_ag(W, r, S, Q, "permutation", N, K, "bf16", out_dtype, dist="int")
    s = csg.Schedule.uniform(W, r, S, Q, "permutation", perm)
    plan = csg.Plan("ag", W * S, N, K, "bf16", out_dtype, s, cfg={"timeout_ms": 1000})
    c, _ = run_ag(plan, chunks, d.A, d.B, out_dtype)
    G = out_to_f64(c, out_dtype)
    R = oracle.ag_gemm(d.A.device_array, d.B.device_array, chunks, order)     # exact integers
    expect = R if out_dtype == "f32" else bf16_rne_of_f64(R)
    assert np.array_equal(G, expect)


def test_arrival_order_does_not_change_a_bit():
    W, r, S, Q, N, K = 4, 1, 256, 2, 512, 512
    _say("order determinism")
    results = []
    for kind, rep in (("ring", 0), ("swizzle1d", 0), ("permutation", 0), ("permutation", 1)):
        w, d, perm, chunks, order = _small_ag(W, r, S, Q, kind, N, K, "bf16", "bf16", rep=0)
        if kind == "permutation":
            perm = si.draw_permutation(77, rep, (W - 1) * Q)
        s = csg.Schedule.uniform(W, r, S, Q, kind, perm)
        plan = csg.Plan("ag", W * S, N, K, "bf16", "bf16", s, cfg={"timeout_ms": 1000})
        c, _ = run_ag(plan, oracle.uniform_schedule(W, r, S, Q, kind, perm)[0], d.A, d.B, "bf16")
        results.append(c.cpu())
    for c in results[1:]:
        assert torch.equal(c, results[0])


def test_identity_weight_copies_every_chunk():
    W, r, S, Q, K = 4, 0, 128, 2, 256
    _say("identity")
    w, d, perm, chunks, order = _small_ag(W, r, S, Q, "ring", K, K, "bf16", "bf16")
    eye = si.Matrix(values=np.eye(K, dtype=np.float32), dtype="bf16",
                    bits=si.f32_to_bf16_bits(np.eye(K, dtype=np.float32)))
    s = csg.Schedule.uniform(W, r, S, Q, "ring")
    plan = csg.Plan("ag", W * S, K, K, "bf16", "bf16", s, cfg={"timeout_ms": 1000})
    c, _ = run_ag(plan, chunks, d.A, eye, "bf16")
    assert np.array_equal(c.cpu().numpy().view(np.uint16), d.A.bits)


def test_poisoned_landing_in_cache_never_reaches_output():
    """Remote rows of the landing buffer hold NaN and were just read (so their lines sit
    in the caches); a tile that read them before its flag, or through a stale line,
    would put NaN into C."""
    W, r, S, Q, N, K = 4, 0, 256, 4, 768, 512
    _say("poison through cache")
    w, d, perm, chunks, order = _small_ag(W, r, S, Q, "ring", N, K, "bf16", "bf16")
    s = csg.Schedule.uniform(W, r, S, Q, "ring")
    plan = csg.Plan("ag", W * S, N, K, "bf16", "bf16", s, cfg={"timeout_ms": 1000})
    R = oracle.ag_gemm(d.A.device_array, d.B.device_array, chunks, order)
    for it in range(3):
        c, _ = run_ag(plan, chunks, d.A, d.B, "bf16", poison_remote=True, touch_remote=True)
        assert_close(out_to_f64(c, "bf16"), R, 2e-2, "poison iteration %d" % it)


@pytest.mark.parametrize("case", [
    # W, r, S, Q, kind, N, K, dtype, out, split
    (4, 0, 256, 4, "ring", 768, 512, "bf16", "bf16", 1),     # 128-byte-aligned chunks: no acquire needed
    (4, 0, 256, 4, "ring", 768, 512, "bf16", "bf16", 2),
    (2, 1, 50, 2, "ring", 64, 16, "f32", "f32", 1),          # 64-byte rows, 25-row chunks: lines straddle chunks
], ids=lambda c: "W%d-r%d-S%d-Q%d-%s-N%d-K%d-%s-%s-split%d" % c)
def test_poisoned_landing_variants(case):
    W, r, S, Q, kind, N, K, dtype, out_dtype, split = case
    _say("poison variant %s" % (case,))
    w, d, perm, chunks, order = _small_ag(W, r, S, Q, kind, N, K, dtype, out_dtype)
    s = csg.Schedule.uniform(W, r, S, Q, kind)
    plan = csg.Plan("ag", W * S, N, K, dtype, out_dtype, s, cfg={"timeout_ms": 1000, "split_k": split})
    R = oracle.ag_gemm(d.A.device_array, d.B.device_array, chunks, order)
    for it in range(3):
        c, _ = run_ag(plan, chunks, d.A, d.B, out_dtype, poison_remote=True, touch_remote=True)
        assert_close(out_to_f64(c, out_dtype), R, tol_for(out_dtype, dtype), "poison iteration %d" % it)


@pytest.mark.parametrize("split", [1, 2, 3])
def test_plan_reuse_with_new_inputs(split):
    """The same plan, buffers reused, inputs changed between calls: a stale cache line
    of the landing buffer or of the split-K partial sums would show as a mismatch."""
    W, r, S, Q, N, K = 4, 1, 256, 2, 512, 640
    _say("plan reuse split=%d" % split)
    s = csg.Schedule.uniform(W, r, S, Q, "swizzle1d")
    plan = csg.Plan("ag", W * S, N, K, "bf16", "bf16", s, cfg={"timeout_ms": 1000, "split_k": split})
    st = streams()
    for rep in range(3):
        w, d, perm, chunks, order = _small_ag(W, r, S, Q, "swizzle1d", N, K, "bf16", "bf16", rep=rep)
        R = oracle.ag_gemm(d.A.device_array, d.B.device_array, chunks, order)
        c, _ = run_ag(plan, chunks, d.A, d.B, "bf16", st=st)
        assert_close(out_to_f64(c, "bf16"), R, 2e-2, "rep %d" % rep)


@pytest.mark.parametrize("split", [1, 2])
def test_back_to_back_calls_into_one_landing_buffer(split):
    """Two calls issued back to back with no synchronisation, the second copying
    different remote rows into the same landing buffer: its copies of a chunk may
    start only once the first call's kernel has read that chunk, so each output
    matches its own inputs."""
    W, r, S, Q, N, K = 4, 1, 256, 2, 512, 512
    _say("back to back split=%d" % split)
    s = csg.Schedule.uniform(W, r, S, Q, "ring")
    chunks, order = oracle.uniform_schedule(W, r, S, Q, "ring")
    plan = csg.Plan("ag", W * S, N, K, "bf16", "bf16", s, cfg={"timeout_ms": 1000, "split_k": split})
    w, d1, _, _, _ = _small_ag(W, r, S, Q, "ring", N, K, "bf16", "bf16", rep=0)
    _, d2, _, _, _ = _small_ag(W, r, S, Q, "ring", N, K, "bf16", "bf16", rep=1)
    A1 = d1.A.device_array.copy()
    A2 = d2.A.device_array.copy()
    for ch in chunks:
        if ch.is_local:                                   # the local shard is shared
            A2[ch.row_begin:ch.row_end] = A1[ch.row_begin:ch.row_end]
    st = streams()
    landing = to_dev(A1).clone()
    for ch in chunks:
        if not ch.is_local:
            landing[ch.row_begin:ch.row_end].zero_()
    stage1, stage2, b = to_dev(A1), to_dev(A2), to_dev(d1.B.device_array)
    c1, c2 = empty_out(W * S, N, "bf16"), empty_out(W * S, N, "bf16")
    nan_fill_(c1)
    nan_fill_(c2)
    torch.cuda.synchronize()
    for _ in range(3):
        plan.ag_gemm(landing, stage1, b, c1, "overlap", st.compute, st.copy)
        plan.ag_gemm(landing, stage2, b, c2, "overlap", st.compute, st.copy)
    plan.check()
    torch.cuda.synchronize()
    R1 = oracle.ag_gemm(A1, d1.B.device_array, chunks, order)
    R2 = oracle.ag_gemm(A2, d1.B.device_array, chunks, order)
    assert_close(out_to_f64(c1, "bf16"), R1, 2e-2, "first call")
    assert_close(out_to_f64(c2, "bf16"), R2, 2e-2, "second call")


def test_repeated_calls_reuse_the_plan():
    W, r, S, Q, N, K = 4, 2, 256, 2, 512, 256
    _say("repeated calls")
    w, d, perm, chunks, order = _small_ag(W, r, S, Q, "swizzle1d", N, K, "bf16", "bf16")
    s = csg.Schedule.uniform(W, r, S, Q, "swizzle1d")
    plan = csg.Plan("ag", W * S, N, K, "bf16", "bf16", s, cfg={"timeout_ms": 1000})
    R = oracle.ag_gemm(d.A.device_array, d.B.device_array, chunks, order)
    c, _ = run_ag(plan, chunks, d.A, d.B, "bf16", repeats=5)
    assert_close(out_to_f64(c, "bf16"), R, 2e-2, "after 5 calls")


RS_SMALL = [
    (4, 1, 256, 2, 512, 320, "bf16", "bf16"),
    (3, 0, 100, 2, 200, 96, "f32", "f32"),        # ragged, straddling
    (8, 5, 64, 1, 256, 128, "bf16", "bf16"),      # 4 chunks per tile row: tiles signal several chunks
]


@pytest.mark.parametrize("case", RS_SMALL, ids=lambda c: "W%d-r%d-S%d-Q%d-N%d-K%d-%s-%s" % c)
@pytest.mark.parametrize("mode", ["overlap", "compute_only"])
def test_rs_small_parity(case, mode):
    W, r, S, Q, N, K, dtype, out_dtype = case
    _say("rs small %s mode=%s" % (case, mode))
    w = si.Workload(103, "rs", "rs", M=W * S, N=N, K=K, dtype=dtype, out_dtype=out_dtype, dist="normal", world=W,
                    rank=r, shard_rows=S, chunks_per_shard=Q, order="rs_ring")
    d = si.draw(w)
    chunks, order = oracle.uniform_schedule(W, r, S, Q, "rs_ring")
    s = csg.Schedule.uniform(W, r, S, Q, "rs_ring")
    plan = csg.Plan("rs", W * S, N, K, dtype, out_dtype, s, cfg={"timeout_ms": 1000})
    c, out = run_rs(plan, d.A, d.B, out_dtype, mode=mode)
    R, Rout, log = oracle.gemm_rs(d.A.device_array, d.B.device_array, chunks, order)
    G = out_to_f64(c, out_dtype)
    assert_close(G, R, tol_for(out_dtype, dtype), "rs C")
    O = out_to_f64(out, out_dtype)
    for ch in chunks:
        rows = slice(ch.row_begin, ch.row_end)
        if ch.is_local or mode == "compute_only":
            assert (O[rows] == 0).all()                  # never sent
        else:
            assert np.array_equal(O[rows], G[rows])      # copy-out of the finished C rows (C was NaN before)


RS_TILE = [
    # W, r, S, Q, N, K, split, backend
    (4, 1, 256, 4, 520, 320, 1, "sdma"),    # 64-row chunks: each 128-row tile writes 2; ragged N
    (4, 2, 512, 2, 512, 256, 1, "sdma"),    # 256-row chunks: 2 row tiles each
    (4, 0, 384, 3, 776, 192, 2, "sdma"),    # split-K
    (8, 5, 256, 2, 256, 128, 1, "kernel"),  # sends from the epilogue
]


@pytest.mark.parametrize("case", RS_TILE, ids=lambda c: "W%d-r%d-S%d-Q%d-N%d-K%d-split%d-%s" % c)
@pytest.mark.parametrize("mode", ["overlap", "compute_only"])
def test_rs_128x256_tiles_parity(case, mode):
    """GEMM + reduce-scatter with 128 x 256 tiles (three-stage ring, 16 x 16 x 32 MFMAs):
    C matches the oracle, every sent chunk's outgoing rows equal C's, and integer inputs
    give the bf16 RNE of the exact sum in every element."""
    W, r, S, Q, N, K, split, backend = case
    _say("rs 128x256 %s mode=%s" % (case, mode))
    for dist in ("normal", "int"):
        w = si.Workload(104, "rs128", "rs", M=W * S, N=N, K=K, dtype="bf16", out_dtype="bf16", dist=dist, world=W,
                        rank=r, shard_rows=S, chunks_per_shard=Q, order="rs_ring")
        d = si.draw(w)
        chunks, order = oracle.uniform_schedule(W, r, S, Q, "rs_ring")
        s = csg.Schedule.uniform(W, r, S, Q, "rs_ring")
        cfg = {"timeout_ms": 1000, "bm": 128, "bn": 256, "bk": 64, "split_k": split}
        if backend == "kernel":
            cfg["copy_backend"] = "kernel"
        plan = csg.Plan("rs", W * S, N, K, "bf16", "bf16", s, cfg=cfg)
        assert (plan.info.bm, plan.info.bn) == (128, 256)
        c, out = run_rs(plan, d.A, d.B, "bf16", mode=mode)
        R, _, _ = oracle.gemm_rs(d.A.device_array, d.B.device_array, chunks, order)
        G = out_to_f64(c, "bf16")
        if dist == "int":
            assert np.array_equal(G, bf16_rne_of_f64(R))
        else:
            assert_close(G, R, tol_for("bf16", "bf16"), "rs 128x256")
        O = out_to_f64(out, "bf16")
        for ch in chunks:
            rows = slice(ch.row_begin, ch.row_end)
            if ch.is_local or mode == "compute_only":
                assert (O[rows] == 0).all()
            else:
                assert np.array_equal(O[rows], G[rows])


@pytest.mark.parametrize("tile", [None, (128, 256), (256, 128), (128, 128)], ids=lambda t: str(t))
def test_grouped_small_parity_with_empty_segments_and_partial_tiles(tile):
    """Experts with empty, tiny and ragged segments, with the default tile and the
    three-stage 16 x 16 x 32 tiles (which cut expert row ranges into more, smaller
    partial tiles)."""
    _say("grouped small tile=%s" % (tile,))
    W, E, N, K = 4, 3, 264, 256
    counts = np.array([[70, 0, 5], [0, 3, 1], [130, 0, 0], [1, 2, 300]], dtype=np.int64)
    chunks, order, gr = oracle.grouped_schedule(W, 1, counts)
    M = int(sum(gr))
    X = si.draw_matrix(104, 0, 0, (M, K), "normal", "bf16")
    B = si.draw_matrix(104, 1, 0, (E, N, K), "normal", "bf16")
    s = csg.Schedule.grouped(W, 1, counts)
    cfg = {"timeout_ms": 1000}
    if tile:
        cfg.update(bm=tile[0], bn=tile[1], bk=64)
    plan = csg.Plan("grouped", M, N, K, "bf16", "bf16", s, group_rows=gr, cfg=cfg)
    c, _ = run_ag(plan, chunks, X, B, "bf16")
    R = oracle.grouped_gemm(X.device_array, B.device_array, chunks, order)
    assert_close(out_to_f64(c, "bf16"), R, 2e-2, "grouped small")


def test_withheld_chunk_times_out_and_plan_recovers():
    """The host releases the last remote chunk long after the kernel's (tiny) wait bound,
    so the kernel must give up with a timeout that names that chunk, and exit normally."""
    W, r, S, Q, N, K = 2, 0, 256, 2, 256, 128
    _say("withheld chunk")
    w, d, perm, chunks, order = _small_ag(W, r, S, Q, "ring", N, K, "bf16", "bf16")
    s = csg.Schedule.uniform(W, r, S, Q, "ring")
    plan = csg.Plan("ag", W * S, N, K, "bf16", "bf16", s, cfg={"timeout_ms": 20})
    plan.set_copy_delays([0.0, 300000.0])            # second remote chunk 300 ms late
    with pytest.raises(csg.CsgError) as ei:
        run_ag(plan, chunks, d.A, d.B, "bf16")
    assert ei.value.status == csg.CSG_ERR_TIMEOUT
    assert ei.value.diag.chunk == order[-1]
    torch.cuda.synchronize()
    plan.set_copy_delays(None)
    c, _ = run_ag(plan, chunks, d.A, d.B, "bf16")
    R = oracle.ag_gemm(d.A.device_array, d.B.device_array, chunks, order)
    assert_close(out_to_f64(c, "bf16"), R, 2e-2, "after recovery")


# ---------------------------------------------------------------------------------
# Split-K and static dispatch: the same results, to the same bar
# ---------------------------------------------------------------------------------
SPLIT_AG = [
    # W, r, S, Q, kind, N, K, dtype, out, split, dispatch
    (4, 0, 300, 2, "ring", 600, 512, "bf16", "bf16", 2, 0),          # 8 K steps, 2 slices, ragged M and N
    (4, 3, 256, 4, "swizzle1d", 520, 640, "bf16", "f32", 3, 0),      # 10 K steps in 3 uneven slices
    (3, 1, 100, 2, "ring", 200, 96, "f32", "f32", 4, 0),             # fp32, 6 K steps in 4 slices
    (2, 1, 512, 1, "permutation", 256, 256, "bf16", "bf16", 8, 0),   # 4 K steps: the split is cut to 4
    (4, 0, 300, 2, "ring", 600, 512, "bf16", "bf16", 1, 2),          # static dispatch, no split
    (4, 3, 256, 4, "swizzle1d", 520, 640, "bf16", "bf16", 2, 2),     # static dispatch with split
]


@pytest.mark.parametrize("case", SPLIT_AG, ids=lambda c: "W%d-r%d-S%d-Q%d-%s-N%d-K%d-%s-%s-split%d-disp%d" % c)
def test_ag_split_k_and_dispatch_parity(case):
    W, r, S, Q, kind, N, K, dtype, out_dtype, split, disp = case
    _say("ag split/dispatch %s" % (case,))
    w, d, perm, chunks, order = _small_ag(W, r, S, Q, kind, N, K, dtype, out_dtype)
    s = csg.Schedule.uniform(W, r, S, Q, kind, perm)
    plan = csg.Plan("ag", W * S, N, K, dtype, out_dtype, s,
                    cfg={"timeout_ms": 1000, "split_k": split, "tile_dispatch": disp})
    R = oracle.ag_gemm(d.A.device_array, d.B.device_array, chunks, order)
    c, _ = run_ag(plan, chunks, d.A, d.B, out_dtype)
    assert_close(out_to_f64(c, out_dtype), R, tol_for(out_dtype, dtype), "ag split")
    # the slices are added in a fixed order: repeated calls give the same bits
    c2, _ = run_ag(plan, chunks, d.A, d.B, out_dtype, repeats=3)
    assert torch.equal(c.cpu(), c2.cpu())


STATIC_GRIDS = [(8, 1), (12, 1), (40, 2), (24, 3)]  # (num_workgroups, split_k): 12 is no multiple of 8


@pytest.mark.parametrize("grid,split", STATIC_GRIDS, ids=lambda v: str(v))
def test_static_dispatch_die_major_slots_cover_every_unit(grid, split):
    """Static dispatch with small grids, several rounds each: a grid that is a multiple
    of 8 deals each round to the dies in consecutive runs of entries, any other grid
    takes entry w + iG; either way every work unit runs exactly once (the plan checks
    the kernel's unit count) and the output matches the oracle."""
    _say("static dispatch grid %d split %d" % (grid, split))
    W, r, S, Q, kind, N, K = 4, 1, 512, 2, "ring", 776, 640
    w, d, perm, chunks, order = _small_ag(W, r, S, Q, kind, N, K, "bf16", "bf16")
    s = csg.Schedule.uniform(W, r, S, Q, kind, perm)
    plan = csg.Plan("ag", W * S, N, K, "bf16", "bf16", s,
                    cfg={"timeout_ms": 1000, "split_k": split, "tile_dispatch": 2, "num_workgroups": grid})
    assert plan.info.num_workgroups == grid
    R = oracle.ag_gemm(d.A.device_array, d.B.device_array, chunks, order)
    c, _ = run_ag(plan, chunks, d.A, d.B, "bf16")
    assert_close(out_to_f64(c, "bf16"), R, tol_for("bf16", "bf16"), "ag static dispatch")


@pytest.mark.parametrize("grid,tail_split,tail_chunks", [(16, 2, 3), (24, 4, 2), (256, 2, 4), (40, 3, 16)],
                         ids=lambda v: str(v))
def test_static_dispatch_shared_tail_ticket(grid, tail_split, tail_chunks):
    """Static dispatch with a tail split: every position before the tail tiles runs on
    its static workgroup, the tail tiles' K-slices on whichever workgroup took them from
    the shared ticket, every position ran, and the output matches the oracle. With
    every chunk in the tail (the last case) the whole list is static."""
    _say("static dispatch shared tail grid %d split %d chunks %d" % (grid, tail_split, tail_chunks))
    W, r, S, Q, kind, N, K = 4, 1, 512, 4, "ring", 776, 640
    w, d, perm, chunks, order = _small_ag(W, r, S, Q, kind, N, K, "bf16", "bf16")
    s = csg.Schedule.uniform(W, r, S, Q, kind, perm)
    plan = csg.Plan("ag", W * S, N, K, "bf16", "bf16", s,
                    cfg={"timeout_ms": 1000, "tile_dispatch": 2, "num_workgroups": grid, "tail_split": tail_split,
                         "tail_chunks": tail_chunks, "trace": 1})
    R = oracle.ag_gemm(d.A.device_array, d.B.device_array, chunks, order)
    c, _ = run_ag(plan, chunks, d.A, d.B, "bf16")
    assert_close(out_to_f64(c, "bf16"), R, tol_for("bf16", "bf16"), "ag static dispatch, shared tail")
    tr = plan.trace()
    assert (tr["t_take"] > 0).all() and (tr["t_end"] >= tr["t_start"]).all()
    info = plan.info
    dm = oracle.dep_map(chunks, order, W * S, N, info.bm, info.bn)
    pos = {int(cid): p for p, cid in enumerate(order)}
    n_chunks = len(chunks)
    critical = [max(pos[int(cid)] for cid in dm.tile_chunks[dm.tile_ptr[t]:dm.tile_ptr[t + 1]]) >= n_chunks - tail_chunks
                for t in range(len(dm.tile_ptr) - 1)]
    per = grid // 8

    def owner(p):
        sl = p % grid
        return (sl % per) * 8 + sl // per

    moved = [i for i in range(len(tr)) if int(tr["workgroup"][i]) != owner(i)]
    assert all(critical[int(tr["raster"][i])] for i in moved), moved[:8]
    if all(critical):
        assert not moved


# ---------------------------------------------------------------------------------
# Smaller bf16 tiles (256x128, 128x256, 128x128): the same results, to the same bar
# ---------------------------------------------------------------------------------
TILE_AG = [
    # W, r, S, Q, kind, N, K, bm, bn, bk, split
    (4, 0, 300, 2, "ring", 600, 512, 256, 128, 64, 1),          # ragged M and N, straddling tiles
    (4, 3, 256, 4, "swizzle1d", 520, 320, 128, 256, 64, 1),     # 2 chunks per 128-row tile
    (2, 1, 512, 1, "permutation", 256, 1024, 128, 128, 64, 1),
    (4, 2, 96, 2, "ring", 200, 192, 128, 128, 64, 1),           # 48-row chunks, ragged N
    (4, 0, 300, 2, "ring", 600, 512, 128, 128, 64, 2),          # with split-K
    (4, 0, 300, 2, "ring", 600, 512, 256, 224, 64, 1),          # 8 x 1 waves: ragged M and N
    (4, 3, 256, 4, "swizzle1d", 896, 320, 256, 224, 64, 1),     # N = 4 x 224
    (2, 1, 512, 1, "permutation", 448, 1024, 256, 224, 64, 2),  # with split-K
]


@pytest.mark.parametrize("case", TILE_AG, ids=lambda c: "W%d-r%d-S%d-Q%d-%s-N%d-K%d-%dx%dx%d-split%d" % c)
@pytest.mark.parametrize("mode", ["overlap", "compute_only"])
def test_ag_tile_shape_parity(case, mode):
    W, r, S, Q, kind, N, K, bm, bn, bk, split = case
    _say("ag tile shape %s mode=%s" % (case, mode))
    w, d, perm, chunks, order = _small_ag(W, r, S, Q, kind, N, K, "bf16", "bf16")
    s = csg.Schedule.uniform(W, r, S, Q, kind, perm)
    plan = csg.Plan("ag", W * S, N, K, "bf16", "bf16", s,
                    cfg={"timeout_ms": 1000, "bm": bm, "bn": bn, "bk": bk, "split_k": split})
    assert (plan.info.bm, plan.info.bn, plan.info.bk) == (bm, bn, bk)
    R = oracle.ag_gemm(d.A.device_array, d.B.device_array, chunks, order)
    c, _ = run_ag(plan, chunks, d.A, d.B, "bf16", mode=mode)
    assert_close(out_to_f64(c, "bf16"), R, tol_for("bf16", "bf16"), "ag tile shape")
    c2, _ = run_ag(plan, chunks, d.A, d.B, "bf16", mode=mode, repeats=3)
    assert torch.equal(c.cpu(), c2.cpu())


RING_DEPTH = [(bm, bn, K, split) for bm, bn in ((128, 256), (256, 128), (128, 128))
              for K, split in ((64, 1), (128, 1), (192, 1), (256, 1), (192, 2), (320, 3))]


@pytest.mark.parametrize("bm,bn,K,split", RING_DEPTH, ids=lambda v: str(v))
def test_three_stage_ring_short_k_bit_exact(bm, bn, K, split):
    """The tiles with a three-stage DMA ring at K steps of 1 to 5 stages per unit (fewer
    stages than the ring holds, exactly as many, a few more), whole and split along K:
    integer inputs give exact sums, so the bf16 output must equal the RNE of the oracle's
    exact value in every element, and repeated calls the same bits."""
    W, r, S, Q, kind, N = 4, 2, 160, 2, "ring", 520
    _say("three-stage ring %dx%d K=%d split=%d" % (bm, bn, K, split))
    w, d, perm, chunks, order = _small_ag(W, r, S, Q, kind, N, K, "bf16", "bf16", dist="int")
    s = csg.Schedule.uniform(W, r, S, Q, kind, perm)
    plan = csg.Plan("ag", W * S, N, K, "bf16", "bf16", s,
                    cfg={"timeout_ms": 1000, "bm": bm, "bn": bn, "bk": 64, "split_k": split})
    assert (plan.info.bm, plan.info.bn) == (bm, bn)
    R = oracle.ag_gemm(d.A.device_array, d.B.device_array, chunks, order)     # exact integers
    for mode in ("overlap", "compute_only"):
        c, _ = run_ag(plan, chunks, d.A, d.B, "bf16", mode=mode, repeats=2)
        assert np.array_equal(out_to_f64(c, "bf16"), bf16_rne_of_f64(R)), mode


def test_ag_256x224_fp32_output_integer_inputs_bit_exact():
    W, r, S, Q, kind, N, K = 4, 1, 256, 2, "ring", 448, 640
    _say("ag 256x224 fp32 out, integer inputs")
    w, d, perm, chunks, order = _small_ag(W, r, S, Q, kind, N, K, "bf16", "f32", dist="int")
    s = csg.Schedule.uniform(W, r, S, Q, kind, perm)
    plan = csg.Plan("ag", W * S, N, K, "bf16", "f32", s, cfg={"timeout_ms": 1000, "bm": 256, "bn": 224, "bk": 64})
    assert (plan.info.bm, plan.info.bn) == (256, 224)
    c, _ = run_ag(plan, chunks, d.A, d.B, "f32")
    R = oracle.ag_gemm(d.A.device_array, d.B.device_array, chunks, order)
    assert np.array_equal(out_to_f64(c, "f32"), R)


TAIL_CASES = [
    # op, W, r, S, Q, kind, N, K, cfg
    ("ag", 4, 0, 300, 2, "ring", 600, 512, {"tail_split": 2, "tail_chunks": 2}),
    ("ag", 2, 1, 512, 1, "permutation", 256, 1024, {"tail_split": 4, "tail_chunks": 1}),
    ("ag", 4, 3, 256, 4, "swizzle1d", 520, 640, {"split_k": 2, "tail_split": 3, "tail_chunks": 5}),
    ("ag", 4, 0, 256, 4, "ring", 512, 512, {"tail_split": 2, "tail_chunks": 4, "num_workgroups": 8}),
    ("rs", 4, 1, 256, 2, "rs_ring", 512, 640, {"tail_split": 2, "tail_chunks": 3}),
    ("ag", 4, 3, 256, 4, "swizzle1d", 520, 640, {"tail_split": 5, "tail_chunks": 6, "tail_taper": 1}),
    ("ag", 4, 0, 256, 4, "ring", 512, 512, {"tail_split": 4, "tail_chunks": 8, "tail_taper": 1, "tile_dispatch": 2,
                                             "num_workgroups": 16}),
    ("rs", 4, 1, 256, 2, "rs_ring", 512, 640, {"tail_split": 3, "tail_chunks": 4, "tail_taper": 1}),
]


@pytest.mark.parametrize("case", TAIL_CASES, ids=lambda c: "%s-W%d-r%d-S%d-Q%d-%s-N%d-K%d-%s" % (
    c[:8] + ("_".join("%s%d" % kv for kv in sorted(c[8].items())),)))
def test_tail_split_parity(case):
    """Tiles on the critical path split along K (the rest whole): same result, to the
    same bar, and every work unit ran."""
    op, W, r, S, Q, kind, N, K, cfg = case
    _say("tail split %s" % (case,))
    cfg = dict(cfg, timeout_ms=1000)
    if op == "rs":
        w = si.Workload(103, "rs", "rs", M=W * S, N=N, K=K, dtype="bf16", out_dtype="bf16", dist="normal", world=W,
                        rank=r, shard_rows=S, chunks_per_shard=Q, order="rs_ring")
        d = si.draw(w)
        chunks, order = oracle.uniform_schedule(W, r, S, Q, "rs_ring")
        plan = csg.Plan("rs", W * S, N, K, "bf16", "bf16", csg.Schedule.uniform(W, r, S, Q, "rs_ring"), cfg=cfg)
        c, out = run_rs(plan, d.A, d.B, "bf16")
        R, _, _ = oracle.gemm_rs(d.A.device_array, d.B.device_array, chunks, order)
        G = out_to_f64(c, "bf16")
        assert_close(G, R, 2e-2, "rs tail")
        O = out_to_f64(out, "bf16")
        for ch in chunks:
            if not ch.is_local:
                assert np.array_equal(O[ch.row_begin:ch.row_end], G[ch.row_begin:ch.row_end])
        return
    w, d, perm, chunks, order = _small_ag(W, r, S, Q, kind, N, K, "bf16", "bf16")
    plan = csg.Plan("ag", W * S, N, K, "bf16", "bf16", csg.Schedule.uniform(W, r, S, Q, kind, perm), cfg=cfg)
    R = oracle.ag_gemm(d.A.device_array, d.B.device_array, chunks, order)
    for mode in ("overlap", "compute_only"):
        c, _ = run_ag(plan, chunks, d.A, d.B, "bf16", mode=mode)
        assert_close(out_to_f64(c, "bf16"), R, 2e-2, "ag tail %s" % mode)


@pytest.mark.parametrize("op,S_,C_", [("ag", 6, 5), ("ag", 3, 12), ("rs", 4, 3)])
def test_tapered_tail_split_unit_count(op, S_, C_):
    """The tapered tail split gives the tiles of the j-th tail chunk (from the last
    arrival, or the first emission) ceil(S / (1 + j (S - 1) / (C - 1))) K-slices: the
    plan's unit count equals that sum over the oracle's dependence map, and the output
    matches the oracle."""
    W, r, S, Q, N, K = 4, 1, 256, 4, 520, 640
    kind = "rs_ring" if op == "rs" else "ring"
    _say("tapered tail %s S=%d C=%d" % (op, S_, C_))
    chunks, order = oracle.uniform_schedule(W, r, S, Q, kind)
    cfg = {"timeout_ms": 1000, "tail_split": S_, "tail_chunks": C_, "tail_taper": 1}
    plan = csg.Plan(op, W * S, N, K, "bf16", "bf16", csg.Schedule.uniform(W, r, S, Q, kind), cfg=cfg)
    info = plan.info
    dm = oracle.dep_map(chunks, order, W * S, N, info.bm, info.bn, producer=(op == "rs"))
    pos = {int(cid): p for p, cid in enumerate(order)}
    n_chunks, KT = len(chunks), K // info.bk
    expect = 0
    for t in range(len(dm.tile_ptr) - 1):
        ps = [pos[int(cid)] for cid in dm.tile_chunks[dm.tile_ptr[t]:dm.tile_ptr[t + 1]]]
        j = (n_chunks - 1 - max(ps)) if op == "ag" else min(ps)
        sp = 1
        if j < C_:
            sp = -(-S_ * (C_ - 1) // (C_ - 1 + j * (S_ - 1)))    # ceil
        expect += min(sp, KT)
    assert info.n_units == expect
    if op == "rs":
        w = si.Workload(103, "rs", "rs", M=W * S, N=N, K=K, dtype="bf16", out_dtype="bf16", dist="normal", world=W,
                        rank=r, shard_rows=S, chunks_per_shard=Q, order="rs_ring")
        d = si.draw(w)
        c, out = run_rs(plan, d.A, d.B, "bf16")
        R, _, _ = oracle.gemm_rs(d.A.device_array, d.B.device_array, chunks, order)
    else:
        w, d, perm, chunks, order = _small_ag(W, r, S, Q, kind, N, K, "bf16", "bf16")
        c, _ = run_ag(plan, chunks, d.A, d.B, "bf16")
        R = oracle.ag_gemm(d.A.device_array, d.B.device_array, chunks, order)
    assert_close(out_to_f64(c, "bf16"), R, 2e-2, "tapered tail %s" % op)


def test_grouped_tail_split_parity():
    _say("grouped tail split")
    W, E, N, K = 4, 3, 264, 512
    counts = np.array([[70, 0, 5], [0, 3, 1], [130, 0, 0], [1, 2, 300]], dtype=np.int64)
    chunks, order, gr = oracle.grouped_schedule(W, 3, counts)
    M = int(sum(gr))
    X = si.draw_matrix(106, 0, 0, (M, K), "normal", "bf16")
    B = si.draw_matrix(106, 1, 0, (E, N, K), "normal", "bf16")
    plan = csg.Plan("grouped", M, N, K, "bf16", "bf16", csg.Schedule.grouped(W, 3, counts), group_rows=gr,
                    cfg={"timeout_ms": 1000, "tail_split": 4, "tail_chunks": 3})
    c, _ = run_ag(plan, chunks, X, B, "bf16")
    R = oracle.grouped_gemm(X.device_array, B.device_array, chunks, order)
    assert_close(out_to_f64(c, "bf16"), R, 2e-2, "grouped tail")


@pytest.mark.parametrize("split", [2, 5])
def test_split_k_integer_inputs_bit_exact(split):
    W, r, S, Q, N, K = 4, 2, 192, 3, 384, 640
    _say("integer bit-exact split=%d" % split)
    w, d, perm, chunks, order = _small_ag(W, r, S, Q, "permutation", N, K, "bf16", "f32", dist="int")
    s = csg.Schedule.uniform(W, r, S, Q, "permutation", perm)
    plan = csg.Plan("ag", W * S, N, K, "bf16", "f32", s, cfg={"timeout_ms": 1000, "split_k": split})
    c, _ = run_ag(plan, chunks, d.A, d.B, "f32")
    R = oracle.ag_gemm(d.A.device_array, d.B.device_array, chunks, order)
    assert np.array_equal(out_to_f64(c, "f32"), R)


@pytest.mark.parametrize("split", [2, 3])
def test_rs_split_k_parity(split):
    """A chunk's flag rises only after the last slice of its last tile has written C."""
    W, r, S, Q, N, K = 4, 1, 256, 2, 512, 640
    _say("rs split=%d" % split)
    w = si.Workload(103, "rs", "rs", M=W * S, N=N, K=K, dtype="bf16", out_dtype="bf16", dist="normal", world=W,
                    rank=r, shard_rows=S, chunks_per_shard=Q, order="rs_ring")
    d = si.draw(w)
    chunks, order = oracle.uniform_schedule(W, r, S, Q, "rs_ring")
    s = csg.Schedule.uniform(W, r, S, Q, "rs_ring")
    plan = csg.Plan("rs", W * S, N, K, "bf16", "bf16", s, cfg={"timeout_ms": 1000, "split_k": split})
    c, out = run_rs(plan, d.A, d.B, "bf16")
    R, _, _ = oracle.gemm_rs(d.A.device_array, d.B.device_array, chunks, order)
    G = out_to_f64(c, "bf16")
    assert_close(G, R, 2e-2, "rs split C")
    O = out_to_f64(out, "bf16")
    for ch in chunks:
        rows = slice(ch.row_begin, ch.row_end)
        if ch.is_local:
            assert (O[rows] == 0).all()
        else:
            assert np.array_equal(O[rows], G[rows])


def test_grouped_split_k_parity():
    _say("grouped split")
    W, E, N, K = 4, 3, 264, 512
    counts = np.array([[70, 0, 5], [0, 3, 1], [130, 0, 0], [1, 2, 300]], dtype=np.int64)
    chunks, order, gr = oracle.grouped_schedule(W, 2, counts)
    M = int(sum(gr))
    X = si.draw_matrix(105, 0, 0, (M, K), "normal", "bf16")
    B = si.draw_matrix(105, 1, 0, (E, N, K), "normal", "bf16")
    s = csg.Schedule.grouped(W, 2, counts)
    plan = csg.Plan("grouped", M, N, K, "bf16", "bf16", s, group_rows=gr, cfg={"timeout_ms": 1000, "split_k": 3})
    c, _ = run_ag(plan, chunks, X, B, "bf16")
    R = oracle.grouped_gemm(X.device_array, B.device_array, chunks, order)
    assert_close(out_to_f64(c, "bf16"), R, 2e-2, "grouped split")


# ---------------------------------------------------------------------------------
# Full-size workloads, sampled rows, in the benchmark's launch configuration
# ---------------------------------------------------------------------------------
def _full(cfg_id):
    w = si.WORKLOADS[cfg_id]
    d = si.draw(w)
    if w.op == "grouped":
        chunks, order, gr = oracle.grouped_schedule(w.world, w.rank, d.counts)
        s = csg.Schedule.grouped(w.world, w.rank, d.counts)
        return w, d, chunks, order, s, gr
    chunks, order = oracle.uniform_schedule(w.world, w.rank, w.shard_rows, w.chunks_per_shard, w.order, d.perm)
    s = csg.Schedule.uniform(w.world, w.rank, w.shard_rows, w.chunks_per_shard, w.order, d.perm)
    return w, d, chunks, order, s, None


@pytest.mark.parametrize("cfg_id,tuned", [(1, False), (2, False), (2, True), (3, False), (3, True), (4, False),
                                          (4, True), (5, False), (5, True)])
def test_full_size_workload_sampled(cfg_id, tuned):
    """Each workload at full size with the library's default plan and, where bench.py
    measures a tuned plan configuration, with that one."""
    import bench
    w, d, chunks, order, s, gr = _full(cfg_id)
    cfg = dict(bench.TUNED_PLAN_CFG[cfg_id]) if tuned else None
    _say("full size %s plan %s" % (w.name, cfg))
    plan = csg.Plan(w.op, w.M, w.N, w.K, w.dtype, w.out_dtype, s, group_rows=gr, cfg=cfg)
    if d.delays_us is not None:
        plan.set_copy_delays(d.delays_us)
    rows = sample_rows(chunks, extra=24, seed=cfg_id, M=w.M) if w.M > 256 else list(range(w.M))
    tol = tol_for(w.out_dtype, w.dtype)
    if w.op == "rs":
        c, out = run_rs(plan, d.A, d.B, w.out_dtype)
        R, _, _ = oracle.gemm_rs(d.A.device_array, d.B.device_array, chunks, order, row_subset=rows)
        G = out_to_f64(c[rows], w.out_dtype)
        assert_close(G, R[rows], tol, w.name)
        O = out_to_f64(out[rows], w.out_dtype)
        remote = np.array([not chunks[next(i for i, ch in enumerate(chunks) if ch.row_begin <= r < ch.row_end)].is_local
                           for r in rows])
        assert np.array_equal(O[remote], G[remote])
        return
    c, _ = run_ag(plan, chunks, d.A, d.B, w.out_dtype)
    if w.op == "grouped":
        R = oracle.grouped_gemm(d.A.device_array, d.B.device_array, chunks, order, row_subset=rows)
    else:
        R = oracle.ag_gemm(d.A.device_array, d.B.device_array, chunks, order, row_subset=rows)
    assert_close(out_to_f64(c[rows], w.out_dtype), R[rows], tol, w.name)


@pytest.mark.parametrize("op", ["ag", "rs"])
def test_plan_destroyed_right_after_a_call_waits_for_its_work(op):
    """A plan destroyed straight after an overlap call (no check, no synchronisation)
    must first wait for its kernel and copies, which still read the plan's signals and
    tables; the caller's outputs are then complete."""
    W, r, S, Q, N, K = 4, 1, 256, 2, 512, 512
    _say("destroy right after a call: %s" % op)
    st = streams()
    if op == "ag":
        w, d, perm, chunks, order = _small_ag(W, r, S, Q, "ring", N, K, "bf16", "bf16")
        s = csg.Schedule.uniform(W, r, S, Q, "ring")
        plan = csg.Plan("ag", W * S, N, K, "bf16", "bf16", s, cfg={"timeout_ms": 1000})
        a = to_dev(d.A.device_array)
        landing = a.clone()
        for ch in chunks:
            if not ch.is_local:
                landing[ch.row_begin:ch.row_end].zero_()
        b = to_dev(d.B.device_array)
        c = empty_out(W * S, N, "bf16")
        torch.cuda.synchronize()
        plan.ag_gemm(landing, a, b, c, "overlap", st.compute, st.copy)
        plan.close()
        torch.cuda.synchronize()
        R = oracle.ag_gemm(d.A.device_array, d.B.device_array, chunks, order)
        assert_close(out_to_f64(c, "bf16"), R, 2e-2, "ag after destroy")
        assert torch.equal(landing, a)
    else:
        w = si.Workload(103, "rs", "rs", M=W * S, N=N, K=K, dtype="bf16", out_dtype="bf16", dist="normal", world=W,
                        rank=r, shard_rows=S, chunks_per_shard=Q, order="rs_ring")
        d = si.draw(w)
        chunks, order = oracle.uniform_schedule(W, r, S, Q, "rs_ring")
        s = csg.Schedule.uniform(W, r, S, Q, "rs_ring")
        plan = csg.Plan("rs", W * S, N, K, "bf16", "bf16", s, cfg={"timeout_ms": 1000})
        a, b = to_dev(d.A.device_array), to_dev(d.B.device_array)
        c, out = empty_out(W * S, N, "bf16"), empty_out(W * S, N, "bf16")
        out.zero_()
        torch.cuda.synchronize()
        plan.gemm_rs(a, b, c, out, "overlap", st.compute, st.copy)
        plan.close()
        torch.cuda.synchronize()
        R, _, _ = oracle.gemm_rs(d.A.device_array, d.B.device_array, chunks, order)
        G, O = out_to_f64(c, "bf16"), out_to_f64(out, "bf16")
        assert_close(G, R, 2e-2, "rs after destroy")
        for ch in chunks:
            if not ch.is_local:
                assert np.array_equal(O[ch.row_begin:ch.row_end], G[ch.row_begin:ch.row_end])
    s.close()


# ---------------------------------------------------------------------------------
# The LDS-staged epilogue (bf16 output, 256 x 256 and 128 x 256 tiles): rows written
# whole from LDS, with ragged row tiles and a last column tile that ends in a half
# 16-byte piece (N = 8 k + 4), on the consumer and on the producer. C sits at the start
# of a larger buffer whose tail holds a sentinel: nothing may be written past C's end.
# ---------------------------------------------------------------------------------
@pytest.mark.parametrize("op,bm", [("ag", 256), ("ag", 128), ("rs", 256)])
@pytest.mark.parametrize("N", [260, 516, 772])
def test_staged_epilogue_ragged_edges(op, bm, N):
    W, r, S, Q, K = 4, 1, 200, 2, 192
    M = W * S
    _say("staged epilogue %s bm=%d N=%d" % (op, bm, N))
    cfg = {"timeout_ms": 1000, "bm": bm, "bn": 256, "bk": 64}
    st = streams()
    guard = 4096
    flat = torch.full((M * N + guard,), 0x7fc1, dtype=torch.int16, device="cuda")  # bf16 NaN bits
    c = flat[:M * N].view(M, N)
    if op == "ag":
        w, d, perm, chunks, order = _small_ag(W, r, S, Q, "ring", N, K, "bf16", "bf16")
        s = csg.Schedule.uniform(W, r, S, Q, "ring")
        plan = csg.Plan("ag", M, N, K, "bf16", "bf16", s, cfg=cfg)
        a = to_dev(d.A.device_array)
        landing = a.clone()
        for ch in chunks:
            if not ch.is_local:
                landing[ch.row_begin:ch.row_end].zero_()
        torch.cuda.synchronize()
        plan.ag_gemm(landing, a, to_dev(d.B.device_array), c, "overlap", st.compute, st.copy)
        plan.check()
        torch.cuda.synchronize()
        R = oracle.ag_gemm(d.A.device_array, d.B.device_array, chunks, order)
        assert_close(out_to_f64(c, "bf16"), R, tol_for("bf16", "bf16"), "ag staged epilogue")
    else:
        w = si.Workload(103, "rs", "rs", M=M, N=N, K=K, dtype="bf16", out_dtype="bf16", dist="normal", world=W,
                        rank=r, shard_rows=S, chunks_per_shard=Q, order="rs_ring")
        d = si.draw(w)
        chunks, order = oracle.uniform_schedule(W, r, S, Q, "rs_ring")
        s = csg.Schedule.uniform(W, r, S, Q, "rs_ring")
        plan = csg.Plan("rs", M, N, K, "bf16", "bf16", s, cfg=cfg)
        out = empty_out(M, N, "bf16")
        out.zero_()
        torch.cuda.synchronize()
        plan.gemm_rs(to_dev(d.A.device_array), to_dev(d.B.device_array), c, out, "overlap", st.compute, st.copy)
        plan.check()
        torch.cuda.synchronize()
        R, _, _ = oracle.gemm_rs(d.A.device_array, d.B.device_array, chunks, order)
        G = out_to_f64(c, "bf16")
        assert_close(G, R, tol_for("bf16", "bf16"), "rs staged epilogue")
        O = out_to_f64(out, "bf16")
        for ch in chunks:
            if not ch.is_local:
                assert np.array_equal(O[ch.row_begin:ch.row_end], G[ch.row_begin:ch.row_end])
    assert (plan.info.bm, plan.info.bn) == (bm, 256)
    assert bool((flat[M * N:] == 0x7fc1).all()), "a store landed past the end of C"
    plan.close()
    s.close()
