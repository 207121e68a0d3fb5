"""Tile-order and wave-tail options on the GPU (through the C ABI): the intra-chunk
order (intra_order 1, bands of group_m row tiles visited column by column) and the
wave-tail split (each die's last partial wave split along K).

The intra-chunk order only changes which workgroup runs which tile when; each tile's
K order is fixed, so the output is bit-identical to the raster order's, and equal to
the oracle to the usual bar. The wave-tail split adds the slices' fp32 partial sums in
slice order: the oracle's bar, and every work unit run.
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
    from gpu_util import assert_close, out_to_f64, run_ag, run_rs, tol_for


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _ag(cid, W, r, S, Q, kind, N, K, dtype="bf16", out_dtype="bf16", dist="normal"):
    w = si.Workload(cid, "orders", "ag", M=W * S, N=N, K=K, dtype=dtype, out_dtype=out_dtype, dist=dist,
                    world=W, rank=r, shard_rows=S, chunks_per_shard=Q, order=kind)
    d = si.draw(w)
    perm = si.draw_permutation(cid, 0, (W - 1) * Q) if kind == "permutation" else None
    chunks, order = oracle.uniform_schedule(W, r, S, Q, kind, perm)
    return d, perm, chunks, order


ORDER_CASES = [
    # W, r, S, Q, kind, N, K, group_m, extra cfg
    (4, 1, 1024, 1, "ring", 1280, 512, 2, {}),                       # 4 row tiles per chunk
    (4, 2, 768, 2, "permutation", 1000, 384, 3, {}),                 # ragged N, 384-row chunks straddling tiles
    (2, 0, 1024, 2, "ring", 768, 256, 8, {"tile_dispatch": 2}),      # static, die-major
    (4, 0, 1024, 1, "ring", 512, 512, 2, {"bm": 128, "bn": 128}),    # smaller tiles
]


@pytest.mark.parametrize("case", ORDER_CASES, ids=lambda c: "W%d-r%d-S%d-Q%d-%s-N%d-K%d-g%d" % c[:8])
def test_intra_order_is_bit_identical_to_raster_and_matches_oracle(case):
    W, r, S, Q, kind, N, K, G, extra = case
    _say("intra order %s" % (case,))
    d, perm, chunks, order = _ag(181, W, r, S, Q, kind, N, K)
    outs = []
    for io in (0, 1):
        cfg = dict(extra, timeout_ms=1000, intra_order=io, group_m=G)
        plan = csg.Plan("ag", W * S, N, K, "bf16", "bf16", csg.Schedule.uniform(W, r, S, Q, kind, perm), cfg=cfg)
        m = plan.get_map()
        dm = oracle.dep_map(chunks, order, W * S, N, plan.info.bm, plan.info.bn, intra_order=io, group_m=G)
        assert np.array_equal(m["tile_order"], dm.order)
        c, _ = run_ag(plan, chunks, d.A, d.B, "bf16", poison_remote=True)
        outs.append(out_to_f64(c, "bf16"))
        plan.close()
    R = oracle.ag_gemm(d.A.device_array, d.B.device_array, chunks, order)
    assert_close(outs[1], R, tol_for("bf16", "bf16"), "intra order 1")
    assert np.array_equal(outs[0], outs[1])


def test_intra_order_rs_and_grouped():
    _say("intra order: GEMM-RS and grouped")
    W, r, S, Q, N, K = 4, 1, 512, 1, 768, 512
    w = si.Workload(182, "rs", "rs", M=W * S, N=N, K=K, dtype="bf16", out_dtype="bf16", dist="normal", world=W,
                    rank=r, shard_rows=S, chunks_per_shard=Q, order="rs_ring")
    d = si.draw(w)
    chunks, order = oracle.uniform_schedule(W, r, S, Q, "rs_ring")
    plan = csg.Plan("rs", W * S, N, K, "bf16", "bf16", csg.Schedule.uniform(W, r, S, Q, "rs_ring"),
                    cfg={"timeout_ms": 1000, "intra_order": 1, "group_m": 2})
    c, out = run_rs(plan, d.A, d.B, "bf16")
    R, _, _ = oracle.gemm_rs(d.A.device_array, d.B.device_array, chunks, order)
    G = out_to_f64(c, "bf16")
    assert_close(G, R, 2e-2, "rs intra order")
    O = out_to_f64(out, "bf16")
    for ch in chunks:
        if not ch.is_local:
            assert np.array_equal(O[ch.row_begin:ch.row_end], G[ch.row_begin:ch.row_end])
    counts = np.array([[700, 0, 50], [0, 300, 10], [1300, 0, 0], [10, 200, 900]], dtype=np.int64)
    gchunks, gorder, gr = oracle.grouped_schedule(4, 3, counts)
    M = int(sum(gr))
    X = si.draw_matrix(183, 0, 0, (M, 512), "normal", "bf16")
    B = si.draw_matrix(183, 1, 0, (3, 520, 512), "normal", "bf16")
    gplan = csg.Plan("grouped", M, 520, 512, "bf16", "bf16", csg.Schedule.grouped(4, 3, counts), group_rows=gr,
                     cfg={"timeout_ms": 1000, "intra_order": 1, "group_m": 2})
    c, _ = run_ag(gplan, gchunks, X, B, "bf16")
    R = oracle.grouped_gemm(X.device_array, B.device_array, gchunks, gorder)
    assert_close(out_to_f64(c, "bf16"), R, 2e-2, "grouped intra order")


TAIL_WAVE = [
    # W, r, S, Q, kind, N, K, tail_wave, extra
    (4, 0, 2560, 5, "permutation", 1792, 1024, 2, {}),   # 40 row tiles x 7: 280 tiles on 256 workgroups
    (2, 1, 5120, 4, "ring", 1792, 512, 4, {"intra_order": 1, "group_m": 2}),  # 3 tiles per die into 4 slices
    (4, 0, 512, 2, "ring", 768, 512, 2, {"num_workgroups": 16}),   # 2 workgroups per die, 3 tiles each
]


@pytest.mark.parametrize("case", TAIL_WAVE, ids=lambda c: "W%d-r%d-S%d-Q%d-%s-N%d-K%d-tw%d" % c[:8])
def test_wave_tail_split_parity(case):
    W, r, S, Q, kind, N, K, tw, extra = case
    _say("wave-tail split %s" % (case,))
    d, perm, chunks, order = _ag(184, W, r, S, Q, kind, N, K)
    plan = csg.Plan("ag", W * S, N, K, "bf16", "bf16", csg.Schedule.uniform(W, r, S, Q, kind, perm),
                    cfg=dict(extra, timeout_ms=1000, tail_wave=tw))
    n_tiles = plan.info.n_tiles
    assert plan.info.n_units > n_tiles, "no tile was split"
    R = oracle.ag_gemm(d.A.device_array, d.B.device_array, chunks, order)
    for mode in ("overlap", "compute_only"):
        c, _ = run_ag(plan, chunks, d.A, d.B, "bf16", mode=mode, poison_remote=True)
        assert_close(out_to_f64(c, "bf16"), R, 2e-2, "wave tail %s" % mode)


def test_wave_tail_split_integer_inputs_bit_exact():
    """Integer inputs: every partial sum is exact in fp32, so split slices add up to
    the oracle's value bit for bit."""
    _say("wave-tail split, integer inputs")
    W, r, S, Q, N, K = 4, 2, 2560, 5, 1792, 640
    d, perm, chunks, order = _ag(185, W, r, S, Q, "permutation", N, K, out_dtype="f32", dist="int")
    plan = csg.Plan("ag", W * S, N, K, "bf16", "f32", csg.Schedule.uniform(W, r, S, Q, "permutation", perm),
                    cfg={"timeout_ms": 1000, "tail_wave": 2})
    assert plan.info.n_units > plan.info.n_tiles
    c, _ = run_ag(plan, chunks, d.A, d.B, "f32")
    R = oracle.ag_gemm(d.A.device_array, d.B.device_array, chunks, order)
    assert np.array_equal(out_to_f64(c, "f32"), R)
