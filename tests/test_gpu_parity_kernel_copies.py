"""GPU parity of the kernel copy backend (CSG_COPY_KERNEL) against the CPU oracle,
through the C ABI.

With this backend the persistent GEMM kernel moves the chunks itself (Section 5.2,
load/store realizations): for AG and grouped GEMM the first copy workgroups to start
copy the remote chunks staging -> landing in arrival order and raise each chunk's
ready word; for GEMM-RS a tile of a sent chunk stores its output rows into the
outgoing buffer as well. The checks are those of the copy-engine path: C against the
oracle (same tolerances), every remote chunk landed (AG) or sent (RS), local rows
of the outgoing buffer untouched, no poisoned landing row reaching C.
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
    from gpu_util import (assert_close, bf16_rne_of_f64, empty_out, nan_fill_, out_to_f64, run_ag, run_rs, sample_rows,
                          streams, to_dev, tol_for)


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _kc(**kw):
    cfg = {"timeout_ms": 1000, "copy_backend": "kernel"}
    cfg.update(kw)
    return cfg


def _small_ag(W, r, S, Q, kind, N, K, dtype, out_dtype, dist="normal", cfg_id=111):
    w = si.Workload(cfg_id, "small", "ag", M=W * S, N=N, K=K, dtype=dtype, out_dtype=out_dtype, dist=dist,
                    world=W, rank=r, shard_rows=S, chunks_per_shard=Q, order=kind)
    d = si.draw(w)
    perm = si.draw_permutation(cfg_id, 0, (W - 1) * Q) if kind == "permutation" else None
    chunks, order = oracle.uniform_schedule(W, r, S, Q, kind, perm)
    return d, perm, chunks, order


AG_CASES = [
    # W, r, S, Q, kind, N, K, dtype, out, copy_workgroups, num_workgroups
    (2, 0, 128, 2, "permutation", 256, 256, "f32", "f32", 0, 0),    # the 256^3 fp32 workload, default copiers
    (3, 1, 100, 2, "ring", 200, 96, "f32", "f32", 3, 0),            # ragged M and N, straddling tiles
    (4, 0, 300, 2, "ring", 600, 512, "bf16", "bf16", 1, 0),         # one copy workgroup, h = 150
    (4, 3, 256, 4, "swizzle1d", 520, 320, "bf16", "bf16", 64, 0),   # 4 chunks per 256-row tile
    (2, 1, 512, 1, "permutation", 256, 1024, "bf16", "f32", 16, 8),  # more copiers than workgroups
    (2, 1, 50, 2, "ring", 64, 16, "f32", "f32", 4, 0),              # 64-byte rows: lines straddle chunks
]
AG_IDS = ["W%d-r%d-S%d-Q%d-%s-N%d-K%d-%s-%s-cw%d-g%d" % c for c in AG_CASES]


@pytest.mark.parametrize("case", AG_CASES, ids=AG_IDS)
@pytest.mark.parametrize("mode", ["overlap", "compute_only"])
def test_kernel_copies_ag_parity(case, mode):
    W, r, S, Q, kind, N, K, dtype, out_dtype, cw, g = case
    _say("kernel copies ag %s mode=%s" % (case, mode))
    d, perm, chunks, order = _small_ag(W, r, S, Q, kind, N, K, dtype, out_dtype)
    s = csg.Schedule.uniform(W, r, S, Q, kind, perm)
    plan = csg.Plan("ag", W * S, N, K, dtype, out_dtype, s, cfg=_kc(copy_workgroups=cw, num_workgroups=g))
    # overlap: remote landing rows hold NaN and sit in the caches before the call
    c, landing = run_ag(plan, chunks, d.A, d.B, out_dtype, mode=mode, poison_remote=mode == "overlap",
                        touch_remote=mode == "overlap")
    R = oracle.ag_gemm(d.A.device_array, d.B.device_array, chunks, order)
    assert_close(out_to_f64(c, out_dtype), R, tol_for(out_dtype, dtype), "kernel copies ag")
    if mode == "overlap":
        assert torch.equal(landing.cpu(), to_dev(d.A.device_array).cpu())


@pytest.mark.parametrize("case", AG_CASES[1:5], ids=AG_IDS[1:5])
def test_kernel_copies_ag_copy_only(case):
    """Copy-only: the copy workgroups alone run; every remote chunk lands, no tile runs."""
    W, r, S, Q, kind, N, K, dtype, out_dtype, cw, g = case
    _say("kernel copies ag copy-only %s" % (case,))
    d, perm, chunks, order = _small_ag(W, r, S, Q, kind, N, K, dtype, out_dtype)
    s = csg.Schedule.uniform(W, r, S, Q, kind, perm)
    plan = csg.Plan("ag", W * S, N, K, dtype, out_dtype, s, cfg=_kc(copy_workgroups=cw, num_workgroups=g))
    c, landing = run_ag(plan, chunks, d.A, d.B, out_dtype, mode="copy_only", poison_remote=True)
    assert torch.equal(landing.cpu(), to_dev(d.A.device_array).cpu())
    assert np.isnan(out_to_f64(c, out_dtype)).all()           # C untouched


@pytest.mark.parametrize("out_dtype", ["f32", "bf16"])
def test_kernel_copies_integer_inputs_bit_exact(out_dtype):
    W, r, S, Q, N, K = 4, 2, 192, 3, 384, 640
    _say("kernel copies integer bit-exact out=%s" % out_dtype)
    d, perm, chunks, order = _small_ag(W, r, S, Q, "permutation", N, K, "bf16", out_dtype, dist="int")
    s = csg.Schedule.uniform(W, r, S, Q, "permutation", perm)
    plan = csg.Plan("ag", W * S, N, K, "bf16", out_dtype, s, cfg=_kc(copy_workgroups=5))
    c, _ = run_ag(plan, chunks, d.A, d.B, out_dtype)
    R = oracle.ag_gemm(d.A.device_array, d.B.device_array, chunks, order)
    expect = R if out_dtype == "f32" else bf16_rne_of_f64(R)
    assert np.array_equal(out_to_f64(c, out_dtype), expect)


def test_kernel_copies_with_release_delays():
    W, r, S, Q, N, K = 4, 1, 256, 4, 512, 256
    _say("kernel copies with delays")
    d, perm, chunks, order = _small_ag(W, r, S, Q, "permutation", N, K, "bf16", "bf16")
    s = csg.Schedule.uniform(W, r, S, Q, "permutation", perm)
    plan = csg.Plan("ag", W * S, N, K, "bf16", "bf16", s, cfg=_kc(copy_workgroups=8))
    delays = np.random.default_rng(5).uniform(0.0, 20.0, size=(W - 1) * Q).astype(np.float32)
    plan.set_copy_delays(delays)
    R = oracle.ag_gemm(d.A.device_array, d.B.device_array, chunks, order)
    c, landing = run_ag(plan, chunks, d.A, d.B, "bf16", poison_remote=True, repeats=2)
    assert_close(out_to_f64(c, "bf16"), R, 2e-2, "kernel copies with delays")
    assert torch.equal(landing.cpu(), to_dev(d.A.device_array).cpu())
    plan.set_copy_delays(None)
    c, _ = run_ag(plan, chunks, d.A, d.B, "bf16", poison_remote=True)
    assert_close(out_to_f64(c, "bf16"), R, 2e-2, "kernel copies, delays cleared")


@pytest.mark.parametrize("split", [1, 3])
def test_kernel_copies_repeated_calls(split):
    W, r, S, Q, N, K = 4, 0, 256, 2, 768, 512
    _say("kernel copies repeated calls split=%d" % split)
    d, perm, chunks, order = _small_ag(W, r, S, Q, "ring", N, K, "bf16", "bf16")
    s = csg.Schedule.uniform(W, r, S, Q, "ring")
    plan = csg.Plan("ag", W * S, N, K, "bf16", "bf16", s, cfg=_kc(split_k=split))
    R = oracle.ag_gemm(d.A.device_array, d.B.device_array, chunks, order)
    c, _ = run_ag(plan, chunks, d.A, d.B, "bf16", poison_remote=True, touch_remote=True, repeats=4)
    assert_close(out_to_f64(c, "bf16"), R, 2e-2, "after 4 calls")


@pytest.mark.parametrize("split", [1, 3])
def test_kernel_copies_grouped_parity(split):
    _say("kernel copies grouped split=%d" % split)
    W, E, N, K = 4, 3, 264, 256
    counts = np.array([[70, 0, 5], [0, 3, 1], [130, 0, 0], [1, 2, 300]], dtype=np.int64)
    chunks, order, gr = oracle.grouped_schedule(W, 1, counts)
    M = int(sum(gr))
    X = si.draw_matrix(114, 0, 0, (M, K), "normal", "bf16")
    B = si.draw_matrix(114, 1, 0, (E, N, K), "normal", "bf16")
    s = csg.Schedule.grouped(W, 1, counts)
    plan = csg.Plan("grouped", M, N, K, "bf16", "bf16", s, group_rows=gr, cfg=_kc(split_k=split, copy_workgroups=6))
    c, landing = run_ag(plan, chunks, X, B, "bf16", poison_remote=True)
    R = oracle.grouped_gemm(X.device_array, B.device_array, chunks, order)
    assert_close(out_to_f64(c, "bf16"), R, 2e-2, "kernel copies grouped")
    assert torch.equal(landing.cpu(), to_dev(X.device_array).cpu())


# GEMM-RS sends from the epilogue: every chunk must start on a multiple of bm
# (256 for bf16, 64 for fp32)
RS_CASES = [
    # W, r, S, Q, N, K, dtype, out, split
    (4, 1, 512, 2, 512, 320, "bf16", "bf16", 1),
    (3, 0, 128, 2, 200, 96, "f32", "f32", 1),       # ragged N
    (8, 5, 64, 1, 256, 128, "f32", "f32", 1),
    (4, 1, 512, 2, 512, 320, "bf16", "bf16", 2),
    (4, 2, 512, 2, 520, 384, "bf16", "bf16", 3),    # ragged N, split in 3
]
RS_IDS = ["W%d-r%d-S%d-Q%d-N%d-K%d-%s-%s-split%d" % c for c in RS_CASES]


def _rs_inputs(case, cfg_id=113):
    W, r, S, Q, N, K, dtype, out_dtype, split = case
    w = si.Workload(cfg_id, "rs", "rs", M=W * S, N=N, K=K, dtype=dtype, out_dtype=out_dtype, dist="normal", world=W,
                    rank=r, shard_rows=S, chunks_per_shard=Q, order="rs_ring")
    d = si.draw(w)
    chunks, order = oracle.uniform_schedule(W, r, S, Q, "rs_ring")
    s = csg.Schedule.uniform(W, r, S, Q, "rs_ring")
    plan = csg.Plan("rs", W * S, N, K, dtype, out_dtype, s, cfg=_kc(split_k=split))
    return d, chunks, order, plan


@pytest.mark.parametrize("case", RS_CASES, ids=RS_IDS)
@pytest.mark.parametrize("mode", ["overlap", "compute_only"])
def test_kernel_copies_rs_parity(case, mode):
    dtype, out_dtype = case[6], case[7]
    _say("kernel copies rs %s mode=%s" % (case, mode))
    d, chunks, order, plan = _rs_inputs(case)
    c, out = run_rs(plan, d.A, d.B, out_dtype, mode=mode, repeats=2)
    R, _, _ = oracle.gemm_rs(d.A.device_array, d.B.device_array, chunks, order)
    G = out_to_f64(c, out_dtype)
    assert_close(G, R, tol_for(out_dtype, dtype), "kernel copies rs C")
    O = out_to_f64(out, out_dtype)
    for ch in chunks:
        rows = slice(ch.row_begin, ch.row_end)
        if ch.is_local or mode == "compute_only":
            assert (O[rows] == 0).all()                  # never sent
        else:
            assert np.array_equal(O[rows], G[rows])


@pytest.mark.parametrize("case", RS_CASES[:3], ids=RS_IDS[:3])
def test_kernel_copies_rs_copy_only(case):
    """Copy-only after a compute-only call: copy workgroups move the sent chunks' rows."""
    out_dtype = case[7]
    _say("kernel copies rs copy-only %s" % (case,))
    d, chunks, order, plan = _rs_inputs(case)
    M, N = d.A.values.shape[0], d.B.values.shape[0]
    st = streams()
    a, b = to_dev(d.A.device_array), to_dev(d.B.device_array)
    c = empty_out(M, N, out_dtype)
    nan_fill_(c)
    out = empty_out(M, N, out_dtype)
    out.zero_()
    torch.cuda.synchronize()
    plan.gemm_rs(a, b, c, out, "compute_only", st.compute, st.copy)
    plan.gemm_rs(a, b, c, out, "copy_only", st.compute, st.copy)
    plan.check()
    torch.cuda.synchronize()
    G, O = out_to_f64(c, out_dtype), out_to_f64(out, out_dtype)
    for ch in chunks:
        rows = slice(ch.row_begin, ch.row_end)
        assert (O[rows] == 0).all() if ch.is_local else np.array_equal(O[rows], G[rows])


# ---------------------------------------------------------------------------------
# Full-size workloads, sampled rows
# ---------------------------------------------------------------------------------
@pytest.mark.parametrize("cfg_id", [2, 3, 4, 5])
def test_kernel_copies_full_size_sampled(cfg_id):
    w = si.WORKLOADS[cfg_id]
    d = si.draw(w)
    _say("kernel copies full size %s" % w.name)
    if w.op == "grouped":
        chunks, order, gr = oracle.grouped_schedule(w.world, w.rank, d.counts)
        s = csg.Schedule.grouped(w.world, w.rank, d.counts)
    else:
        gr = None
        chunks, order = oracle.uniform_schedule(w.world, w.rank, w.shard_rows, w.chunks_per_shard, w.order, d.perm)
        s = csg.Schedule.uniform(w.world, w.rank, w.shard_rows, w.chunks_per_shard, w.order, d.perm)
    plan = csg.Plan(w.op, w.M, w.N, w.K, w.dtype, w.out_dtype, s, group_rows=gr, cfg={"copy_backend": "kernel"})
    if d.delays_us is not None:
        plan.set_copy_delays(d.delays_us)
    rows = sample_rows(chunks, extra=24, seed=cfg_id, M=w.M)
    tol = tol_for(w.out_dtype, w.dtype)
    if w.op == "rs":
        c, out = run_rs(plan, d.A, d.B, w.out_dtype)
        R, _, _ = oracle.gemm_rs(d.A.device_array, d.B.device_array, chunks, order, row_subset=rows)
        G = out_to_f64(c[rows], w.out_dtype)
        assert_close(G, R[rows], tol, w.name)
        O = out_to_f64(out[rows], w.out_dtype)
        remote = np.array([not next(ch for ch in chunks if ch.row_begin <= r < ch.row_end).is_local for r in rows])
        assert np.array_equal(O[remote], G[remote])
        assert (O[~remote] == 0).all()
        return
    c, landing = run_ag(plan, chunks, d.A, d.B, w.out_dtype, poison_remote=True)
    if w.op == "grouped":
        R = oracle.grouped_gemm(d.A.device_array, d.B.device_array, chunks, order, row_subset=rows)
    else:
        R = oracle.ag_gemm(d.A.device_array, d.B.device_array, chunks, order, row_subset=rows)
    assert_close(out_to_f64(c[rows], w.out_dtype), R[rows], tol, w.name)
    assert torch.equal(landing, to_dev(d.A.device_array))
