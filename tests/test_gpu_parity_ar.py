"""GPU parity of GEMM + AllReduce on one rank (csg_gemm_ar) against the CPU oracle,
through the C ABI.

Checked after each call: the all-reduced own rows of C (this rank's partial plus the
other ranks' partial sums, added in the kernel's epilogue) against the oracle within
the tolerances of the other ops; the other shards' rows of C equal, bit for bit, the
reduced rows their owners sent; the outgoing buffer holds this rank's partial of
every non-local chunk (against the oracle) and, bit for bit, its reduced own rows.
Integer inputs make every sum exact, so those runs compare bit for bit.
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
    from gpu_util import assert_close, empty_out, nan_fill_, out_to_f64, sample_rows, streams, to_dev, tol_for


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _inputs(W, r, S, Q, N, K, dtype, out_dtype, dist="normal", cfg_id=131):
    w = si.Workload(cfg_id, "ar", "ar", M=W * S, N=N, K=K, dtype=dtype, out_dtype=out_dtype, dist=dist, world=W,
                    rank=r, shard_rows=S, chunks_per_shard=Q, order="rs_ring")
    d = si.draw(w)
    chunks, order = oracle.uniform_schedule(W, r, S, Q, "rs_ring")
    return w, d, chunks, order


def run_ar(plan, d, out_dtype, mode="overlap", repeats=1, st=None):
    M, N = d.A.values.shape[0], d.B.values.shape[0]
    st = st or streams()
    a, b = to_dev(d.A.device_array), to_dev(d.B.device_array)
    p_stage = to_dev(d.partials.device_array)
    p_land = p_stage.clone() if mode == "compute_only" else torch.zeros_like(p_stage)
    if mode != "compute_only":
        nan_fill_(p_land)                           # a partial read before it landed would show as NaN
    red = to_dev(d.reduced.device_array)
    c = empty_out(M, N, out_dtype)
    nan_fill_(c)
    out = empty_out(M, N, out_dtype)
    out.zero_()
    torch.cuda.synchronize()
    for _ in range(repeats):
        plan.gemm_ar(a, b, c, out, p_stage, p_land, red, mode, st.compute, st.copy)
    plan.check()
    torch.cuda.synchronize()
    return c, out


def _check(c, out, d, chunks, order, out_dtype, dtype, mode, exact=False):
    R, Rout, _ = oracle.gemm_ar(d.A.device_array, d.B.device_array, chunks, order, d.partials.values,
                                d.reduced.values)
    G, O = out_to_f64(c, out_dtype), out_to_f64(out, out_dtype)
    tol = tol_for(out_dtype, dtype)
    red_bits = d.reduced.device_array
    c_bits = c.cpu().numpy().view(np.uint16) if out_dtype == "bf16" else c.cpu().numpy()
    for ch in chunks:
        rows = slice(ch.row_begin, ch.row_end)
        if ch.is_local:
            if exact:
                assert np.array_equal(G[rows], R[rows])
            else:
                assert_close(G[rows], R[rows], tol, "reduced own rows")
            if mode == "overlap":
                assert np.array_equal(O[rows], G[rows])           # the reduced chunk was sent
            else:
                assert (O[rows] == 0).all()
        elif mode == "overlap":
            assert np.array_equal(c_bits[rows], red_bits[rows])   # arrived from its owner
            if exact:
                assert np.array_equal(O[rows], Rout[rows])
            else:
                assert_close(O[rows], Rout[rows], tol, "sent partial rows")
        else:                                                   # compute-only: the partial stays in C
            assert_close(G[rows], Rout[rows], tol, "partial rows")
            assert (O[rows] == 0).all()


AR_CASES = [
    # W, r, S, Q, N, K, dtype, out
    (4, 1, 256, 2, 512, 320, "bf16", "bf16"),
    (8, 5, 256, 1, 256, 128, "bf16", "bf16"),      # 8 ranks, one chunk per shard
    (3, 0, 128, 2, 200, 96, "f32", "f32"),         # ragged N, fp32 (64-row tiles)
    (2, 1, 512, 4, 520, 192, "bf16", "f32"),       # ragged N, own shard last rows, fp32 out
    (4, 2, 512, 2, 520, 192, "bf16", "bf16"),      # ragged N, bf16 out: two own row tiles, 3 peers
]
AR_IDS = ["W%d-r%d-S%d-Q%d-N%d-K%d-%s-%s" % c for c in AR_CASES]


@pytest.mark.parametrize("case", AR_CASES, ids=AR_IDS)
@pytest.mark.parametrize("mode", ["overlap", "compute_only"])
def test_ar_small_parity(case, mode):
    W, r, S, Q, N, K, dtype, out_dtype = case
    _say("ar small %s mode=%s" % (case, mode))
    w, d, chunks, order = _inputs(W, r, S, Q, N, K, dtype, out_dtype)
    s = csg.Schedule.uniform(W, r, S, Q, "rs_ring")
    plan = csg.Plan("ar", W * S, N, K, dtype, out_dtype, s, cfg={"timeout_ms": 1000})
    c, out = run_ar(plan, d, out_dtype, mode=mode, repeats=2)
    _check(c, out, d, chunks, order, out_dtype, dtype, mode)


def test_ar_integer_inputs_bit_exact():
    W, r, S, Q, N, K = 4, 2, 256, 2, 384, 640
    _say("ar integer bit-exact")
    w, d, chunks, order = _inputs(W, r, S, Q, N, K, "bf16", "f32", dist="int")
    s = csg.Schedule.uniform(W, r, S, Q, "rs_ring")
    plan = csg.Plan("ar", W * S, N, K, "bf16", "f32", s, cfg={"timeout_ms": 1000})
    c, out = run_ar(plan, d, "f32")
    _check(c, out, d, chunks, order, "f32", "bf16", "overlap", exact=True)


def test_ar_copy_only_sends_what_c_holds():
    W, r, S, Q, N, K = 4, 3, 256, 2, 256, 128
    _say("ar copy-only")
    w, d, chunks, order = _inputs(W, r, S, Q, N, K, "bf16", "bf16")
    s = csg.Schedule.uniform(W, r, S, Q, "rs_ring")
    plan = csg.Plan("ar", W * S, N, K, "bf16", "bf16", s, cfg={"timeout_ms": 1000})
    st = streams()
    c, out = run_ar(plan, d, "bf16", st=st)
    held = c.clone()
    out2 = torch.zeros_like(out)
    p_stage = to_dev(d.partials.device_array)
    p_land = torch.zeros_like(p_stage)
    red = to_dev(d.reduced.device_array)
    torch.cuda.synchronize()
    plan.gemm_ar(to_dev(d.A.device_array), to_dev(d.B.device_array), c, out2, p_stage, p_land, red, "copy_only",
                 st.compute, st.copy)
    plan.check()
    torch.cuda.synchronize()
    assert torch.equal(out2, held)                 # every chunk sent, as c held it
    assert torch.equal(c, held)                    # the arriving reduced rows equal what was there
    assert torch.equal(p_land, p_stage)            # every partial landed


def test_ar_full_size_sampled():
    w = si.WORKLOADS[6]
    d = si.draw(w)
    _say("ar full size %s" % w.name)
    chunks, order = oracle.uniform_schedule(w.world, w.rank, w.shard_rows, w.chunks_per_shard, w.order)
    s = csg.Schedule.uniform(w.world, w.rank, w.shard_rows, w.chunks_per_shard, w.order)
    plan = csg.Plan("ar", w.M, w.N, w.K, w.dtype, w.out_dtype, s)
    c, out = run_ar(plan, d, w.out_dtype)
    rows = sample_rows(chunks, extra=24, seed=6, M=w.M)
    R, Rout, _ = oracle.gemm_ar(d.A.device_array, d.B.device_array, chunks, order, d.partials.values,
                                d.reduced.values, row_subset=rows)
    own = [i for i in rows if w.rank * w.shard_rows <= i < (w.rank + 1) * w.shard_rows]
    other = [i for i in rows if i not in own]
    G, O = out_to_f64(c[rows], w.out_dtype), out_to_f64(out[rows], w.out_dtype)
    idx = {row: k for k, row in enumerate(rows)}
    assert_close(G[[idx[i] for i in own]], R[own], 2e-2, "reduced own rows")
    assert np.array_equal(c.cpu().numpy().view(np.uint16)[other], d.reduced.device_array[other])
    assert_close(O[[idx[i] for i in other]], Rout[other], 2e-2, "sent partial rows")
    assert np.array_equal(O[[idx[i] for i in own]], G[[idx[i] for i in own]])


def _sweep_case(i):
    g = np.random.default_rng([137, i])
    dtype, out_dtype = [("bf16", "bf16"), ("bf16", "bf16"), ("bf16", "f32"), ("f32", "f32")][int(g.integers(0, 4))]
    bm = 256 if dtype == "bf16" else 64          # the own shard starts and ends on tile rows
    W = int(g.integers(2, 9))
    r = int(g.integers(0, W))
    S = bm * int(g.integers(1, 4 if dtype == "bf16" else 9))
    Q = [q for q in (1, 2, 4, 8) if S % q == 0][int(g.integers(0, 4))]
    step = 64 if dtype == "bf16" else 16
    K = step * int(g.integers(1, 9))
    N = 4 * int(g.integers(1, 150))
    mode = "compute_only" if g.random() < 0.25 else "overlap"
    dist = "int" if g.random() < 0.25 else "normal"
    return W, r, S, Q, N, K, dtype, out_dtype, mode, dist


AR_SWEEP = list(range(12))


@pytest.mark.parametrize("i", AR_SWEEP, ids=lambda i: "%d-W%d-r%d-S%d-Q%d-N%d-K%d-%s-%s-%s-%s" % ((i,) + _sweep_case(i)))
def test_ar_sweep_parity(i):
    """Seeded sweep: ranks, own-shard rows (multiples of the tile height), chunks per
    shard, N, K, dtypes, mode and input distribution drawn per case; integer inputs are
    compared bit for bit."""
    W, r, S, Q, N, K, dtype, out_dtype, mode, dist = _sweep_case(i)
    _say("ar sweep %d %s" % (i, (W, r, S, Q, N, K, dtype, out_dtype, mode, dist)))
    w, d, chunks, order = _inputs(W, r, S, Q, N, K, dtype, out_dtype, dist=dist, cfg_id=1370 + i)
    s = csg.Schedule.uniform(W, r, S, Q, "rs_ring")
    plan = csg.Plan("ar", W * S, N, K, dtype, out_dtype, s, cfg={"timeout_ms": 1000})
    c, out = run_ar(plan, d, out_dtype, mode=mode)
    _check(c, out, d, chunks, order, out_dtype, dtype, mode, exact=(dist == "int" and out_dtype == "f32"))
