"""Back-to-back all-gather GEMM calls gathering into different landing buffers (GPU,
through the C ABI).

A call's copy of a chunk must wait only for kernels that read the same landing rows: for
the same buffer, until the kernel that read it last has finished reading that chunk; for
a buffer overlapping another one, until that buffer's last reader has finished reading
every chunk; for a disjoint buffer, for nothing. Consecutive calls take different inputs
(three sets that share their local rows and differ in the remote ones) and write
separate outputs, so a copy that overwrote rows a kernel was still reading would show in
that kernel's output.
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
    from gpu_util import DEV, assert_close, empty_out, nan_fill_, out_to_f64, streams, to_dev, tol_for

W, R, S, Q, KIND, N, K = 4, 1, 512, 2, "ring", 512, 2048


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _inputs(n_sets):
    """n_sets inputs A_k sharing the local shard's rows (every call multiplies by the
    first set's B)."""
    chunks, order = oracle.uniform_schedule(W, R, S, Q, KIND)
    sets = []
    for k in range(n_sets):
        w = si.Workload(151, "landing", "ag", M=W * S, N=N, K=K, dtype="bf16", out_dtype="bf16", dist="normal",
                        world=W, rank=R, shard_rows=S, chunks_per_shard=Q, order=KIND)
        d = si.draw(w, rep=k)
        sets.append(d)
    base = sets[0].A.device_array
    for d in sets[1:]:
        bits = d.A.device_array.copy()
        bits[R * S:(R + 1) * S] = base[R * S:(R + 1) * S]
        d.A = si.Matrix(values=si.bf16_bits_to_f32(bits), dtype="bf16", bits=bits)
    return chunks, order, sets


@pytest.mark.parametrize("n_buffers", [1, 2, 3])
def test_back_to_back_calls_into_landing_buffers_in_turn(n_buffers):
    _say("landing buffers in turn: %d" % n_buffers)
    chunks, order, sets = _inputs(3)
    M = W * S
    st = streams()
    b = to_dev(sets[0].B.device_array)
    stage = [to_dev(d.A.device_array) for d in sets]
    landings = []
    for _ in range(n_buffers):
        l = stage[0].clone()
        for c in chunks:
            if not c.is_local:
                nan_fill_(l[c.row_begin:c.row_end])
        landings.append(l)
    calls = 7
    outs = [empty_out(M, N, "bf16") for _ in range(calls)]
    for o in outs:
        nan_fill_(o)
    s = csg.Schedule.uniform(W, R, S, Q, KIND)
    plan = csg.Plan("ag", M, N, K, "bf16", "bf16", s, cfg={"timeout_ms": 2000})
    torch.cuda.synchronize()
    for i in range(calls):
        plan.ag_gemm(landings[i % n_buffers], stage[i % 3], b, outs[i], "overlap", st.compute, st.copy)
    plan.check()
    torch.cuda.synchronize()
    refs = [oracle.ag_gemm(d.A.device_array, sets[0].B.device_array, chunks, order) for d in sets]
    for i in range(calls):
        assert_close(out_to_f64(outs[i], "bf16"), refs[i % 3], tol_for("bf16", "bf16"), "call %d" % i)


def test_overlapping_landing_buffers_wait_for_every_chunk():
    """Two landing buffers that are views of one allocation, S rows apart, used in turn.
    Every row of the allocation holds fixed content, and each call's input is the
    allocation's rows under its view, so the copies into either view write consistent
    data; the calls must each finish correctly (the copies into one view wait until the
    kernel that read the other view has read all of it)."""
    _say("overlapping landing buffers")
    M = W * S
    w = si.Workload(152, "landing-overlap", "ag", M=M + S, N=N, K=K, dtype="bf16", out_dtype="bf16",
                    dist="normal", world=W, rank=R, shard_rows=S, chunks_per_shard=Q, order=KIND)
    d = si.draw(w)
    chunks, order = oracle.uniform_schedule(W, R, S, Q, KIND)
    big = to_dev(d.A.device_array)                  # (M + S) x K rows of fixed content
    views = [big[0:M], big[S:S + M]]
    stages = [v.clone() for v in views]
    b = to_dev(d.B.device_array)
    st = streams()
    s = csg.Schedule.uniform(W, R, S, Q, KIND)
    plan = csg.Plan("ag", M, N, K, "bf16", "bf16", s, cfg={"timeout_ms": 2000})
    calls = 6
    outs = [empty_out(M, N, "bf16") for _ in range(calls)]
    torch.cuda.synchronize()
    for i in range(calls):
        plan.ag_gemm(views[i % 2], stages[i % 2], b, outs[i], "overlap", st.compute, st.copy)
    plan.check()
    torch.cuda.synchronize()
    bits = d.A.device_array
    refs = [oracle.ag_gemm(np.ascontiguousarray(bits[o:o + M]), d.B.device_array, chunks, order) for o in (0, S)]
    for i in range(calls):
        assert_close(out_to_f64(outs[i], "bf16"), refs[i % 2], tol_for("bf16", "bf16"), "call %d" % i)


@pytest.mark.parametrize("n_buffers", [1, 2])
def test_calls_alternating_compute_streams(n_buffers):
    """Back-to-back calls whose compute stream alternates between two streams: the
    plan's kernels must still run in call order (each call's state set is cleared by
    the previous call's kernel, and copies wait for the last reader of their rows), so
    every output matches its own inputs."""
    _say("alternating compute streams: %d landing buffers" % n_buffers)
    chunks, order, sets = _inputs(3)
    M = W * S
    sts = [streams(), streams()]
    b = to_dev(sets[0].B.device_array)
    stage = [to_dev(d.A.device_array) for d in sets]
    landings = []
    for _ in range(n_buffers):
        l = stage[0].clone()
        for c in chunks:
            if not c.is_local:
                nan_fill_(l[c.row_begin:c.row_end])
        landings.append(l)
    calls = 6
    outs = [empty_out(M, N, "bf16") for _ in range(calls)]
    for o in outs:
        nan_fill_(o)
    s = csg.Schedule.uniform(W, R, S, Q, KIND)
    plan = csg.Plan("ag", M, N, K, "bf16", "bf16", s, cfg={"timeout_ms": 2000})
    torch.cuda.synchronize()
    for i in range(calls):
        st = sts[i % 2]
        plan.ag_gemm(landings[i % n_buffers], stage[i % 3], b, outs[i], "overlap", st.compute, st.copy)
    plan.check()
    torch.cuda.synchronize()
    refs = [oracle.ag_gemm(d.A.device_array, sets[0].B.device_array, chunks, order) for d in sets]
    for i in range(calls):
        assert_close(out_to_f64(outs[i], "bf16"), refs[i % 3], tol_for("bf16", "bf16"), "call %d" % i)


def test_copy_only_call_on_a_busy_stream_then_other_streams():
    """A copy-only call queues a prologue (it clears a per-call state set) and no kernel.
    Queued on a stream that is still busy with other work, that prologue runs late; the
    calls that follow on other compute streams must wait for it, or it would clear the
    state of a kernel already running. Every overlap call's output must match its inputs."""
    _say("copy-only call on a busy stream, then calls on two other streams")
    chunks, order, sets = _inputs(3)
    M = W * S
    sts = [streams(), streams(), streams()]
    b = to_dev(sets[0].B.device_array)
    stage = [to_dev(d.A.device_array) for d in sets]
    landing = stage[0].clone()
    modes = ["overlap", "copy_only", "overlap", "overlap", "copy_only", "overlap", "overlap"]
    outs = [empty_out(M, N, "bf16") for _ in modes]
    for o in outs:
        nan_fill_(o)
    s = csg.Schedule.uniform(W, R, S, Q, KIND)
    plan = csg.Plan("ag", M, N, K, "bf16", "bf16", s, cfg={"timeout_ms": 2000})
    x = torch.randn(2048, 2048, device=DEV)
    torch.cuda.synchronize()
    for i, mode in enumerate(modes):
        if mode == "copy_only":
            st = sts[2]
            with torch.cuda.stream(st.compute):
                y = x
                for _ in range(8):          # a few ms of unrelated work ahead of the prologue
                    y = torch.mm(y, x)
        else:
            st = sts[i % 2]
        plan.ag_gemm(landing, stage[i % 3], b, outs[i], mode, st.compute, st.copy)
    plan.check()
    torch.cuda.synchronize()
    refs = [oracle.ag_gemm(d.A.device_array, sets[0].B.device_array, chunks, order) for d in sets]
    for i, mode in enumerate(modes):
        if mode == "overlap":
            assert_close(out_to_f64(outs[i], "bf16"), refs[i % 3], tol_for("bf16", "bf16"), "call %d" % i)
