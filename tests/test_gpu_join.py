"""csg_plan_join and copy-only calls (GPU, through the C ABI).

A copy-only call returns once its copies are issued; csg_plan_join then makes a stream
wait for them on the device, so work queued behind the join reads the copied rows
without a host wait. For GEMM-RS the join follows the copy-outs that complete after the
call returns. The MFMA microbenchmark returns a rate below the dense bf16 peak.
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


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.mark.parametrize("delays", [False, True])
def test_copy_only_then_join_orders_a_stream_after_the_copies(delays):
    _say("copy-only + join, delays=%s" % delays)
    W, R, S, Q, N, K = 4, 2, 256, 2, 256, 1024
    w = si.Workload(161, "join", "ag", M=W * S, N=N, K=K, dtype="bf16", out_dtype="bf16", dist="normal",
                    world=W, rank=R, shard_rows=S, chunks_per_shard=Q, order="ring")
    d = si.draw(w)
    chunks, order = oracle.uniform_schedule(W, R, S, Q, "ring")
    stage = to_dev(d.A.device_array)
    landing = stage.clone()
    for c in chunks:
        if not c.is_local:
            nan_fill_(landing[c.row_begin:c.row_end])
    b = to_dev(d.B.device_array)
    out = empty_out(W * S, N, "bf16")
    st = streams()
    s = csg.Schedule.uniform(W, R, S, Q, "ring")
    plan = csg.Plan("ag", W * S, N, K, "bf16", "bf16", s, cfg={"timeout_ms": 2000})
    if delays:
        plan.set_copy_delays(np.full(sum(1 for c in chunks if not c.is_local), 30.0, dtype=np.float32))
    reader = torch.cuda.Stream(device=DEV)
    torch.cuda.synchronize()
    plan.ag_gemm(landing, stage, b, out, "copy_only", st.compute, st.copy)
    plan.join(reader)
    with torch.cuda.stream(reader):
        snap = landing.clone()       # ordered after the copies on the device
    plan.check()
    torch.cuda.synchronize()
    assert torch.equal(snap, stage)
    # the plan runs on afterwards, from the landed rows
    plan.ag_gemm(landing, stage, b, out, "compute_only", st.compute, st.copy)
    plan.check()
    torch.cuda.synchronize()
    ref = oracle.ag_gemm(d.A.device_array, d.B.device_array, chunks, order)
    assert_close(out_to_f64(out, "bf16"), ref, tol_for("bf16", "bf16"), "compute-only after copy-only")


def test_join_follows_gemm_rs_copy_outs():
    _say("GEMM-RS overlap + join")
    W, R, S, Q, N, K = 4, 1, 256, 2, 512, 512
    w = si.Workload(162, "join-rs", "rs", M=W * S, N=N, K=K, dtype="bf16", out_dtype="bf16", dist="normal",
                    world=W, rank=R, shard_rows=S, chunks_per_shard=Q, order="rs_ring")
    d = si.draw(w)
    chunks, order = oracle.uniform_schedule(W, R, S, Q, "rs_ring")
    a = to_dev(d.A.device_array)
    b = to_dev(d.B.device_array)
    c = empty_out(W * S, N, "bf16")
    outgoing = empty_out(W * S, N, "bf16")
    nan_fill_(outgoing)
    st = streams()
    s = csg.Schedule.uniform(W, R, S, Q, "rs_ring")
    plan = csg.Plan("rs", W * S, N, K, "bf16", "bf16", s, cfg={"timeout_ms": 2000})
    torch.cuda.synchronize()
    for _ in range(3):
        plan.gemm_rs(a, b, c, outgoing, "overlap", st.compute, st.copy)
        plan.join(st.compute)
        with torch.cuda.stream(st.compute):
            snap = outgoing.clone()  # after the kernel and the copy-outs, no host wait
    plan.check()
    torch.cuda.synchronize()
    ref = oracle.gemm_rows(d.A.device_array, d.B.device_array, range(W * S))
    got = out_to_f64(snap, "bf16")
    sent = np.zeros(W * S, dtype=bool)
    for ch in chunks:
        if not ch.is_local:
            sent[ch.row_begin:ch.row_end] = True
    assert_close(got[sent], ref[sent], tol_for("bf16", "bf16"), "outgoing rows after join")
    assert np.isnan(got[~sent]).all()          # the own shard is never sent


def test_mfma_microbenchmark_is_below_the_dense_peak():
    _say("MFMA microbenchmark")
    tf, ms, ghz = csg.csg_measure_mfma_peak(0, 800)
    assert 100.0 < tf < 2600.0, tf
    assert ms > 0.0
    assert 0.5 < ghz < 3.0, ghz
