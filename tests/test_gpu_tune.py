"""GPU: the autotuner measures every candidate of a small search space through the C
ABI, records the ones the library rejects, and the plan it keeps computes the
oracle's result."""
import sys

import numpy as np
import pytest

import oracle
import paper_2601_20595_amd as csg
import seeded_inputs as si
from paper_2601_20595_amd import tune

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    from gpu_util import assert_close, empty_out, nan_fill_, out_to_f64, streams, to_dev


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def test_tune_ag_chunk_split_and_backends():
    W, r, S, N, K = 4, 1, 512, 512, 512
    _say("tune ag")
    w = si.Workload(121, "tune", "ag", M=W * S, N=N, K=K, dtype="bf16", out_dtype="bf16", dist="normal", world=W,
                    rank=r, shard_rows=S, chunks_per_shard=2, order="ring")
    d = si.draw(w)
    st = streams()
    staging = to_dev(d.A.device_array)
    landing = staging.clone()
    b = to_dev(d.B.device_array)
    c = empty_out(W * S, N, "bf16")
    cands = tune.search_space("ag", chunk_splits=(1, 2, 4), dispatch=(1,), split_k=(1, 2), tail=((0, 0),),
                              copy_workgroups=(16,))
    make = tune.uniform_plan_factory("ag", W * S, N, K, "bf16", "bf16", W, r, S, "ring", default_q=2)

    def call(plan, mode):
        plan.ag_gemm(landing, staging, b, c, mode, st.compute, st.copy)

    res, plan = tune.autotune(make, call, cands, steps=4, warmup=1, keep_best=True)
    assert len(res.trials) == len(cands) == 12
    assert all(t.status == "ok" and t.ms_per_step > 0 for t in res.trials)
    assert res.best_ms == min(t.ms_per_step for t in res.trials)
    # the kept plan, on fresh landing rows (remote rows poisoned), gives the oracle's C
    q = res.best.chunks_per_shard
    chunks, order = oracle.uniform_schedule(W, r, S, q, "ring")
    for ch in chunks:
        if not ch.is_local:
            nan_fill_(landing[ch.row_begin:ch.row_end])
    nan_fill_(c)
    torch.cuda.synchronize()
    call(plan, "overlap")
    plan.check()
    torch.cuda.synchronize()
    assert_close(out_to_f64(c, "bf16"), oracle.ag_gemm(d.A.device_array, d.B.device_array, chunks, order), 2e-2,
                 "tuned ag")
    plan.close()


def test_tune_rs_records_rejected_epilogue_sends():
    W, r, S, N, K = 4, 2, 512, 512, 256
    _say("tune rs")
    w = si.Workload(122, "tune", "rs", M=W * S, N=N, K=K, dtype="bf16", out_dtype="bf16", dist="normal", world=W,
                    rank=r, shard_rows=S, chunks_per_shard=2, order="rs_ring")
    d = si.draw(w)
    st = streams()
    a, b = to_dev(d.A.device_array), to_dev(d.B.device_array)
    c, out = empty_out(W * S, N, "bf16"), empty_out(W * S, N, "bf16")
    out.zero_()
    # Q = 4: 128-row chunks, which a 256-row tile would mix: the epilogue realization is rejected
    cands = tune.search_space("rs", chunk_splits=(2, 4), dispatch=(1,), split_k=(1,), tail=((0, 0),))
    make = tune.uniform_plan_factory("rs", W * S, N, K, "bf16", "bf16", W, r, S, "rs_ring", default_q=2)

    def call(plan, mode):
        plan.gemm_rs(a, b, c, out, mode, st.compute, st.copy)

    res, plan = tune.autotune(make, call, cands, steps=4, warmup=1, keep_best=True)
    status = {(t.candidate.chunks_per_shard, t.candidate.cfg_dict().get("copy_backend", 0)): t.status
              for t in res.trials}
    assert status[(4, 1)].startswith("rejected")
    assert status[(2, 1)] == "ok" and status[(2, 0)] == "ok" and status[(4, 0)] == "ok"
    chunks, order = oracle.uniform_schedule(W, r, S, res.best.chunks_per_shard, "rs_ring")
    nan_fill_(c)
    out.zero_()
    torch.cuda.synchronize()
    call(plan, "overlap")
    plan.check()
    torch.cuda.synchronize()
    R, _, _ = oracle.gemm_rs(d.A.device_array, d.B.device_array, chunks, order)
    G, O = out_to_f64(c, "bf16"), out_to_f64(out, "bf16")
    assert_close(G, R, 2e-2, "tuned rs")
    for ch in chunks:
        rows = slice(ch.row_begin, ch.row_end)
        assert (O[rows] == 0).all() if ch.is_local else np.array_equal(O[rows], G[rows])
    plan.close()
