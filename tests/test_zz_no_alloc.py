"""csg_ag_gemm_noalloc: the all-gather GEMM on the library's static device scratch,
checked against csg_ag_gemm on a plan with the same chunk realization (copy
workgroups), and against the oracle. Two calls in a row on one device, the second with
a smaller input, so the second reuses the scratch the first filled."""
import sys

import numpy as np
import pytest

import oracle
import paper_2601_20595_amd as csg
import seeded_inputs as si

torch = pytest.importorskip("torch")

if torch.cuda.is_available():
    from gpu_util import DEV, assert_close, empty_out, nan_fill_, out_to_f64, streams, to_dev, tol_for


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _case(cid, W, R, S, Q, N, K, dtype, out_dtype, kind):
    dist = "normal" if dtype == "bf16" else "uniform"
    w = si.Workload(cid, "noalloc", "ag", M=W * S, N=N, K=K, dtype=dtype, out_dtype=out_dtype, dist=dist,
                    world=W, rank=R, shard_rows=S, chunks_per_shard=Q, order=kind)
    d = si.draw(w)
    perm = si.draw_permutation(cid, 0, (W - 1) * Q) if kind == "permutation" else None
    chunks, order = oracle.uniform_schedule(W, R, S, Q, kind, perm)
    return w, d, perm, chunks, order


def _poisoned_landing(stage, chunks):
    landing = stage.clone()
    for c in chunks:
        if not c.is_local:
            nan_fill_(landing[c.row_begin:c.row_end])
    return landing


@pytest.mark.gpu
def test_noalloc_matches_the_plan_entry_point_on_two_calls():
    cases = [  # the second call is smaller than the first
        (171, 8, 3, 512, 2, 1024, 1024, "bf16", "bf16", "permutation", "overlap"),
        (172, 4, 1, 256, 2, 512, 512, "bf16", "bf16", "ring", "overlap"),
    ]
    st = streams()
    for cid, W, R, S, Q, N, K, dt, odt, kind, mode in cases:
        _say("noalloc case %d: W=%d S=%d Q=%d N=%d K=%d %s %s" % (cid, W, S, Q, N, K, kind, mode))
        w, d, perm, chunks, order = _case(cid, W, R, S, Q, N, K, dt, odt, kind)
        M = W * S
        stage = to_dev(d.A.device_array)
        b = to_dev(d.B.device_array)
        sched = csg.Schedule.uniform(W, R, S, Q, kind, perm)
        # the allocation-free call
        land_na = _poisoned_landing(stage, chunks)
        c_na = empty_out(M, N, odt)
        nan_fill_(c_na)
        torch.cuda.synchronize()
        csg.csg_ag_gemm_noalloc(sched, M, N, K, dt, odt, land_na, stage, b, c_na, mode, copy_workgroups=16,
                                device=0, stream=st.compute)
        torch.cuda.synchronize()
        # the existing entry point, same chunk realization
        plan = csg.Plan("ag", M, N, K, dt, odt, sched, cfg={"copy_backend": "kernel", "copy_workgroups": 16})
        land_p = _poisoned_landing(stage, chunks)
        c_p = empty_out(M, N, odt)
        plan.ag_gemm(land_p, stage, b, c_p, mode, st.compute, st.copy)
        plan.check()
        torch.cuda.synchronize()
        plan.close()
        assert torch.equal(land_na, stage), "the copy workgroups left landing rows unfilled"
        got, want = out_to_f64(c_na, odt), out_to_f64(c_p, odt)
        ref = oracle.ag_gemm(d.A.device_array, d.B.device_array, chunks, order)
        assert_close(got, ref, tol_for(dt, odt), "noalloc vs oracle, case %d" % cid)
        assert_close(want, ref, tol_for(dt, odt), "plan vs oracle, case %d" % cid)
        # same kernel, same tile K order: the two entry points agree bit for bit
        assert np.array_equal(got, want), "noalloc and plan outputs differ, case %d" % cid


@pytest.mark.gpu
def test_noalloc_modes_and_fp32():
    st = streams()
    # compute-only (the landing buffer already full), fp32 in and out
    w, d, perm, chunks, order = _case(173, 2, 0, 128, 2, 256, 256, "f32", "f32", "permutation")
    M, N, K = 256, 256, 256
    a = to_dev(d.A.device_array)
    b = to_dev(d.B.device_array)
    c = empty_out(M, N, "f32")
    sched = csg.Schedule.uniform(2, 0, 128, 2, "permutation", perm)
    _say("noalloc compute-only fp32")
    csg.csg_ag_gemm_noalloc(sched, M, N, K, "f32", "f32", a, a, b, c, "compute_only", device=0, stream=st.compute)
    torch.cuda.synchronize()
    ref = oracle.ag_gemm(d.A.device_array, d.B.device_array, chunks, order)
    assert_close(out_to_f64(c, "f32"), ref, tol_for("f32", "f32"), "noalloc compute-only fp32")
    # copy-only: the copy workgroups alone move the remote rows, then overlap again
    _say("noalloc copy-only then overlap, bf16")
    w, d, perm, chunks, order = _case(174, 4, 2, 256, 4, 512, 1024, "bf16", "bf16", "ring")
    M, N, K = 1024, 512, 1024
    stage = to_dev(d.A.device_array)
    b = to_dev(d.B.device_array)
    land = _poisoned_landing(stage, chunks)
    c = empty_out(M, N, "bf16")
    sched = csg.Schedule.uniform(4, 2, 256, 4, "ring")
    csg.csg_ag_gemm_noalloc(sched, M, N, K, "bf16", "bf16", land, stage, b, c, "copy_only", copy_workgroups=8,
                            device=0, stream=st.compute)
    torch.cuda.synchronize()
    assert torch.equal(land, stage)
    land2 = _poisoned_landing(stage, chunks)
    csg.csg_ag_gemm_noalloc(sched, M, N, K, "bf16", "bf16", land2, stage, b, c, "overlap", copy_workgroups=8,
                            device=0, stream=st.compute)
    torch.cuda.synchronize()
    ref = oracle.ag_gemm(d.A.device_array, d.B.device_array, chunks, order)
    assert_close(out_to_f64(c, "bf16"), ref, tol_for("bf16", "bf16"), "noalloc overlap after copy-only")


def test_noalloc_rejects_inputs_beyond_the_scratch_before_queueing():
    """Host-side checks only: dummy device addresses are never dereferenced."""
    big = csg.Schedule.uniform(2, 0, 4096 * 2, 4096, "ring")          # 8192 chunks
    ptr = 1 << 20
    with pytest.raises(csg.CsgError) as e:
        csg.csg_ag_gemm_noalloc(big, 4096 * 4, 256, 64, "bf16", "bf16", ptr, ptr, ptr, ptr, "overlap")
    assert e.value.status == csg.CSG_ERR_UNSUPPORTED and "4096 chunks" in str(e.value)
    wide = csg.Schedule.uniform(1, 0, 65536, 1, "ring")                # 256 x 257 tiles
    with pytest.raises(csg.CsgError) as e:
        csg.csg_ag_gemm_noalloc(wide, 65536, 65536 + 256, 64, "bf16", "bf16", ptr, ptr, ptr, ptr, "compute_only")
    assert e.value.status == csg.CSG_ERR_UNSUPPORTED and "no-alloc scratch" in str(e.value)
    s = csg.Schedule.uniform(2, 0, 128, 2, "ring")
    with pytest.raises(csg.CsgError) as e:                              # M differs from the chunks' rows
        csg.csg_ag_gemm_noalloc(s, 100, 64, 64, "bf16", "bf16", ptr, ptr, ptr, ptr, "overlap")
    assert e.value.status == csg.CSG_ERR_INVALID
    with pytest.raises(csg.CsgError) as e:                              # K not a multiple of 64
        csg.csg_ag_gemm_noalloc(s, 256, 64, 60, "bf16", "bf16", ptr, ptr, ptr, ptr, "overlap")
    assert e.value.status == csg.CSG_ERR_UNSUPPORTED
