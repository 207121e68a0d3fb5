"""GPU parity of chunk-scheduled ring attention (csg_ring_attn) against the CPU oracle,
through the C ABI.

The oracle is fp64 softmax attention over all keys (oracle.attention). The kernel
reads bf16 inputs, accumulates scores and outputs in fp32 with bf16 probabilities, and
stores bf16 outputs; outputs and log-sum-exps are compared with the max relative
error metric used for the GEMMs (<= 2e-2 with bf16). Remote key/value rows start as
NaN and sit in the caches before the call, so a tile that read a chunk before it
landed, or through a stale line, would put NaN into the output.
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
    from gpu_util import DEV, assert_close, nan_fill_, streams, to_dev


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _bf16(t):
    return si.bf16_bits_to_f32(t.cpu().numpy().view(np.uint16)).astype(np.float64)


def _case(W, r, Sh, Qc, kind, Sq, H, Hkv, cfg_id=141, dist="normal"):
    w = si.Workload(cfg_id, "attn", "attn", M=Sq, N=0, K=0, dtype="bf16", out_dtype="bf16", dist=dist, world=W,
                    rank=r, shard_rows=Sh, chunks_per_shard=Qc, order=kind,
                    extras={"heads": H, "kv_heads": Hkv, "head_dim": 128})
    d = si.draw(w)
    perm = si.draw_permutation(cfg_id, 0, (W - 1) * Qc) if kind == "permutation" else None
    chunks, order = oracle.uniform_schedule(W, r, Sh, Qc, kind, perm)
    s = csg.Schedule.uniform(W, r, Sh, Qc, kind, perm)
    return w, d, chunks, order, s


def run_attn(plan, d, chunks, mode="overlap", repeats=1, poison=True, st=None):
    st = st or streams()
    q = to_dev(d.A.device_array)
    k_st, v_st = to_dev(d.B.device_array), to_dev(d.V.device_array)
    k_l, v_l = k_st.clone(), v_st.clone()
    if mode != "compute_only":
        for ch in chunks:
            if not ch.is_local:
                if poison:
                    nan_fill_(k_l[ch.row_begin:ch.row_end])
                    nan_fill_(v_l[ch.row_begin:ch.row_end])
                else:
                    k_l[ch.row_begin:ch.row_end].zero_()
                    v_l[ch.row_begin:ch.row_end].zero_()
        _ = k_l.sum().item() + v_l.sum().item()     # remote rows now sit in the caches
    Sq, H, D = d.A.values.shape
    o = torch.empty((Sq, H, D), dtype=torch.int16, device=DEV)
    nan_fill_(o)
    lse = torch.full((H, Sq), float("nan"), dtype=torch.float32, device=DEV)
    torch.cuda.synchronize()
    for _ in range(repeats):
        plan.ring_attn(q, k_l, v_l, k_st, v_st, o, lse, mode, st.compute, st.copy)
    plan.check()
    torch.cuda.synchronize()
    if mode == "overlap":
        assert torch.equal(k_l, k_st) and torch.equal(v_l, v_st)    # every chunk landed
    return o, lse


def _check(o, lse, d, rows=None):
    Q = d.A.values if rows is None else d.A.values[rows]
    R, L = oracle.attention(Q, d.B.values, d.V.values)
    G = _bf16(o) if rows is None else _bf16(o)[rows]
    GL = lse.cpu().numpy().astype(np.float64)
    GL = GL if rows is None else GL[:, rows]
    assert_close(G.reshape(G.shape[0], -1), R.reshape(R.shape[0], -1), 2e-2, "attention output")
    assert_close(GL, L, 2e-2, "log-sum-exp")


ATTN_CASES = [
    # W, r, Sh, Qc, kind, Sq, H, Hkv
    (2, 0, 128, 1, "ring", 100, 4, 2),           # ragged query rows, grouped heads
    (4, 2, 256, 2, "ring", 256, 8, 8),
    (4, 1, 256, 4, "permutation", 64, 4, 1),     # 64-key chunks, one key/value head
    (8, 5, 512, 2, "swizzle1d", 384, 32, 8),     # 8B-like heads
]
ATTN_IDS = ["W%d-r%d-S%d-Q%d-%s-Sq%d-H%d-Hkv%d" % c for c in ATTN_CASES]


@pytest.mark.parametrize("case", ATTN_CASES, ids=ATTN_IDS)
@pytest.mark.parametrize("mode", ["overlap", "compute_only"])
def test_ring_attention_parity(case, mode):
    W, r, Sh, Qc, kind, Sq, H, Hkv = case
    _say("ring attention %s mode=%s" % (case, mode))
    w, d, chunks, order, s = _case(W, r, Sh, Qc, kind, Sq, H, Hkv)
    plan = csg.AttnPlan(H, Hkv, 128, Sq, s, cfg={"timeout_ms": 1000})
    o, lse = run_attn(plan, d, chunks, mode=mode)
    _check(o, lse, d)


@pytest.mark.parametrize("growing", [True, False], ids=["growing", "shrinking"])
def test_ring_attention_scores_drifting_across_chunks(growing):
    """Key rows of the chunk at arrival position p are scaled by 1 + 2p (growing) or by
    1 + 2 (n - 1 - p) (shrinking), so the row maxima rise by far more than the softmax's
    running reference tolerates at every chunk (the reference has to move, and the
    accumulated sums be rescaled, again and again), or fall steeply (later weights
    underflow against an early maximum). The scaled keys are rounded to bf16 and the
    oracle sees exactly those values."""
    _say("ring attention drifting scores growing=%s" % growing)
    W, r, Sh, Qc, kind, Sq, H, Hkv = 4, 1, 256, 2, "ring", 256, 4, 2
    w, d, chunks, order, s = _case(W, r, Sh, Qc, kind, Sq, H, Hkv, cfg_id=143)
    n = len(order)
    kv = d.B.values.copy()
    for p, c in enumerate(order):
        ch = chunks[int(c)]
        f = 1 + 2 * (p if growing else n - 1 - p)
        kv[ch.row_begin:ch.row_end] *= f
    bits = si.f32_to_bf16_bits(kv)
    d.B = si.Matrix(values=si.bf16_bits_to_f32(bits), dtype="bf16", bits=bits)
    plan = csg.AttnPlan(H, Hkv, 128, Sq, s, cfg={"timeout_ms": 1000})
    o, lse = run_attn(plan, d, chunks)
    _check(o, lse, d)


def test_ring_attention_repeated_calls():
    _say("ring attention repeated calls")
    w, d, chunks, order, s = _case(4, 3, 256, 2, "ring", 200, 8, 4)
    plan = csg.AttnPlan(8, 4, 128, 200, s, cfg={"timeout_ms": 1000})
    o, lse = run_attn(plan, d, chunks, repeats=4)
    _check(o, lse, d)


def test_ring_attention_full_size_sampled():
    w = si.WORKLOADS[7]
    d = si.draw(w)
    _say("ring attention full size %s" % w.name)
    chunks, order = oracle.uniform_schedule(w.world, w.rank, w.shard_rows, w.chunks_per_shard, w.order)
    s = csg.Schedule.uniform(w.world, w.rank, w.shard_rows, w.chunks_per_shard, w.order)
    e = w.extras
    plan = csg.AttnPlan(e["heads"], e["kv_heads"], e["head_dim"], w.M, s)
    o, lse = run_attn(plan, d, chunks)
    rows = sorted(set([0, 1, 127, 128, w.M - 1] + list(np.random.default_rng(7).integers(0, w.M, 27))))
    _check(o, lse, d, rows=rows)


def test_ring_attention_withheld_chunk_times_out_and_plan_recovers():
    """The host releases the last remote key/value chunk long after the kernel's (tiny)
    wait bound: the kernel must give up with a timeout that names that chunk and exit
    normally, and the plan must then run correctly without the delay."""
    _say("ring attention withheld chunk")
    W, r, Sh, Qc, kind, Sq, H, Hkv = 2, 0, 256, 2, "ring", 128, 4, 2
    w, d, chunks, order, s = _case(W, r, Sh, Qc, kind, Sq, H, Hkv, cfg_id=144)
    plan = csg.AttnPlan(H, Hkv, 128, Sq, s, cfg={"timeout_ms": 20})
    plan.set_copy_delays([0.0, 300000.0])            # second remote chunk 300 ms late
    with pytest.raises(csg.CsgError) as ei:
        run_attn(plan, d, chunks)
    assert ei.value.status == csg.CSG_ERR_TIMEOUT
    assert ei.value.diag.chunk == order[-1]
    torch.cuda.synchronize()
    plan.set_copy_delays(None)
    o, lse = run_attn(plan, d, chunks)
    _check(o, lse, d)
