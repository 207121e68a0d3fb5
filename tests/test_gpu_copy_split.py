"""GPU parity with chunk copies cut into pieces on several copy engines (plan field
copy_split): every byte of every chunk lands before the tiles that read it, the
product matches the oracle, and reduce-scatter copy-outs equal the finished rows.

A fresh plan's engines are idle, so the first copies of its first call are cut
(a 1 MiB chunk in two pieces, a 2,048,000-byte one in three, the last piece not a
multiple of the 64 KiB piece step); copies released one by one by the copy delays
find idle engines each time. Chunks under 1 MiB stay whole.
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
    from gpu_util import assert_close, out_to_f64, run_ag, run_rs, sample_rows, tol_for


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


AG_CASES = [
    # W, r, S, Q, N, K, copy_split, delay_us, repeats
    (4, 1, 1024, 2, 256, 1024, 4, 0.0, 1),    # 1 MiB chunks: two pieces
    (4, 2, 1000, 1, 264, 1024, 4, 0.0, 1),    # 2,048,000-byte chunks: three pieces, ragged N
    (8, 3, 512, 1, 128, 2048, 2, 40.0, 1),    # 2 MiB chunks released 40 us apart
    (4, 0, 1024, 2, 256, 1024, 2, 0.0, 3),    # back to back into one landing buffer
    (4, 0, 96, 2, 128, 512, 4, 0.0, 1),       # 48 KiB chunks: whole
]


@pytest.mark.parametrize("case", AG_CASES, ids=lambda c: "W%d-r%d-S%d-Q%d-N%d-K%d-cs%d-d%g-x%d" % c)
def test_ag_copy_split_lands_every_byte(case):
    W, r, S, Q, N, K, split, delay, repeats = case
    _say("ag copy_split %s" % (case,))
    w = si.Workload(105, "copy_split", "ag", M=W * S, N=N, K=K, dtype="bf16", out_dtype="bf16", dist="normal",
                    world=W, rank=r, shard_rows=S, chunks_per_shard=Q, order="ring")
    d = si.draw(w)
    chunks, order = oracle.uniform_schedule(W, r, S, Q, "ring")
    s = csg.Schedule.uniform(W, r, S, Q, "ring")
    plan = csg.Plan("ag", W * S, N, K, "bf16", "bf16", s, cfg={"timeout_ms": 1000, "copy_split": split})
    if delay:
        plan.set_copy_delays([delay] * ((W - 1) * Q))
    c, landing = run_ag(plan, chunks, d.A, d.B, "bf16", poison_remote=True, repeats=repeats)
    # the landing buffer was NaN in every remote row: each byte must have been copied
    assert np.array_equal(landing.cpu().numpy().view(np.uint16), d.A.bits)
    rows = sample_rows(chunks, extra=32, seed=W * 100 + r, M=W * S)
    R = oracle.ag_gemm(d.A.device_array, d.B.device_array, chunks, order, row_subset=rows)
    assert_close(out_to_f64(c[rows], "bf16"), R[rows], tol_for("bf16", "bf16"), "copy_split ag")


@pytest.mark.parametrize("case", [
    # W, r, S, Q, N, K, copy_split
    (4, 1, 1024, 2, 1024, 256, 4),    # 1 MiB output chunks: two pieces
    (4, 3, 768, 1, 1400, 192, 3),     # 2,150,400-byte chunks: three pieces, ragged N
], ids=lambda c: "W%d-r%d-S%d-Q%d-N%d-K%d-cs%d" % c)
def test_rs_copy_split_sends_finished_rows(case):
    W, r, S, Q, N, K, split = case
    _say("rs copy_split %s" % (case,))
    w = si.Workload(106, "copy_split_rs", "rs", M=W * S, N=N, K=K, dtype="bf16", out_dtype="bf16", dist="normal",
                    world=W, rank=r, shard_rows=S, chunks_per_shard=Q, order="rs_ring")
    d = si.draw(w)
    chunks, order = oracle.uniform_schedule(W, r, S, Q, "rs_ring")
    s = csg.Schedule.uniform(W, r, S, Q, "rs_ring")
    plan = csg.Plan("rs", W * S, N, K, "bf16", "bf16", s, cfg={"timeout_ms": 1000, "copy_split": split})
    for it in range(2):
        c, out = run_rs(plan, d.A, d.B, "bf16")
        G = out_to_f64(c, "bf16")
        O = out_to_f64(out, "bf16")
        for ch in chunks:
            rows = slice(ch.row_begin, ch.row_end)
            if ch.is_local:
                assert (O[rows] == 0).all()
            else:
                assert np.array_equal(O[rows], G[rows]), "chunk %d, call %d" % (ch.row_begin, it)
    rows = sample_rows(chunks, extra=32, seed=r, M=W * S)
    R, _, _ = oracle.gemm_rs(d.A.device_array, d.B.device_array, chunks, order, row_subset=rows)
    assert_close(G[rows], R[rows], tol_for("bf16", "bf16"), "copy_split rs")


def test_grouped_copy_split_parity():
    """Segments from 1 KiB to about 1.7 MiB: the large ones are cut, the small ones not."""
    _say("grouped copy_split")
    W, E, N, K = 4, 3, 256, 4096
    counts = np.array([[210, 0, 5], [0, 3, 130], [64, 1, 0], [1, 2, 129]], dtype=np.int64)
    chunks, order, gr = oracle.grouped_schedule(W, 2, counts)
    M = int(sum(gr))
    X = si.draw_matrix(107, 0, 0, (M, K), "normal", "bf16")
    B = si.draw_matrix(107, 1, 0, (E, N, K), "normal", "bf16")
    s = csg.Schedule.grouped(W, 2, counts)
    plan = csg.Plan("grouped", M, N, K, "bf16", "bf16", s, group_rows=gr,
                    cfg={"timeout_ms": 1000, "copy_split": 4})
    c, landing = run_ag(plan, chunks, X, B, "bf16", poison_remote=True)
    assert np.array_equal(landing.cpu().numpy().view(np.uint16), X.bits)
    R = oracle.grouped_gemm(X.device_array, B.device_array, chunks, order)
    assert_close(out_to_f64(c, "bf16"), R, 2e-2, "grouped copy_split")
