"""GPU parity over a seeded sweep of schedules the fixed cases do not reach.

Each case draws, from its own seed:
- a chunking of M into chunks of uneven height (1 to 200 rows), dealt to ranks in
  contiguous runs;
- a random arrival (or emission) order over all chunks, local ones included;
- N (a multiple of 4) and K (a multiple of the main loop's K step);
- the dtypes and a plan configuration: split-K, tail splits, static dispatch, tile
  shapes, and copy workgroups instead of the engines.
The GPU result is compared with the oracle element by element, to the same bar as the
fixed cases: max relative error <= 2e-2 with bf16 and <= 1e-4 for fp32 end to end, and
bit for bit where the inputs are small integers (every product and partial sum exact).
Grouped GEMM cases draw a routing-count matrix with empty segments.
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
    from gpu_util import assert_close, bf16_rne_of_f64, out_to_f64, run_ag, run_rs, to_dev, tol_for

SWEEP_SEED = 211
N_CASES = 48

# plan configurations the sweep picks from (the tile shapes are bf16-only)
CFGS_AG = [{}, {"split_k": 2}, {"split_k": 3}, {"tile_dispatch": 2}, {"tail_split": 2, "tail_chunks": 2},
           {"bm": 256, "bn": 128}, {"bm": 128, "bn": 256}, {"bm": 128, "bn": 128}, {"bm": 256, "bn": 224},
           {"copy_backend": "kernel", "copy_workgroups": 8}, {"split_k": 2, "tile_dispatch": 2}]
CFGS_RS = [{}, {"split_k": 2}, {"tile_dispatch": 2}, {"tail_split": 2, "tail_chunks": 1}]
CFGS_F32 = [{}, {"split_k": 2}, {"tile_dispatch": 2}]


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _chunks(g, rank):
    """Uneven chunks over M, dealt to ranks in contiguous runs; returns (chunks, W)."""
    n = int(g.integers(1, 25))
    sizes = [int(x) for x in g.integers(1, 201, size=n)]
    W = int(g.integers(2, min(n, 8) + 1)) if n > 1 else 1
    cuts = sorted(set(int(x) for x in g.choice(np.arange(1, n), size=W - 1, replace=False))) if W > 1 else []
    owner = np.searchsorted(np.array(cuts, dtype=np.int64), np.arange(n), side="right")
    rank = rank % W
    chunks, row = [], 0
    for i, h in enumerate(sizes):
        chunks.append(oracle.Chunk(row, row + h, int(owner[i]), 0, bool(owner[i] == rank)))
        row += h
    return chunks, W


def _case(i):
    g = np.random.default_rng([SWEEP_SEED, i])
    kind = "grouped" if i % 6 == 5 else ("rs" if i % 3 == 1 else "ag")
    dt = [("bf16", "bf16"), ("bf16", "bf16"), ("bf16", "f32"), ("f32", "f32")][int(g.integers(0, 4))]
    if kind == "grouped":
        dt = ("bf16", "bf16")
    in_dt, out_dt = dt
    step = 64 if in_dt == "bf16" else 16
    K = step * int(g.integers(1, (1024 if in_dt == "bf16" else 256) // step + 1))
    N = 4 * int(g.integers(1, 176))
    dist = "int" if g.random() < 0.25 else "normal"
    mode = "compute_only" if g.random() < 0.2 else "overlap"
    if in_dt == "f32":
        cfg = CFGS_F32[int(g.integers(0, len(CFGS_F32)))]
    elif kind == "rs":
        cfg = CFGS_RS[int(g.integers(0, len(CFGS_RS)))]
    elif kind == "grouped":
        cfg = CFGS_AG[int(g.integers(0, 5))]
    else:
        cfg = CFGS_AG[int(g.integers(0, len(CFGS_AG)))]
    cfg = dict(cfg)
    if out_dt == "f32" and cfg.get("bm", 256) * 1000 + cfg.get("bn", 256) not in (256256, 256224):
        cfg.pop("bm")   # the smaller tiles are built for bf16 output only
        cfg.pop("bn")
    return g, kind, in_dt, out_dt, N, K, dist, mode, cfg


CASES = list(range(N_CASES))


def _ids(i):
    _, kind, in_dt, out_dt, N, K, dist, mode, cfg = _case(i)
    return "%d-%s-%s-%s-N%d-K%d-%s-%s-%s" % (i, kind, in_dt, out_dt, N, K, dist, mode,
                                             "_".join("%s%s" % kv for kv in sorted(cfg.items())) or "default")


@pytest.mark.parametrize("i", CASES, ids=_ids)
def test_sweep_parity(i):
    g, kind, in_dt, out_dt, N, K, dist, mode, cfg = _case(i)
    cfg["timeout_ms"] = 1000
    _say("sweep case %s" % _ids(i))
    if kind == "grouped":
        W, E = int(g.integers(2, 9)), int(g.integers(1, 6))
        rank = int(g.integers(0, W))
        counts = g.integers(0, 120, size=(W, E)).astype(np.int64)
        counts[g.random(size=(W, E)) < 0.3] = 0
        if counts.sum() == 0:
            counts[0, 0] = 1
        chunks, order, gr = oracle.grouped_schedule(W, rank, counts)
        M = int(sum(gr))
        X = si.draw_matrix(SWEEP_SEED, 0, i, (M, K), dist, in_dt)
        B = si.draw_matrix(SWEEP_SEED, 1, i, (E, N, K), dist, in_dt)
        s = csg.Schedule.grouped(W, rank, counts)
        plan = csg.Plan("grouped", M, N, K, in_dt, out_dt, s, group_rows=gr, cfg=cfg)
        c, landing = run_ag(plan, chunks, X, B, out_dt, mode=mode)
        R = oracle.grouped_gemm(X.device_array, B.device_array, chunks, order)
        A = X
    else:
        chunks, W = _chunks(g, int(g.integers(0, 8)))
        order = [int(x) for x in g.permutation(len(chunks))]
        M = chunks[-1].row_end
        A = si.draw_matrix(SWEEP_SEED, 0, i, (M, K), dist, in_dt)
        B = si.draw_matrix(SWEEP_SEED, 1, i, (N, K), dist, in_dt)
        s = csg.Schedule.create([(c.row_begin, c.row_end, c.src_rank, c.group, int(c.is_local)) for c in chunks], order)
        plan = csg.Plan(kind, M, N, K, in_dt, out_dt, s, cfg=cfg)
        if kind == "ag":
            c, landing = run_ag(plan, chunks, A, B, out_dt, mode=mode)
            R = oracle.ag_gemm(A.device_array, B.device_array, chunks, order)
        else:
            c, out = run_rs(plan, A, B, out_dt, mode=mode)
            R, Rout, _ = oracle.gemm_rs(A.device_array, B.device_array, chunks, order)
    G = out_to_f64(c, out_dt)
    if dist == "int":
        expect = R if out_dt == "f32" else bf16_rne_of_f64(R)
        assert np.array_equal(G, expect), "integer inputs: result differs from the exact product"
    else:
        assert_close(G, R, tol_for(out_dt, in_dt), "sweep case %d" % i)
    if kind in ("ag", "grouped") and mode == "overlap":
        assert torch.equal(landing.cpu(), to_dev(A.device_array).cpu()), "a remote chunk did not land"
    if kind == "rs":
        O = out_to_f64(out, out_dt)
        for ch in chunks:
            rows = slice(ch.row_begin, ch.row_end)
            if ch.is_local or mode == "compute_only":
                assert (O[rows] == 0).all(), "a chunk that is not sent reached the outgoing buffer"
            else:
                assert np.array_equal(O[rows], G[rows]), "a sent chunk differs from its rows of C"
    plan.close()
    s.close()
