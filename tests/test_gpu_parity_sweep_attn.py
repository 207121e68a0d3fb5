"""GPU parity of chunk-scheduled ring attention over a seeded sweep of schedules.

Each case draws, from its own seed:
- key/value chunks of uneven height (multiples of the kernel's 64-key block), dealt to
  ranks in contiguous runs;
- a random arrival order;
- a ragged number of query rows;
- heads grouped onto fewer key/value heads;
- overlap or compute-only mode.
Outputs and log-sum-exps are compared with the fp64 oracle over all keys, to the bar
of the fixed attention cases (max relative error <= 2e-2 with bf16).
"""
import os
import sys
from types import SimpleNamespace

import numpy as np
import pytest

import oracle
import paper_2601_20595_amd as csg
import seeded_inputs as si

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
if torch.cuda.is_available():
    from test_gpu_parity_attn import _check, run_attn

SWEEP_SEED = 223
N_CASES = 16
BLOCK_KV = 64
HEAD_DIM = 128


def _case(i):
    g = np.random.default_rng([SWEEP_SEED, i])
    n = int(g.integers(2, 17))
    heights = [BLOCK_KV * int(x) for x in g.integers(1, 9, size=n)]
    W = int(g.integers(2, min(n, 8) + 1))
    cuts = sorted(int(x) for x in g.choice(np.arange(1, n), size=W - 1, replace=False))
    owner = np.searchsorted(np.array(cuts, dtype=np.int64), np.arange(n), side="right")
    rank = int(g.integers(0, W))
    chunks, row = [], 0
    for k, h in enumerate(heights):
        chunks.append(oracle.Chunk(row, row + h, int(owner[k]), 0, bool(owner[k] == rank)))
        row += h
    order = [int(x) for x in g.permutation(n)]
    Hkv = [1, 2, 4, 8][int(g.integers(0, 4))]
    H = Hkv * [1, 2, 4][int(g.integers(0, 3))]
    Sq = int(g.integers(1, 301))
    mode = "compute_only" if g.random() < 0.25 else "overlap"
    return chunks, order, W, rank, H, Hkv, Sq, mode


def _ids(i):
    chunks, order, W, rank, H, Hkv, Sq, mode = _case(i)
    return "%d-W%d-chunks%d-S%d-Sq%d-H%d-Hkv%d-%s" % (i, W, len(chunks), chunks[-1].row_end, Sq, H, Hkv, mode)


@pytest.mark.parametrize("i", list(range(N_CASES)), ids=_ids)
def test_attention_sweep_parity(i):
    chunks, order, W, rank, H, Hkv, Sq, mode = _case(i)
    print("attention sweep case %s" % _ids(i), flush=True)
    S = chunks[-1].row_end
    d = SimpleNamespace(A=si.draw_matrix(SWEEP_SEED, 0, i, (Sq, H, HEAD_DIM), "normal", "bf16", scale=1.0),
                        B=si.draw_matrix(SWEEP_SEED, 1, i, (S, Hkv, HEAD_DIM), "normal", "bf16", scale=1.0),
                        V=si.draw_matrix(SWEEP_SEED, 2, i, (S, Hkv, HEAD_DIM), "normal", "bf16", scale=1.0))
    s = csg.Schedule.create([(c.row_begin, c.row_end, c.src_rank, c.group, int(c.is_local)) for c in chunks], order)
    plan = csg.AttnPlan(H, Hkv, HEAD_DIM, Sq, s, cfg={"timeout_ms": 1000})
    o, lse = run_attn(plan, d, chunks, mode=mode)
    _check(o, lse, d)
    plan.close()
    s.close()
