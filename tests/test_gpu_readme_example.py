"""The usage example in README.md runs as written, and its result is right.

The example's Python block is executed as is; its output C (bf16 bits) is then compared
with the oracle's all-gather GEMM of the same A and B, to the bf16 bar of the parity
tests (max relative error <= 2e-2), on sampled rows of every chunk.
"""
import os
import re

import numpy as np
import pytest

import oracle

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _example_source() -> str:
    text = open(os.path.join(ROOT, "README.md")).read()
    blocks = re.findall(r"```python\n(.*?)```", text, re.S)
    assert len(blocks) == 1, "README.md should hold one Python example"
    return blocks[0]


def test_readme_example_runs_and_is_right():
    ns = {}
    exec(compile(_example_source(), "README.md example", "exec"), ns)
    torch.cuda.synchronize()
    a = ns["a_staging"].cpu().numpy().view(np.uint16)
    b = ns["b"].cpu().numpy().view(np.uint16)
    c = ns["c"]
    M, world, rank = ns["M"], ns["world"], ns["rank"]
    chunks, order = oracle.uniform_schedule(world, rank, M // world, 4, "ring")
    rows = sorted({r for ch in chunks for r in (ch.row_begin, ch.row_end - 1)} | set(range(0, M, 997)))
    R = oracle.ag_gemm(a, b, chunks, order, row_subset=rows)[rows]
    import seeded_inputs as si
    G = si.bf16_bits_to_f32(c.cpu().numpy().view(np.uint16)[rows]).astype(np.float64)
    assert oracle.max_rel_error(G, R) <= 2e-2
    assert torch.equal(ns["a_landing"], ns["a_staging"])     # every remote chunk landed
