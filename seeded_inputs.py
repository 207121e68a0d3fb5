"""Seeded synthetic inputs for the chunk-scheduled GEMM workloads.

This module is shared by the CPU oracle, the tests and the benchmark. It only
draws random numbers and lays them out; it holds none of the method's
arithmetic (no schedule templates, no dependence maps, no products). Every
random quantity the method consumes -- matrix values, the arrival permutation
of remote chunks, copy delays, token routing -- is drawn here and handed to
both the oracle and the HIP path as plain arrays.

Generators are ``numpy.random.default_rng([cfg_id, stream, rep])`` with the
streams

    0 = A / X values, 1 = B values, 2 = arrival permutation,
    3 = copy delays,  4 = token routing,
    5 = the peers' partial sums (GEMM-AR), 6 = the other shards' reduced rows (GEMM-AR),
    7 = attention values (Q, then K, then V, from one generator).

Workload shapes are tensor-parallel FFN slices of Llama-3-8B-like
(hidden 4096, FFN 14336/8 = 1792) and Llama-3-70B-like (hidden 8192,
FFN 28672/8 = 3584) layers, the model families the paper's GEMM evaluation
uses (Evaluation, Workloads paragraph). The paper's measurements use model
shapes, not a dataset, so no dataset is stood in for.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional

import numpy as np

STREAM_A, STREAM_B, STREAM_PERM, STREAM_DELAY, STREAM_ROUTE = 0, 1, 2, 3, 4
STREAM_PARTIALS, STREAM_REDUCED, STREAM_ATTN = 5, 6, 7


def rng(cfg_id: int, stream: int, rep: int = 0) -> np.random.Generator:
    return np.random.default_rng([int(cfg_id), int(stream), int(rep)])


# ----------------------------------------------------------------------------
# bf16 encoding of drawn values (round-to-nearest-even from fp32). This is how
# inputs are *drawn* as bf16; it is not part of the method.
# ----------------------------------------------------------------------------
def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """fp32 array -> uint16 bf16 bit patterns, round to nearest even (no NaN inputs)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    r = (u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


@dataclass
class Matrix:
    """A drawn matrix: ``values`` (float32, exactly the stored values) and, for
    bf16, the raw ``bits`` (uint16) that are copied to the device."""
    values: np.ndarray
    dtype: str                      # "bf16" | "f32"
    bits: Optional[np.ndarray] = None

    @property
    def device_array(self) -> np.ndarray:
        return self.bits if self.dtype == "bf16" else self.values


def draw_matrix(cfg_id: int, stream: int, rep: int, shape, dist: str, dtype: str,
                scale: float = 0.02) -> Matrix:
    g = rng(cfg_id, stream, rep)
    if dist == "uniform":          # U[-1, 1)
        v = g.uniform(-1.0, 1.0, size=shape).astype(np.float32)
    elif dist == "normal":         # N(0, scale)
        v = g.standard_normal(size=shape, dtype=np.float32) * np.float32(scale)
    elif dist == "int":            # integers in {-2..2}: every product and partial sum exact
        v = g.integers(-2, 3, size=shape).astype(np.float32)
    else:
        raise ValueError(dist)
    if dtype == "bf16":
        bits = f32_to_bf16_bits(v)
        return Matrix(values=bf16_bits_to_f32(bits), dtype="bf16", bits=bits)
    if dtype == "f32":
        return Matrix(values=np.ascontiguousarray(v), dtype="f32")
    raise ValueError(dtype)


def draw_permutation(cfg_id: int, rep: int, n: int) -> np.ndarray:
    """A seeded permutation of 0..n-1 (int32)."""
    return rng(cfg_id, STREAM_PERM, rep).permutation(n).astype(np.int32)


def draw_delays_us(cfg_id: int, rep: int, n: int, hi: float = 20.0) -> np.ndarray:
    """Per-copy gap delays, U[0, hi] microseconds (float32), one per remote chunk in
    arrival order."""
    return rng(cfg_id, STREAM_DELAY, rep).uniform(0.0, hi, size=n).astype(np.float32)


def draw_topk_routing(cfg_id: int, rep: int, n_tokens: int, n_experts: int, topk: int,
                      zipf_s: float) -> np.ndarray:
    """For every token, ``topk`` distinct experts drawn without replacement with
    weights proportional to (e+1)^-zipf_s. Uses the Gumbel-top-k construction
    (equivalent to successive sampling without replacement). Returns int32
    [n_tokens, topk]."""
    g = rng(cfg_id, STREAM_ROUTE, rep)
    logw = -zipf_s * np.log(np.arange(1, n_experts + 1, dtype=np.float64))
    gumbel = g.gumbel(size=(n_tokens, n_experts))
    keys = logw[None, :] + gumbel
    top = np.argsort(-keys, axis=1, kind="stable")[:, :topk]
    return top.astype(np.int32)


# ----------------------------------------------------------------------------
# Workload descriptions
# ----------------------------------------------------------------------------
@dataclass
class Workload:
    """One workload of the benchmark/test suite. ``op`` is "ag", "rs", "ar" (GEMM +
    all-reduce), "grouped" or "attn" (ring attention: M = query rows of this rank,
    shard_rows = key rows per rank, heads / kv_heads / head_dim in ``extras``)."""
    cfg_id: int
    name: str
    op: str
    M: int
    N: int
    K: int
    dtype: str                      # input dtype "bf16" | "f32"
    out_dtype: str
    dist: str
    world: int
    rank: int = 0
    shard_rows: int = 0             # S (ag / rs)
    chunks_per_shard: int = 0       # Q (ag / rs)
    order: str = "ring"             # ring | swizzle1d | permutation | rs_ring
    delays: bool = False
    # grouped GEMM (all-to-all dispatch + per-expert GEMM)
    n_tokens: int = 0
    n_experts: int = 0
    topk: int = 0
    zipf_s: float = 0.0
    extras: dict = field(default_factory=dict)

    @property
    def flops(self) -> float:
        if self.op == "attn":
            # two products (scores and weighted values) per query row, key row and head
            e = self.extras
            return 4.0 * self.M * self.world * self.shard_rows * e["head_dim"] * e["heads"]
        return 2.0 * self.M * self.N * self.K


WORKLOADS = {
    1: Workload(1, "ag_w2_f32_256", "ag", M=256, N=256, K=256, dtype="f32", out_dtype="f32",
                dist="uniform", world=2, shard_rows=128, chunks_per_shard=2, order="permutation"),
    2: Workload(2, "ag_w8_bf16_8192x4096x1792", "ag", M=8192, N=1792, K=4096, dtype="bf16",
                out_dtype="bf16", dist="normal", world=8, shard_rows=1024, chunks_per_shard=4,
                order="ring"),
    3: Workload(3, "rs_w8_bf16_8192x1792x4096", "rs", M=8192, N=4096, K=1792, dtype="bf16",
                out_dtype="bf16", dist="normal", world=8, shard_rows=1024, chunks_per_shard=4,
                order="rs_ring"),
    4: Workload(4, "ag_fine_w8_bf16_16384x8192x3584", "ag", M=16384, N=3584, K=8192, dtype="bf16",
                out_dtype="bf16", dist="normal", world=8, shard_rows=2048, chunks_per_shard=16,
                order="permutation", delays=True),
    5: Workload(5, "a2a_grouped_e8_bf16_32768x4096x1792", "grouped", M=32768, N=1792, K=4096,
                dtype="bf16", out_dtype="bf16", dist="normal", world=8, n_tokens=16384,
                n_experts=8, topk=2, zipf_s=1.2),
    # GEMM + all-reduce: the row-parallel down-projection of the 8B-like layer, K = 14336 / 8
    # per rank, all-reduced over 8 ranks (reduce-scatter then all-gather of 4 chunks per shard)
    6: Workload(6, "ar_w8_bf16_8192x1792x4096", "ar", M=8192, N=4096, K=1792, dtype="bf16",
                out_dtype="bf16", dist="normal", world=8, shard_rows=1024, chunks_per_shard=4,
                order="rs_ring"),
    # sequence-parallel ring attention, 8B-like heads (32 query heads, 8 key/value heads,
    # head dim 128), a 32768-token sequence over 8 ranks: 4096 queries and 4096 keys per
    # rank, key/value shards arriving in ring order, 2 chunks per shard
    7: Workload(7, "ring_attn_w8_bf16_h32kv8_s32768_d128", "attn", M=4096, N=0, K=0, dtype="bf16",
                out_dtype="bf16", dist="normal", world=8, shard_rows=4096, chunks_per_shard=2,
                order="ring", extras={"heads": 32, "kv_heads": 8, "head_dim": 128}),
}


@dataclass
class Drawn:
    """All random draws of one workload replicate."""
    A: Matrix                       # M x K (ag/rs) or routed X (grouped, M = tokens*topk)
    B: Matrix                       # N x K (ag/rs) or E x N x K (grouped); stored K-contiguous
    perm: Optional[np.ndarray] = None        # permutation of the remote chunks (ag "permutation")
    delays_us: Optional[np.ndarray] = None   # per remote chunk in arrival order
    routing: Optional[np.ndarray] = None     # grouped: [n_tokens, topk] expert ids
    counts: Optional[np.ndarray] = None      # grouped: [world, n_experts] rows per (source, expert)
    tokens: Optional[Matrix] = None          # grouped: un-routed token matrix
    partials: Optional[Matrix] = None        # ar: [world-1, S, N] the peers' partial sums of this
                                             # rank's shard, peers in ascending rank order
    reduced: Optional[Matrix] = None         # ar: [M, N] reduced rows the other shards' owners send
    V: Optional[Matrix] = None               # attn: values [S, kv_heads, head_dim] (A = queries
                                             # [Sq, heads, head_dim], B = keys [S, kv_heads, head_dim])


def grouped_layout(routing: np.ndarray, world: int, n_experts: int):
    """Lay routed (token, expert) pairs out expert-major, then by source rank, then
    by token id. Token t comes from source rank t // (n_tokens / world).
    Returns (row_token [rows] int64, counts [world, n_experts] int64)."""
    n_tokens, topk = routing.shape
    per_src = n_tokens // world
    tok = np.repeat(np.arange(n_tokens, dtype=np.int64), topk)
    exp = routing.reshape(-1).astype(np.int64)
    src = tok // per_src
    order = np.lexsort((tok, src, exp))
    counts = np.zeros((world, n_experts), dtype=np.int64)
    np.add.at(counts, (src, exp), 1)
    return tok[order], counts


def draw(w: Workload, rep: int = 0, dist: Optional[str] = None, M: Optional[int] = None,
         N: Optional[int] = None, K: Optional[int] = None) -> Drawn:
    """Draw every random input of workload ``w`` (optionally overriding the value
    distribution or shrinking the shape for small test cases)."""
    dist = dist or w.dist
    M = M or w.M
    N = N or w.N
    K = K or w.K
    cid = w.cfg_id
    if w.op in ("ag", "rs", "ar"):
        A = draw_matrix(cid, STREAM_A, rep, (M, K), dist, w.dtype)
        B = draw_matrix(cid, STREAM_B, rep, (N, K), dist, w.dtype)
        d = Drawn(A=A, B=B)
        S, Q = w.shard_rows, w.chunks_per_shard
        n_remote = (w.world - 1) * Q
        if w.op == "ar":
            # values spread like a partial product of A and B (and a sum of world of them)
            part_scale = 0.02 * 0.02 * float(np.sqrt(K))
            d.partials = draw_matrix(cid, STREAM_PARTIALS, rep, (w.world - 1, S, N), dist, w.out_dtype,
                                     scale=part_scale)
            d.reduced = draw_matrix(cid, STREAM_REDUCED, rep, (M, N), dist, w.out_dtype,
                                    scale=part_scale * float(np.sqrt(w.world)))
        if w.op == "ag" and w.order == "permutation":
            d.perm = draw_permutation(cid, rep, n_remote)
        if w.delays:
            d.delays_us = draw_delays_us(cid, rep, n_remote)
        return d
    if w.op == "attn":
        e = w.extras
        S = w.world * w.shard_rows
        g = rng(cid, STREAM_ATTN, rep)
        mats = []
        for shape in ((M, e["heads"], e["head_dim"]), (S, e["kv_heads"], e["head_dim"]),
                      (S, e["kv_heads"], e["head_dim"])):
            if dist == "int":
                v = g.integers(-2, 3, size=shape).astype(np.float32)
            else:
                v = g.standard_normal(size=shape, dtype=np.float32)
            if w.dtype == "bf16":
                bits = f32_to_bf16_bits(v)
                mats.append(Matrix(values=bf16_bits_to_f32(bits), dtype="bf16", bits=bits))
            else:
                mats.append(Matrix(values=np.ascontiguousarray(v), dtype="f32"))
        return Drawn(A=mats[0], B=mats[1], V=mats[2])
    if w.op == "grouped":
        routing = draw_topk_routing(cid, rep, w.n_tokens, w.n_experts, w.topk, w.zipf_s)
        row_token, counts = grouped_layout(routing, w.world, w.n_experts)
        tokens = draw_matrix(cid, STREAM_A, rep, (w.n_tokens, K), dist, w.dtype)
        vals = np.ascontiguousarray(tokens.values[row_token])
        bits = None if tokens.bits is None else np.ascontiguousarray(tokens.bits[row_token])
        X = Matrix(values=vals, dtype=w.dtype, bits=bits)
        B = draw_matrix(cid, STREAM_B, rep, (w.n_experts, N, K), dist, w.dtype)
        return Drawn(A=X, B=B, routing=routing, counts=counts, tokens=tokens)
    raise ValueError(w.op)
