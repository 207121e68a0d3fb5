"""Oracle: the chunk-scheduled GEMMs, computed chunk by chunk in schedule order.

TEST INFRASTRUCTURE ONLY. Nothing in the product path may import this module.

The fused operator keeps the numerical meaning of the plain local GEMM (Overview,
architecture and output paragraph): whatever the chunk order, C = A . B^T with B
stored N x K (the annotated local kernel's ``tl.dot(a, b.T)``). The oracle
therefore walks the schedule in order and, for every chunk, computes the plain
GEMM rows that chunk makes available (all-gather, grouped) or produces
(reduce-scatter), in fp64 with k ascending (see ref_gemm.c).
"""
from __future__ import annotations

import ctypes
import math
import os
from typing import Optional, Sequence

import numpy as np

from .schedule import Chunk

_LIB = None


def _lib():
    global _LIB
    if _LIB is None:
        from .build import LIB, build
        if not os.path.exists(LIB):
            build()
        lib = ctypes.CDLL(LIB)
        i64, vp, ci = ctypes.c_int64, ctypes.c_void_p, ctypes.c_int
        lib.oracle_gemm_rows.argtypes = [vp, ci, vp, ci, i64, i64, vp, i64, vp]
        lib.oracle_gemm_rows.restype = None
        lib.oracle_gemm_elems.argtypes = [vp, ci, vp, ci, i64, vp, vp, i64, vp]
        lib.oracle_gemm_elems.restype = None
        lib.oracle_num_threads.restype = ci
        _LIB = lib
    return _LIB


def num_threads() -> int:
    return int(_lib().oracle_num_threads())


def _dt(arr: np.ndarray) -> int:
    if arr.dtype == np.uint16:
        return 0
    if arr.dtype == np.float32:
        return 1
    raise TypeError("oracle inputs are bf16 bit patterns (uint16) or float32, got %s" % arr.dtype)


def gemm_rows(A: np.ndarray, B_nk: np.ndarray, rows: Sequence[int]) -> np.ndarray:
    """fp64 rows ``rows`` of A . B_nk^T. A is [*, K], B_nk is [N, K]."""
    A = np.ascontiguousarray(A)
    B_nk = np.ascontiguousarray(B_nk)
    N, K = B_nk.shape
    assert A.shape[1] == K
    r = np.ascontiguousarray(np.asarray(rows, dtype=np.int64))
    assert r.size == 0 or (r.min() >= 0 and r.max() < A.shape[0])
    out = np.empty((r.size, N), dtype=np.float64)
    if r.size:
        _lib().oracle_gemm_rows(A.ctypes.data, _dt(A), B_nk.ctypes.data, _dt(B_nk), N, K,
                                r.ctypes.data, r.size, out.ctypes.data)
    return out


def gemm_elems(A: np.ndarray, B_nk: np.ndarray, ii, jj) -> np.ndarray:
    A = np.ascontiguousarray(A)
    B_nk = np.ascontiguousarray(B_nk)
    K = B_nk.shape[1]
    ii = np.ascontiguousarray(np.asarray(ii, dtype=np.int64))
    jj = np.ascontiguousarray(np.asarray(jj, dtype=np.int64))
    out = np.empty(ii.size, dtype=np.float64)
    if ii.size:
        _lib().oracle_gemm_elems(A.ctypes.data, _dt(A), B_nk.ctypes.data, _dt(B_nk), K,
                                 ii.ctypes.data, jj.ctypes.data, ii.size, out.ctypes.data)
    return out


def ag_gemm(A: np.ndarray, B_nk: np.ndarray, chunks: Sequence[Chunk], order: Sequence[int],
            row_subset: Optional[Sequence[int]] = None) -> np.ndarray:
    """AllGather + GEMM on one rank: as chunk ``order[p]`` of A lands, compute the
    C rows it covers. Returns C (fp64, M x N); with ``row_subset`` only those rows
    are computed (others stay NaN)."""
    M = A.shape[0]
    N = B_nk.shape[0]
    C = np.full((M, N), np.nan, dtype=np.float64)
    want = None if row_subset is None else set(int(r) for r in row_subset)
    for c in order:
        ch = chunks[int(c)]
        rows = [r for r in range(ch.row_begin, ch.row_end) if want is None or r in want]
        if rows:
            C[rows] = gemm_rows(A, B_nk, rows)
    return C


def gemm_rs(A: np.ndarray, B_nk: np.ndarray, chunks: Sequence[Chunk], order: Sequence[int],
            row_subset: Optional[Sequence[int]] = None):
    """GEMM + ReduceScatter on one rank: produce C chunk by chunk in emission order;
    every non-local chunk is also sent (written to the outgoing buffer). Returns
    (C, outgoing, emission_log) with emission_log the chunk ids in emission order."""
    M = A.shape[0]
    N = B_nk.shape[0]
    C = np.full((M, N), np.nan, dtype=np.float64)
    out = np.full((M, N), np.nan, dtype=np.float64)
    want = None if row_subset is None else set(int(r) for r in row_subset)
    log = []
    for c in order:
        ch = chunks[int(c)]
        rows = [r for r in range(ch.row_begin, ch.row_end) if want is None or r in want]
        if rows:
            C[rows] = gemm_rows(A, B_nk, rows)
            if not ch.is_local:
                out[rows] = C[rows]
        log.append(int(c))
    return C, out, log


def gemm_ar(A: np.ndarray, B_nk: np.ndarray, chunks: Sequence[Chunk], order: Sequence[int],
            partials: np.ndarray, reduced_in: np.ndarray, row_subset: Optional[Sequence[int]] = None):
    """GEMM + AllReduce on one rank (Evaluation: the GEMM-AR operator; Section 5.1,
    Fig. of communication schedules, the partition-based AllReduce pattern), taken as
    a reduce-scatter followed by an all-gather over the rank's row shards.

    Every rank r holds a K-slice A_r, B_r of a row-parallel product; the all-reduced
    result is sum_r A_r . B_r^T. On this rank:
      - its partial P = A . B_nk^T is produced chunk by chunk in emission order;
      - a non-local chunk is sent to its owner (reduce-scatter half):
        outgoing[rows] = P[rows];
      - an own (local) chunk is reduced with the other ranks' partials of the same
        rows, partials[j] for the j-th other rank in ascending rank order, stored as
        [world-1, S, N] over the own shard S (rows own0 .. own0+S-1):
        C[rows] = P[rows] + sum_j partials[j][rows - own0]; it is then sent to every
        other rank (all-gather half): outgoing[rows] = C[rows];
      - a non-local chunk's final rows come from its owner: C[rows] = reduced_in[rows].
    Returns (C, outgoing, emission_log)."""
    M = A.shape[0]
    N = B_nk.shape[0]
    C = np.full((M, N), np.nan, dtype=np.float64)
    out = np.full((M, N), np.nan, dtype=np.float64)
    own = [ch for ch in chunks if ch.is_local]
    own0 = min(ch.row_begin for ch in own)
    want = None if row_subset is None else set(int(r) for r in row_subset)
    log = []
    for c in order:
        ch = chunks[int(c)]
        rows = [r for r in range(ch.row_begin, ch.row_end) if want is None or r in want]
        if rows:
            P = gemm_rows(A, B_nk, rows)
            if ch.is_local:
                red = P.copy()
                for j in range(partials.shape[0]):
                    red += partials[j][np.asarray(rows) - own0].astype(np.float64)
                C[rows] = red
                out[rows] = red
            else:
                out[rows] = P
                C[rows] = reduced_in[rows].astype(np.float64)
        log.append(int(c))
    return C, out, log


def grouped_gemm(X: np.ndarray, B_enk: np.ndarray, chunks: Sequence[Chunk], order: Sequence[int],
                 row_subset: Optional[Sequence[int]] = None) -> np.ndarray:
    """All-to-all + grouped GEMM on one rank: as the (source, expert) segment
    ``order[p]`` lands, compute its rows with that expert's weight B_e (N x K)."""
    M = X.shape[0]
    N = B_enk.shape[1]
    C = np.full((M, N), np.nan, dtype=np.float64)
    want = None if row_subset is None else set(int(r) for r in row_subset)
    for c in order:
        ch = chunks[int(c)]
        rows = [r for r in range(ch.row_begin, ch.row_end) if want is None or r in want]
        if rows:
            C[rows] = gemm_rows(X, B_enk[ch.group], rows)
    return C


# ----------------------------------------------------------------------------
# Tiny-input references used to pin the above (pure Python, small sizes only)
# ----------------------------------------------------------------------------
def exact_dot_fsum(a_row: Sequence[float], b_row: Sequence[float]) -> float:
    """Correctly rounded dot product of float32/bf16 values: each product is exact
    in fp64 and math.fsum rounds the exact sum once."""
    return math.fsum(float(x) * float(y) for x, y in zip(a_row, b_row))


# ----------------------------------------------------------------------------
# Comparison metric
# ----------------------------------------------------------------------------
def max_rel_error(G: np.ndarray, R: np.ndarray) -> float:
    """max_ij |G - R| / max(|R_ij|, rms(R)): an elementwise relative error whose
    denominator is floored at the output's RMS so entries near zero do not blow
    it up."""
    G = np.asarray(G, dtype=np.float64)
    R = np.asarray(R, dtype=np.float64)
    rms = math.sqrt(float(np.mean(R * R))) if R.size else 0.0
    den = np.maximum(np.abs(R), rms)
    den = np.where(den == 0, 1.0, den)
    return float(np.max(np.abs(G - R) / den)) if R.size else 0.0
