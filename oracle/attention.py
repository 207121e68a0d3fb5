"""Oracle: attention over key/value chunks that arrive in a ring (test infrastructure).

Sequence-parallel ring attention (Evaluation, the Ring-Attn operator; Section 5.1,
Fig. of communication schedules, the ring pattern): rank r holds the queries of its
sequence shard and, eventually, every rank's keys and values, which reach it chunk by
chunk in ring order. The result does not depend on that order: for every query row
and head it is softmax attention over all keys,

    O[q, h, :] = sum_j p_j V[j, g(h), :],   p_j = exp(s_j - m) / l,
    s_j = scale * Q[q, h, :] . K[j, g(h), :],  m = max_j s_j,  l = sum_j exp(s_j - m),
    LSE[h, q] = m + log(l)  (natural log),

with g(h) = h // (heads / kv_heads) the key/value head a query head reads (grouped
heads). The oracle writes that definition out in fp64 (`attention`), and, as a second
function, the chunk-by-chunk form that merges per-chunk partial results with their
log-sum-exp in arrival order (`attention_chunked`): it is the algorithm's structure,
and its agreement with the definition is one of the pins.

Layouts: Q and O are [Sq, H, D], K and V are [S, Hkv, D] (sequence-major), LSE is
[H, Sq]. Inputs are float32 values (bf16 inputs are passed as their float32 values).
"""
from __future__ import annotations

from typing import Optional, Sequence

import numpy as np

from .schedule import Chunk


def attention(Q: np.ndarray, K: np.ndarray, V: np.ndarray, scale: Optional[float] = None):
    """Plain softmax attention in fp64. Returns (O [Sq, H, D], LSE [H, Sq])."""
    Sq, H, D = Q.shape
    S, Hkv, _ = K.shape
    assert H % Hkv == 0 and V.shape == K.shape
    G = H // Hkv
    scale = 1.0 / np.sqrt(D) if scale is None else scale
    O = np.empty((Sq, H, D), dtype=np.float64)
    LSE = np.empty((H, Sq), dtype=np.float64)
    for h in range(H):
        q = Q[:, h, :].astype(np.float64)
        k = K[:, h // G, :].astype(np.float64)
        v = V[:, h // G, :].astype(np.float64)
        s = (q @ k.T) * scale                       # [Sq, S]
        m = s.max(axis=1, keepdims=True)
        e = np.exp(s - m)
        l = e.sum(axis=1, keepdims=True)
        O[:, h, :] = (e @ v) / l
        LSE[h] = (m + np.log(l))[:, 0]
    return O, LSE


def attention_chunked(Q: np.ndarray, K: np.ndarray, V: np.ndarray, chunks: Sequence[Chunk],
                      order: Sequence[int], scale: Optional[float] = None):
    """The same attention computed as the chunk schedule delivers the keys: for each
    chunk in arrival order, the partial result over that chunk's keys (its own
    maximum, normaliser and weighted values) is merged into the running one by
    rescaling both to the larger maximum. Returns (O, LSE)."""
    Sq, H, D = Q.shape
    S, Hkv, _ = K.shape
    G = H // Hkv
    scale = 1.0 / np.sqrt(D) if scale is None else scale
    m = np.full((H, Sq), -np.inf)
    l = np.zeros((H, Sq))
    acc = np.zeros((H, Sq, D))
    for c in order:
        ch = chunks[int(c)]
        rows = slice(ch.row_begin, ch.row_end)
        for h in range(H):
            q = Q[:, h, :].astype(np.float64)
            k = K[rows, h // G, :].astype(np.float64)
            v = V[rows, h // G, :].astype(np.float64)
            s = (q @ k.T) * scale
            mc = s.max(axis=1)
            e = np.exp(s - mc[:, None])
            m_new = np.maximum(m[h], mc)
            a_old = np.exp(m[h] - m_new)
            a_new = np.exp(mc - m_new)
            l[h] = l[h] * a_old + e.sum(axis=1) * a_new
            acc[h] = acc[h] * a_old[:, None] + (e @ v) * a_new[:, None]
            m[h] = m_new
    O = np.transpose(acc / l[:, :, None], (1, 0, 2))
    return O, m + np.log(l)


def attention_fsum(q, ks, vs, scale):
    """One query row against keys ks and values vs, pure Python with math.fsum: the
    reference for tiny inputs."""
    import math
    s = [scale * math.fsum(float(a) * float(b) for a, b in zip(q, k)) for k in ks]
    m = max(s)
    e = [math.exp(x - m) for x in s]
    l = math.fsum(e)
    out = [math.fsum(w * float(v[d]) for w, v in zip(e, vs)) / l for d in range(len(vs[0]))]
    return out, m + math.log(l)
