"""Pins for the oracle's ring attention (CPU only).

Fixed by mathematics, not by the oracle: brute force with exactly summed dot products
and weights (math.fsum) on tiny inputs; closed forms (equal scores give the mean of
the values and LSE = log S; one key gives its value; equal values give that value);
the grouped-head mapping against single-head attention; and the chunk-merged form
agreeing with the plain definition in every arrival order.
"""
import math

import numpy as np
import pytest

import oracle


def _rand(shape, seed, scale=1.0):
    return (np.random.default_rng(seed).standard_normal(shape) * scale).astype(np.float32)


@pytest.mark.parametrize("Sq,S,H,Hkv,D", [(1, 1, 1, 1, 1), (3, 5, 2, 1, 4), (4, 7, 4, 2, 3), (2, 9, 3, 3, 8)])
def test_brute_force_fsum(Sq, S, H, Hkv, D):
    Q, K, V = _rand((Sq, H, D), 1), _rand((S, Hkv, D), 2), _rand((S, Hkv, D), 3)
    O, LSE = oracle.attention(Q, K, V)
    scale = 1.0 / math.sqrt(D)
    for q in range(Sq):
        for h in range(H):
            g = h // (H // Hkv)
            o, lse = oracle.attention_fsum(Q[q, h], [K[j, g] for j in range(S)], [V[j, g] for j in range(S)], scale)
            np.testing.assert_allclose(O[q, h], o, rtol=1e-12, atol=1e-13)
            assert abs(LSE[h, q] - lse) < 1e-12


def test_closed_forms():
    Sq, S, H, D = 3, 6, 2, 5
    Q, V = _rand((Sq, H, D), 4), _rand((S, H, D), 5)
    O, LSE = oracle.attention(Q, np.zeros((S, H, D), np.float32), V)          # equal scores
    np.testing.assert_allclose(O, np.broadcast_to(V.astype(np.float64).mean(axis=0), O.shape), atol=1e-14)
    np.testing.assert_allclose(LSE, math.log(S), atol=1e-14)
    K1, V1 = _rand((1, H, D), 6), _rand((1, H, D), 7)                          # one key
    O, LSE = oracle.attention(Q, K1, V1)
    np.testing.assert_allclose(O, np.broadcast_to(V1[0].astype(np.float64), O.shape), atol=1e-14)
    np.testing.assert_allclose(LSE, np.einsum("qhd,hd->hq", Q.astype(np.float64), K1[0].astype(np.float64)) / math.sqrt(D),
                               atol=1e-12)
    row = _rand((1, H, D), 8)                                                  # equal values
    O, _ = oracle.attention(Q, _rand((S, H, D), 9), np.repeat(row, S, axis=0))
    np.testing.assert_allclose(O, np.broadcast_to(row[0].astype(np.float64), O.shape), atol=1e-13)


def test_grouped_heads_read_their_kv_head():
    Sq, S, H, Hkv, D = 4, 8, 6, 2, 4
    Q, K, V = _rand((Sq, H, D), 10), _rand((S, Hkv, D), 11), _rand((S, Hkv, D), 12)
    O, LSE = oracle.attention(Q, K, V)
    for h in range(H):
        g = h // (H // Hkv)
        o1, l1 = oracle.attention(Q[:, h:h + 1], K[:, g:g + 1], V[:, g:g + 1])
        assert np.array_equal(O[:, h], o1[:, 0]) and np.array_equal(LSE[h], l1[0])


@pytest.mark.parametrize("W,r,Sh,Qc,kind", [(2, 0, 8, 2, "ring"), (4, 1, 6, 3, "ring"), (4, 2, 4, 2, "permutation"),
                                             (8, 7, 2, 1, "swizzle1d")])
def test_chunked_merge_equals_definition_in_any_order(W, r, Sh, Qc, kind):
    Sq, H, Hkv, D = 5, 4, 2, 8
    S = W * Sh
    Q, K, V = _rand((Sq, H, D), 13, 2.0), _rand((S, Hkv, D), 14, 2.0), _rand((S, Hkv, D), 15)
    perm = list(np.random.default_rng(3).permutation((W - 1) * Qc)) if kind == "permutation" else None
    chunks, order = oracle.uniform_schedule(W, r, Sh, Qc, kind, perm)
    O, LSE = oracle.attention(Q, K, V)
    Oc, Lc = oracle.attention_chunked(Q, K, V, chunks, order)
    np.testing.assert_allclose(Oc, O, rtol=0, atol=1e-12)
    np.testing.assert_allclose(Lc, LSE, rtol=0, atol=1e-12)
    Or, Lr = oracle.attention_chunked(Q, K, V, chunks, list(reversed(order)))
    np.testing.assert_allclose(Or, O, rtol=0, atol=1e-12)
