"""Pins for the oracle's chunk-by-chunk GEMMs (CPU only).

What fixes the expected values here is the mathematics, not the oracle:
  * brute force: the correctly rounded dot product (exact fp64 products summed by
    math.fsum) on tiny inputs, within the error bound of sequential summation;
  * a library routine: numpy's fp64 matmul on mid-size inputs (C = A . B^T);
  * exactness: small-integer inputs give exact integer products, checked against
    int64 matmul, and B = I gives C = A;
  * invariance: the chunk order must not change a single bit of C
    (the fused operator keeps the plain GEMM's meaning).
"""
import math

import numpy as np
import pytest

import oracle
import seeded_inputs as si


def _draw(shape, dist, dtype, stream, rep=0, cfg=90):
    return si.draw_matrix(cfg, stream, rep, shape, dist, dtype)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("M,N,K", [(1, 1, 1), (3, 5, 7), (16, 16, 16), (9, 4, 13)])
def test_brute_force_fsum(dtype, M, N, K):
    A = _draw((M, K), "uniform", dtype, 0, rep=M * 100 + K)
    B = _draw((N, K), "uniform", dtype, 1, rep=N * 100 + K)
    C = oracle.gemm_rows(A.device_array, B.device_array, range(M))
    for i in range(M):
        for j in range(N):
            exact = oracle.exact_dot_fsum(A.values[i], B.values[j])
            bound = K * 2.0 ** -53 * sum(abs(float(x) * float(y)) for x, y in zip(A.values[i], B.values[j]))
            assert abs(C[i, j] - exact) <= bound
            # transposed-operand guard: element (i, j) uses row j of B (N x K layout)
    # elementwise entry point agrees bit for bit with the row entry point
    ii, jj = np.meshgrid(np.arange(M), np.arange(N), indexing="ij")
    E = oracle.gemm_elems(A.device_array, B.device_array, ii.ravel(), jj.ravel())
    assert np.array_equal(E.reshape(M, N), C)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_numpy_crosscheck(dtype):
    M, N, K = 48, 40, 72
    A = _draw((M, K), "normal", dtype, 0)
    B = _draw((N, K), "normal", dtype, 1)
    C = oracle.gemm_rows(A.device_array, B.device_array, range(M))
    R = A.values.astype(np.float64) @ B.values.astype(np.float64).T
    scale = np.abs(A.values.astype(np.float64)) @ np.abs(B.values.astype(np.float64)).T
    assert np.all(np.abs(C - R) <= 2 * K * 2.0 ** -53 * scale)


def test_integer_inputs_exact():
    M, N, K = 64, 48, 200
    A = _draw((M, K), "int", "bf16", 0)
    B = _draw((N, K), "int", "f32", 1)
    C = oracle.gemm_rows(A.device_array, B.device_array, range(M))
    R = A.values.astype(np.int64) @ B.values.astype(np.int64).T
    assert np.array_equal(C, R.astype(np.float64))


def test_identity_weight_returns_A():
    K = 64
    A = _draw((96, K), "normal", "bf16", 0)
    eye = si.f32_to_bf16_bits(np.eye(K, dtype=np.float32))
    chunks, order = oracle.uniform_schedule(3, 0, 32, 2, "ring")
    C = oracle.ag_gemm(A.device_array, eye, chunks, order)
    assert np.array_equal(C, A.values.astype(np.float64))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_order_invariance_bit_identical(dtype):
    W, S, Q, N, K = 4, 32, 2, 24, 40
    M = W * S
    A = _draw((M, K), "normal", dtype, 0)
    B = _draw((N, K), "normal", dtype, 1)
    ref_chunks, ref_order = oracle.uniform_schedule(1, 0, M, 1, "ring")   # one chunk: unscheduled GEMM
    ref = oracle.ag_gemm(A.device_array, B.device_array, ref_chunks, ref_order)
    assert not np.isnan(ref).any()
    results = []
    for kind in ("ring", "swizzle1d", "rs_ring"):
        ch, od = oracle.uniform_schedule(W, 1, S, Q, kind)
        results.append(oracle.ag_gemm(A.device_array, B.device_array, ch, od))
    for rep in range(3):
        perm = si.draw_permutation(91, rep, (W - 1) * Q)
        ch, od = oracle.uniform_schedule(W, 1, S, Q, "permutation", perm)
        results.append(oracle.ag_gemm(A.device_array, B.device_array, ch, od))
        C, out, log = oracle.gemm_rs(A.device_array, B.device_array, ch, od)
        results.append(C)
        assert log == od
    for C in results:
        assert np.array_equal(C, ref)


def test_rs_outgoing_and_log():
    W, S, Q, N, K = 3, 16, 2, 12, 20
    A = _draw((W * S, K), "normal", "bf16", 0)
    B = _draw((N, K), "normal", "bf16", 1)
    chunks, order = oracle.uniform_schedule(W, 2, S, Q, "rs_ring")
    C, out, log = oracle.gemm_rs(A.device_array, B.device_array, chunks, order)
    assert log == order and chunks[log[-1]].is_local
    for ch in chunks:
        rows = slice(ch.row_begin, ch.row_end)
        if ch.is_local:
            assert np.isnan(out[rows]).all()
        else:
            assert np.array_equal(out[rows], C[rows])


def test_row_subset_matches_full():
    W, S, Q, N, K = 2, 32, 2, 16, 24
    A = _draw((W * S, K), "normal", "f32", 0)
    B = _draw((N, K), "normal", "f32", 1)
    chunks, order = oracle.uniform_schedule(W, 0, S, Q, "ring")
    full = oracle.ag_gemm(A.device_array, B.device_array, chunks, order)
    rows = [0, 5, 33, 63]
    sub = oracle.ag_gemm(A.device_array, B.device_array, chunks, order, row_subset=rows)
    assert np.array_equal(sub[rows], full[rows])
    others = [r for r in range(W * S) if r not in rows]
    assert np.isnan(sub[others]).all()


def test_grouped_matches_per_expert_numpy():
    w = si.Workload(95, "g", "grouped", M=0, N=24, K=32, dtype="bf16", out_dtype="bf16", dist="normal",
                    world=4, n_tokens=64, n_experts=3, topk=2, zipf_s=1.2)
    d = si.draw(w, M=128)
    chunks, order, group_rows = oracle.grouped_schedule(4, 1, d.counts)
    assert sum(group_rows) == 128
    C = oracle.grouped_gemm(d.A.device_array, d.B.device_array, chunks, order)
    off = 0
    for e, n in enumerate(group_rows):
        R = d.A.values[off:off + n].astype(np.float64) @ d.B.values[e].astype(np.float64).T
        assert np.allclose(C[off:off + n], R, rtol=0, atol=1e-15)
        off += n
    # rows of a (source, expert) segment are the tokens that source routed to that expert
    row = 0
    per_src = 64 // 4
    for e in range(3):
        for s in range(4):
            for t in range(s * per_src, (s + 1) * per_src):
                if e in d.routing[t]:
                    assert np.array_equal(d.A.bits[row], d.tokens.bits[t])
                    row += 1


def test_max_rel_error_metric():
    R = np.array([[1.0, -2.0], [0.0, 4.0]])
    assert oracle.max_rel_error(R, R) == 0.0
    rms = math.sqrt((1 + 4 + 0 + 16) / 4)
    G = R.copy()
    G[1, 0] = 0.1                          # near-zero reference entry: denominator is the RMS
    assert oracle.max_rel_error(G, R) == pytest.approx(0.1 / rms)
    G = R.copy()
    G[1, 1] = 4.4
    assert oracle.max_rel_error(G, R) == pytest.approx(0.1)


# ---------------------------------------------------------------------------------
# GEMM + AllReduce (one rank's share)
# ---------------------------------------------------------------------------------
def _ar_case(W, r, S, Q, N, K, dist, dtype="f32", cfg=91):
    """Per-rank K-slices A_s (M x K) and B_s (N x K) of a row-parallel product; rank r's
    view: its own slices, the other ranks' partials of its shard (ascending rank order)
    and the other shards' all-reduced rows."""
    M = W * S
    As = [_draw((M, K), dist, dtype, 0, rep=s, cfg=cfg).values for s in range(W)]      # float32 values
    Bs = [_draw((N, K), dist, dtype, 1, rep=s, cfg=cfg).values for s in range(W)]
    parts = [a.astype(np.float64) @ b.astype(np.float64).T for a, b in zip(As, Bs)]  # numpy fp64 matmul
    full = sum(parts)
    own = slice(r * S, (r + 1) * S)
    partials = np.stack([parts[s][own] for s in range(W) if s != r])
    chunks, order = oracle.uniform_schedule(W, r, S, Q, "rs_ring")
    return As[r], Bs[r], partials, full, parts[r], chunks, order


@pytest.mark.parametrize("W,r,S,Q", [(2, 0, 8, 1), (4, 1, 12, 3), (4, 3, 16, 2), (8, 5, 4, 2)])
def test_ar_equals_the_unsplit_gemm_over_all_ranks_k(W, r, S, Q):
    """An all-reduce of the ranks' K-slice products is the product over the whole K
    (the row-parallel layer's identity): the oracle's reduced own rows, made from its
    own partial plus the others' partials, equal numpy's product of the concatenated
    slices; integer inputs make every sum exact."""
    N, K = 10, 6
    for dist in ("int", "normal"):
        A, B, partials, full, mine, chunks, order = _ar_case(W, r, S, Q, N, K, dist)
        C, out, log = oracle.gemm_ar(A, B, chunks, order, partials, full)
        own = slice(r * S, (r + 1) * S)
        if dist == "int":
            assert np.array_equal(C[own], full[own])
        else:
            np.testing.assert_allclose(C[own], full[own], rtol=0, atol=1e-15 * W * K)
        assert not np.isnan(C).any() and not np.isnan(out).any()
        assert log == list(order)
        for ch in chunks:
            rows = slice(ch.row_begin, ch.row_end)
            if ch.is_local:
                assert np.array_equal(out[rows], C[rows])           # the reduced chunk is sent
            else:
                assert np.array_equal(C[rows], full[rows])          # arrived from its owner
                np.testing.assert_allclose(out[rows], mine[rows], rtol=0, atol=1e-15 * K)   # own partial sent


def test_ar_drops_no_peer():
    """Leaving out any one peer's partial changes the reduced rows."""
    W, r, S, Q, N, K = 4, 2, 8, 2, 6, 5
    A, B, partials, full, mine, chunks, order = _ar_case(W, r, S, Q, N, K, "int")
    C, _, _ = oracle.gemm_ar(A, B, chunks, order, partials, full)
    own = slice(r * S, (r + 1) * S)
    for j in range(W - 1):
        p = partials.copy()
        p[j] = 0
        Cj, _, _ = oracle.gemm_ar(A, B, chunks, order, p, full)
        assert not np.array_equal(Cj[own], C[own])


def test_ar_order_invariance_and_row_subset():
    W, r, S, Q, N, K = 4, 1, 16, 4, 12, 9
    A, B, partials, full, mine, chunks, order = _ar_case(W, r, S, Q, N, K, "normal")
    C, out, _ = oracle.gemm_ar(A, B, chunks, order, partials, full)
    for rep in range(3):
        perm = list(np.random.default_rng(rep).permutation(len(order)))
        C2, out2, log2 = oracle.gemm_ar(A, B, chunks, perm, partials, full)
        assert np.array_equal(C2, C) and np.array_equal(out2, out) and log2 == perm
    rows = [0, 17, 20, 31, 63]
    Cs, outs, _ = oracle.gemm_ar(A, B, chunks, order, partials, full, row_subset=rows)
    assert np.array_equal(Cs[rows], C[rows]) and np.array_equal(outs[rows], out[rows])
