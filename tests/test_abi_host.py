"""The C-ABI library on the host (no GPU): it loads, exports every declared symbol,
and its schedules, dependence maps and tile orders equal the oracle's bit for bit.
No compute call is made here; device work is covered by the -m gpu tests."""
import os
import re

import numpy as np
import pytest

import oracle
import paper_2601_20595_amd as csg
import seeded_inputs as si

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_library_exports_every_declared_symbol():
    header = open(os.path.join(ROOT, "include", "csg.h")).read()
    declared = set(re.findall(r"\b(csg_[a-z_0-9]+)\s*\(", header))
    assert declared == set(csg.ABI_FUNCTIONS)
    lib = csg._lib()
    for name in declared:
        assert hasattr(lib, name), name
    assert csg.csg_version().startswith("csg")
    assert csg.csg_status_str(csg.CSG_ERR_TIMEOUT) == "CSG_ERR_TIMEOUT"


def _oracle_chunks_tuple(chunks):
    return [(c.row_begin, c.row_end, c.src_rank, c.group, int(c.is_local)) for c in chunks]


@pytest.mark.parametrize("kind", ["ring", "swizzle1d", "rs_ring", "permutation"])
@pytest.mark.parametrize("W,r,S,Q", [(1, 0, 64, 1), (2, 1, 128, 2), (8, 0, 1024, 4), (8, 5, 2048, 16), (3, 2, 96, 3)])
def test_uniform_schedule_matches_oracle(kind, W, r, S, Q):
    perm = si.draw_permutation(7, W * 100 + r, (W - 1) * Q) if kind == "permutation" else None
    ch, od = oracle.uniform_schedule(W, r, S, Q, kind, perm)
    s = csg.Schedule.uniform(W, r, S, Q, kind, perm)
    chunks, order = s.get()
    assert chunks == _oracle_chunks_tuple(ch)
    assert order == od


@pytest.mark.parametrize("rep", [0, 1, 2])
def test_grouped_schedule_matches_oracle(rep):
    w = si.WORKLOADS[5]
    routing = si.draw_topk_routing(5, rep, 4096, 8, 2, 1.2)
    _, counts = si.grouped_layout(routing, 8, 8)
    counts[3, 7] = 0                               # force an empty segment
    for r in (0, 5):
        ch, od, gr = oracle.grouped_schedule(8, r, counts)
        s = csg.Schedule.grouped(8, r, counts)
        chunks, order = s.get()
        assert chunks == _oracle_chunks_tuple(ch)
        assert order == od


MAP_CASES = [
    # (op, W, r, S, Q, kind, N, BM, BN)
    ("ag", 2, 0, 128, 2, "permutation", 256, 64, 64),
    ("ag", 8, 0, 1024, 4, "ring", 1792, 256, 256),
    ("ag", 8, 3, 1024, 4, "swizzle1d", 1792, 256, 224),
    ("rs", 8, 0, 1024, 4, "rs_ring", 4096, 256, 256),
    ("rs", 4, 1, 96, 2, "rs_ring", 100, 64, 48),            # straddling, ragged N
    ("ag", 8, 0, 2048, 16, "permutation", 3584, 256, 256),  # 2 chunks per tile
    ("ag", 3, 2, 160, 2, "permutation", 600, 256, 256),     # straddling, ragged M and N
    ("ag", 4, 1, 64, 4, "ring", 64, 96, 32),                # tiles spanning 6 chunks
]


@pytest.mark.parametrize("intra", [(0, 0), (1, 2), (1, 3), (1, 8)], ids=lambda i: "intra%d-g%d" % i)
@pytest.mark.parametrize("case", MAP_CASES, ids=lambda c: "-".join(map(str, c)))
def test_plan_map_matches_oracle_bit_exact(case, intra):
    op, W, r, S, Q, kind, N, BM, BN = case
    io, g = intra
    perm = si.draw_permutation(11, W + r, (W - 1) * Q) if kind == "permutation" else None
    ch, od = oracle.uniform_schedule(W, r, S, Q, kind, perm)
    dm = oracle.dep_map(ch, od, W * S, N, BM, BN, producer=(op == "rs"), intra_order=io, group_m=max(g, 1))
    s = csg.Schedule.uniform(W, r, S, Q, kind, perm)
    p = csg.Plan(op, W * S, N, 64, "bf16", "bf16", s, cfg={"bm": BM, "bn": BN, "intra_order": io, "group_m": g},
                 device=-1)
    m = p.get_map()
    assert np.array_equal(m["tile_ptr"], dm.tile_ptr)
    assert np.array_equal(m["tile_chunks"], dm.tile_chunks)
    assert np.array_equal(m["chunk_ptr"], dm.chunk_ptr)
    assert np.array_equal(m["chunk_tiles"], dm.chunk_tiles)
    assert np.array_equal(m["tile_order"], dm.order)


@pytest.mark.parametrize("intra", [(0, 0), (1, 2)], ids=lambda i: "intra%d-g%d" % i)
@pytest.mark.parametrize("BM,BN", [(256, 256), (128, 64), (96, 128)])
def test_grouped_plan_map_matches_oracle(BM, BN, intra):
    io, g = intra
    routing = si.draw_topk_routing(5, 3, 2048, 8, 2, 1.2)
    _, counts = si.grouped_layout(routing, 8, 8)
    ch, od, gr = oracle.grouped_schedule(8, 2, counts)
    M = sum(gr)
    dm = oracle.dep_map(ch, od, M, 1792, BM, BN, group_rows=gr, intra_order=io, group_m=max(g, 1))
    s = csg.Schedule.grouped(8, 2, counts)
    p = csg.Plan("grouped", M, 1792, 4096, "bf16", "bf16", s, group_rows=gr,
                 cfg={"bm": BM, "bn": BN, "intra_order": io, "group_m": g}, device=-1)
    m = p.get_map()
    assert np.array_equal(m["tile_ptr"], dm.tile_ptr)
    assert np.array_equal(m["tile_chunks"], dm.tile_chunks)
    assert np.array_equal(m["chunk_tiles"], dm.chunk_tiles)
    assert np.array_equal(m["tile_order"], dm.order)


def test_general_schedule_and_order_invariance_of_map_shape():
    chunks = [(0, 40, 0, 0, 1), (40, 100, 1, 0, 0), (100, 128, 1, 0, 0)]
    for order in ([0, 1, 2], [0, 2, 1], [2, 1, 0]):
        s = csg.Schedule.create(chunks, order)
        p = csg.Plan("ag", 128, 64, 64, "bf16", "bf16", s, cfg={"bm": 32, "bn": 64}, device=-1)
        och = [oracle.Chunk(*c[:4], bool(c[4])) for c in chunks]
        dm = oracle.dep_map(och, order, 128, 64, 32, 64)
        m = p.get_map()
        assert np.array_equal(m["tile_chunks"], dm.tile_chunks)
        assert np.array_equal(m["tile_order"], dm.order)


def _status(fn, *a, **k):
    try:
        fn(*a, **k)
    except csg.CsgError as e:
        return e.status
    return csg.CSG_OK


def test_validation_errors():
    bad = [
        ([(0, 4, 0, 0, 1), (5, 8, 1, 0, 0)], [0, 1]),   # gap
        ([(0, 5, 0, 0, 1), (4, 8, 1, 0, 0)], [0, 1]),   # overlap
        ([(0, 4, 0, 0, 1), (4, 8, 1, 0, 0)], [0, 0]),   # not a permutation
        ([(0, 0, 0, 0, 1), (0, 8, 1, 0, 0)], [0, 1]),   # empty chunk
        ([(0, 4, 0, 0, 1), (4, 8, 1, 0, 0)], [0, 2]),   # id out of range
    ]
    for chunks, order in bad:
        assert _status(csg.csg_schedule_create, chunks, order) == csg.CSG_ERR_INVALID
    assert _status(csg.csg_schedule_uniform, 2, 2, 64, 2, "ring") == csg.CSG_ERR_INVALID      # rank >= world
    assert _status(csg.csg_schedule_uniform, 2, 0, 10, 3, "ring") == csg.CSG_ERR_INVALID      # S % Q
    assert _status(csg.csg_schedule_uniform, 2, 0, 64, 2, "permutation", [0, 0]) == csg.CSG_ERR_INVALID
    assert _status(csg.csg_schedule_uniform, 2, 0, 64, 2, "permutation", [0, 5]) == csg.CSG_ERR_INVALID
    assert _status(csg.csg_schedule_grouped, 2, 0, np.zeros((2, 3))) == csg.CSG_ERR_INVALID   # all empty
    s = csg.Schedule.uniform(2, 0, 64, 2, "ring")
    # M must equal the rows the chunks cover
    assert _status(csg.Plan, "ag", 100, 64, 64, "bf16", "bf16", s, device=-1) == csg.CSG_ERR_INVALID
    assert _status(csg.Plan, "ag", 128, 0, 64, "bf16", "bf16", s, device=-1) == csg.CSG_ERR_INVALID
    # group rows only for the grouped op, and must sum to M
    assert _status(csg.Plan, "ag", 128, 64, 64, "bf16", "bf16", s, group_rows=[128], device=-1) == csg.CSG_ERR_INVALID
    g = csg.Schedule.grouped(2, 0, [[3, 1], [2, 0]])
    assert _status(csg.Plan, "grouped", 6, 64, 64, "bf16", "bf16", g, group_rows=[4, 2], device=-1) \
        == csg.CSG_ERR_INVALID
    assert _status(csg.Plan, "grouped", 6, 64, 64, "bf16", "bf16", g, group_rows=[5, 1], device=-1) == csg.CSG_OK
    # bad configuration
    assert _status(csg.Plan, "ag", 128, 64, 64, "bf16", "bf16", s, cfg={"copy_engines": 99}, device=-1) \
        == csg.CSG_ERR_INVALID
    assert _status(csg.Plan, "ag", 128, 64, 64, "bf16", "bf16", s, cfg={"tail_split": -1}, device=-1) \
        == csg.CSG_ERR_INVALID
    for bad in ({"intra_order": 2}, {"intra_order": -1}, {"group_m": -1}, {"tail_wave": 65}, {"tail_wave": -1},
                {"copy_split": -1}, {"copy_split": 33}, {"tail_taper": -1}, {"tail_taper": 2}):
        assert _status(csg.Plan, "ag", 128, 64, 64, "bf16", "bf16", s, cfg=bad, device=-1) == csg.CSG_ERR_INVALID
    # pieces of chunk copies: copy engines only, and not for the all-reduce's copies
    assert _status(csg.Plan, "ag", 128, 64, 64, "bf16", "bf16", s, cfg={"copy_split": 4}, device=-1) == csg.CSG_OK
    assert _status(csg.Plan, "ag", 128, 64, 64, "bf16", "bf16", s, cfg={"copy_split": 4, "copy_backend": 1},
                   device=-1) == csg.CSG_ERR_UNSUPPORTED
    assert _status(csg.Plan, "ar", 128, 64, 64, "bf16", "bf16", s, cfg={"copy_split": 2}, device=-1) \
        == csg.CSG_ERR_UNSUPPORTED
    # a grid given with the wave-tail split must cover every die evenly
    assert _status(csg.Plan, "ag", 128, 64, 64, "bf16", "bf16", s, cfg={"tail_wave": 2, "num_workgroups": 12},
                   device=-1) == csg.CSG_ERR_INVALID
    # split plans: a given grid must cover every die evenly (each die's list gets its share)
    assert _status(csg.Plan, "ag", 128, 64, 64, "bf16", "bf16", s, cfg={"split_k": 2, "num_workgroups": 12},
                   device=-1) == csg.CSG_ERR_INVALID
    assert _status(csg.Plan, "ag", 128, 64, 64, "bf16", "bf16", s, cfg={"split_k": 2, "num_workgroups": 16},
                   device=-1) == csg.CSG_OK


def test_shapes_the_kernels_do_not_cover_are_rejected():
    """K must be a multiple of the main loop's K step (64 for bf16, 16 for fp32) and N a
    multiple of 4 (a store run is four columns): other shapes are refused at plan
    creation, for every GEMM op, instead of reading past a row or storing a partial run."""
    s = csg.Schedule.uniform(2, 0, 256, 2, "ring")
    rs = csg.Schedule.uniform(2, 0, 256, 2, "rs_ring")
    for op, sched in (("ag", s), ("rs", rs), ("ar", rs)):
        assert _status(csg.Plan, op, 512, 64, 96, "bf16", "bf16", sched, device=-1) == csg.CSG_ERR_UNSUPPORTED, op
        assert _status(csg.Plan, op, 512, 64, 24, "f32", "f32", sched, device=-1) == csg.CSG_ERR_UNSUPPORTED, op
        assert _status(csg.Plan, op, 512, 66, 64, "bf16", "bf16", sched, device=-1) == csg.CSG_ERR_UNSUPPORTED, op
        assert _status(csg.Plan, op, 512, 64, 128, "bf16", "bf16", sched, device=-1) == csg.CSG_OK, op
        assert _status(csg.Plan, op, 512, 68, 32, "f32", "f32", sched, device=-1) == csg.CSG_OK, op


def test_every_op_rejects_more_chunks_than_the_kernels_track():
    """The kernels keep one bit per chunk of the chunks a workgroup has seen ready; the
    producers (GEMM-RS, GEMM-AR) wait on that bitmap too, before rewriting a chunk's rows
    of C. A plan with more chunks than the bitmap holds is rejected for every op."""
    W, S, Q = 2, 4096, 4096                      # 8192 one-row chunks
    s = csg.Schedule.uniform(W, 0, S, Q, "rs_ring")
    for op in ("ag", "rs", "ar"):
        try:
            csg.Plan(op, W * S, 64, 64, "bf16", "bf16", s, device=-1)
            raise AssertionError("%s plan with %d chunks accepted" % (op, W * Q))
        except csg.CsgError as e:
            assert e.status == csg.CSG_ERR_UNSUPPORTED, op
            assert "at most 4096 chunks" in str(e), (op, str(e))
    ok = csg.Schedule.uniform(W, 0, 2048, 2048, "rs_ring")   # exactly 4096 chunks
    for op in ("ag", "rs", "ar"):
        assert _status(csg.Plan, op, W * 2048, 64, 64, "bf16", "bf16", ok, device=-1) == csg.CSG_OK, op


def test_kernel_copy_backend_validation():
    s = csg.Schedule.uniform(2, 0, 64, 2, "ring")
    for bad in ({"copy_backend": 2}, {"copy_backend": -1}, {"copy_workgroups": -1}, {"copy_workgroups": 5000}):
        assert _status(csg.Plan, "ag", 128, 64, 64, "bf16", "bf16", s, cfg=bad, device=-1) == csg.CSG_ERR_INVALID
    kc = {"copy_backend": "kernel"}
    assert _status(csg.Plan, "ag", 128, 64, 64, "bf16", "bf16", s, cfg=kc, device=-1) == csg.CSG_OK
    # GEMM-RS sends from the tile epilogue: a tile must not mix rows of two chunks, so
    # every chunk starts on a multiple of bm (256 for bf16 by default, 64 for fp32)
    rs = csg.Schedule.uniform(4, 1, 512, 2, "rs_ring")                 # 256-row chunks
    assert _status(csg.Plan, "rs", 2048, 64, 64, "bf16", "bf16", rs, cfg=kc, device=-1) == csg.CSG_OK
    rs = csg.Schedule.uniform(4, 1, 256, 2, "rs_ring")                 # 128-row chunks
    assert _status(csg.Plan, "rs", 1024, 64, 64, "bf16", "bf16", rs, cfg=kc, device=-1) == csg.CSG_ERR_UNSUPPORTED
    assert _status(csg.Plan, "rs", 1024, 64, 64, "f32", "f32", rs, cfg=kc, device=-1) == csg.CSG_OK
    assert _status(csg.Plan, "rs", 1024, 64, 64, "bf16", "bf16", rs, device=-1) == csg.CSG_OK   # copy engines


def test_host_only_plan_cannot_run_and_delays_are_checked():
    s = csg.Schedule.uniform(4, 0, 64, 2, "ring")
    p = csg.Plan("ag", 256, 64, 64, "bf16", "bf16", s, device=-1)
    assert _status(p.ag_gemm, 16, 16, 16, 16) == csg.CSG_ERR_STATE
    assert _status(p.gemm_rs, 16, 16, 16, 16) == csg.CSG_ERR_INVALID      # wrong op for this plan
    assert _status(p.set_copy_delays, [1.0] * 5) == csg.CSG_ERR_INVALID   # needs 6 (remote chunks)
    assert _status(p.set_copy_delays, [1.0] * 6) == csg.CSG_OK
    assert _status(p.set_copy_delays, [-1.0] * 6) == csg.CSG_ERR_INVALID
    assert _status(p.set_copy_delays, None) == csg.CSG_OK
    assert p.info.num_workgroups == 0
    assert _status(p.kernel_times, 4) == csg.CSG_ERR_STATE               # nothing ever ran
    assert _status(p.kernel_times, -1) == csg.CSG_ERR_INVALID


def test_allreduce_plans_map_like_reduce_scatter_and_validate():
    s = csg.Schedule.uniform(4, 1, 256, 2, "rs_ring")
    ar = csg.Plan("ar", 1024, 320, 64, "bf16", "bf16", s, device=-1)
    rs = csg.Plan("rs", 1024, 320, 64, "bf16", "bf16", s, device=-1)
    m_ar, m_rs = ar.get_map(), rs.get_map()
    for k in m_rs:
        assert np.array_equal(np.asarray(m_ar[k]), np.asarray(m_rs[k])), k
    assert _status(csg.Plan, "ar", 1024, 320, 64, "bf16", "bf16", s, cfg={"split_k": 2}, device=-1) \
        == csg.CSG_ERR_UNSUPPORTED
    assert _status(csg.Plan, "ar", 1024, 320, 64, "bf16", "bf16", s, cfg={"copy_backend": "kernel"}, device=-1) \
        == csg.CSG_ERR_UNSUPPORTED
    # own shard rows 100..199 do not start on a 256-row tile (fp32 tiles are 64 rows: also not)
    s100 = csg.Schedule.uniform(4, 1, 100, 2, "rs_ring")
    assert _status(csg.Plan, "ar", 400, 64, 64, "bf16", "bf16", s100, device=-1) == csg.CSG_ERR_UNSUPPORTED
    assert _status(csg.Plan, "ar", 400, 64, 64, "f32", "f32", s100, device=-1) == csg.CSG_ERR_UNSUPPORTED
    s128 = csg.Schedule.uniform(4, 1, 128, 2, "rs_ring")
    assert _status(csg.Plan, "ar", 512, 64, 64, "f32", "f32", s128, device=-1) == csg.CSG_OK
    # unequal chunks; local chunks that are not contiguous
    uneq = csg.Schedule.create([(0, 64, 0, 0, 1), (64, 192, 1, 0, 0)], [1, 0])
    assert _status(csg.Plan, "ar", 192, 64, 64, "f32", "f32", uneq, device=-1) == csg.CSG_ERR_UNSUPPORTED
    split = csg.Schedule.create([(0, 64, 0, 0, 1), (64, 128, 1, 0, 0), (128, 192, 0, 0, 1), (192, 256, 1, 0, 0)],
                                [1, 3, 0, 2])
    assert _status(csg.Plan, "ar", 256, 64, 64, "f32", "f32", split, device=-1) == csg.CSG_ERR_UNSUPPORTED
    assert _status(ar.gemm_ar, 16, 16, 16, 16, 16, 16, 16) == csg.CSG_ERR_STATE        # host-only plan
    assert _status(rs.gemm_ar, 16, 16, 16, 16, 16, 16, 16) == csg.CSG_ERR_INVALID      # wrong op


def test_attention_plans_validate():
    s = csg.Schedule.uniform(4, 1, 256, 2, "ring")                       # 128-row key chunks
    p = csg.AttnPlan(8, 2, 128, 300, s, device=-1)
    assert p.info.n_chunks == 8
    assert _status(p.ring_attn, 16, 16, 16, 16, 16, 16, 16) == csg.CSG_ERR_STATE          # host-only plan
    assert _status(p.ag_gemm, 16, 16, 16, 16) == csg.CSG_ERR_INVALID                      # not a GEMM plan
    assert _status(csg.AttnPlan, 8, 2, 64, 300, s, device=-1) == csg.CSG_ERR_UNSUPPORTED    # head dim 128 only
    assert _status(csg.AttnPlan, 8, 3, 128, 300, s, device=-1) == csg.CSG_ERR_INVALID       # heads % kv heads
    assert _status(csg.AttnPlan, 8, 2, 128, 0, s, device=-1) == csg.CSG_ERR_INVALID
    assert _status(csg.AttnPlan, 8, 2, 128, 300, s, cfg={"copy_backend": 1}, device=-1) == csg.CSG_ERR_UNSUPPORTED
    odd = csg.Schedule.uniform(4, 1, 96, 1, "ring")                         # 96-row chunks
    assert _status(csg.AttnPlan, 8, 2, 128, 300, odd, device=-1) == csg.CSG_ERR_UNSUPPORTED
    gemm = csg.Plan("ag", 1024, 64, 64, "bf16", "bf16", s, device=-1)
    assert _status(csg.csg_ring_attn, gemm.handle, 16, 16, 16, 16, 16, 16, 16) == csg.CSG_ERR_INVALID


def test_binding_checks_tensor_arguments():
    """The binding checks a tensor before passing its pointer: contiguous, large enough
    for the plan's shape, on a GPU (raw pointers and None pass unchecked)."""
    torch = pytest.importorskip("torch")
    from paper_2601_20595_amd import _buf
    big = torch.zeros(64, 64, dtype=torch.int16)
    with pytest.raises(ValueError, match="contiguous"):
        _buf(big.t(), 64 * 64 * 2, "a")
    with pytest.raises(ValueError, match="holds 8192 bytes"):
        _buf(big, 64 * 64 * 2 + 1, "a")
    with pytest.raises(ValueError, match="GPU tensor"):
        _buf(big, 64 * 64 * 2, "a")
    _buf(None, 1 << 20, "a")
    _buf(12345, 1 << 20, "a")


def _header_structs():
    """Field names and C types of every `typedef struct { ... } name;` in include/csg.h,
    in declaration order (comma-separated declarators expanded)."""
    text = open(os.path.join(os.path.dirname(__file__), "..", "include", "csg.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    out = {}
    for body, name in re.findall(r"typedef struct\s*\{(.*?)\}\s*(\w+)\s*;", text, flags=re.S):
        fields = []
        for decl in body.split(";"):
            decl = decl.strip()
            if not decl:
                continue
            ctype, names = decl.split(None, 1)
            fields += [(n.strip(), ctype) for n in names.split(",")]
        out[name] = fields
    return out


def test_binding_structs_match_the_header():
    """The ctypes structures of the binding list the header's fields in the header's
    order with the same widths, so a field added to the C ABI cannot shift the others."""
    import ctypes
    widths = {"int32_t": ctypes.c_int32, "uint32_t": ctypes.c_uint32, "int64_t": ctypes.c_int64,
              "uint64_t": ctypes.c_uint64}
    structs = _header_structs()
    for name in ("csg_chunk", "csg_plan_cfg", "csg_plan_info", "csg_trace_unit", "csg_diag"):
        assert name in structs, name
        py = getattr(csg, name)._fields_
        assert [f for f, _ in py] == [f for f, _ in structs[name]], name
        for (f, t), (_, ct) in zip(py, structs[name]):
            assert ctypes.sizeof(t) == ctypes.sizeof(widths[ct]), (name, f)
