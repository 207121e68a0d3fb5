"""The autotuner's host logic: the search space and the choice of the best
candidate, with stand-in plans (no GPU)."""
import time

import numpy as np
import pytest

import oracle
import paper_2601_20595_amd as csg
from paper_2601_20595_amd import tune


def test_search_space_shape():
    ag = tune.search_space("ag")
    # backends: sdma + 3 copy-workgroup counts; dispatch 2; (split 1 x tail 2) + (split 2 x no tail)
    assert len(ag) == 4 * 2 * 3
    assert ag[0].cfg_dict() == {} and ag[0].chunks_per_shard is None      # the library's default plan first
    assert len(set(ag)) == len(ag)
    for c in ag:
        d = c.cfg_dict()
        assert not (d.get("split_k", 1) > 1 and d.get("tail_split", 0) > 1)
        assert ("copy_workgroups" in d) == (d.get("copy_backend", 0) == 1)
    rs = tune.search_space("rs", chunk_splits=(1, 2))
    kernel = [c for c in rs if c.cfg_dict().get("copy_backend") == 1]
    assert kernel and all("copy_workgroups" not in c.cfg_dict() for c in kernel)   # sends from the epilogue
    assert {c.chunks_per_shard for c in rs} == {1, 2}
    assert len(tune.search_space("grouped", kernel_copies=False)) == 2 * 3
    with pytest.raises(ValueError):
        tune.search_space("gemm")
    tiled = tune.search_space("ag", kernel_copies=False, tiles=(None, (256, 128), (128, 128)))
    assert len(tiled) == 3 * len(tune.search_space("ag", kernel_copies=False))
    shapes = {(c.cfg_dict().get("bm"), c.cfg_dict().get("bn"), c.cfg_dict().get("bk")) for c in tiled}
    assert shapes == {(None, None, None), (256, 128, 64), (128, 128, 64)}


class _FakePlan:
    def __init__(self, ms, fail=False):
        self.ms, self.fail, self.closed, self.calls = ms, fail, False, 0

    def check(self):
        if self.fail:
            raise csg.CsgError(csg.CSG_ERR_TIMEOUT, "csg_plan_check", "stand-in failure")

    def close(self):
        self.closed = True


def test_autotune_picks_fastest_and_records_rejections():
    cands = tune.search_space("ag", dispatch=(1,), split_k=(1,), tail=((0, 0),), copy_workgroups=(32, 64))
    assert len(cands) == 3
    speed = {0: 3.0, 1: 1.0, 2: None}        # candidate index -> ms per call (None: rejected)
    made = []

    def make(c):
        i = cands.index(c)
        if speed[i] is None:
            raise csg.CsgError(csg.CSG_ERR_UNSUPPORTED, "csg_plan_create", "stand-in rejection")
        p = _FakePlan(speed[i])
        made.append(p)
        return p

    def call(p, mode):
        assert mode == "overlap"
        p.calls += 1
        time.sleep(p.ms * 1e-3)

    res, best_plan = tune.autotune(make, call, cands, steps=3, warmup=1, keep_best=True)
    assert res.best == cands[1]
    assert best_plan is made[1] and not best_plan.closed
    assert made[0].closed                     # measured and released
    assert made[0].calls == 4 and made[1].calls == 4
    st = {t.candidate: t.status for t in res.trials}
    assert st[cands[0]] == "ok" and st[cands[2]].startswith("rejected")
    assert res.best_ms == pytest.approx(1.0, abs=5.0)
    assert [r["status"] for r in res.table()] == ["ok", "ok", st[cands[2]]]


def test_autotune_failures_and_empty():
    cands = tune.search_space("ag", dispatch=(1,), split_k=(1,), tail=((0, 0),), copy_workgroups=(32,))
    plans = [_FakePlan(0.1, fail=True), _FakePlan(0.2)]
    res, keep = tune.autotune(lambda c: plans[cands.index(c)], lambda p, m: None, cands, steps=1, warmup=0)
    assert keep is None and res.best == cands[1]
    assert res.trials[0].status.startswith("failed") and plans[0].closed and plans[1].closed
    with pytest.raises(ValueError):
        tune.autotune(lambda c: None, lambda p, m: None, [])
    with pytest.raises(RuntimeError):
        tune.autotune(lambda c: _FakePlan(0, fail=True), lambda p, m: None, cands[:1], steps=1, warmup=0)


def test_uniform_plan_factory_builds_host_plans_and_rejects_unaligned_epilogue_sends():
    make = tune.uniform_plan_factory("rs", 1024, 64, 64, "bf16", "bf16", world=4, rank=1, shard_rows=256,
                                     order="rs_ring", default_q=1, device=-1)
    kernel = tune.Candidate(2, (("copy_backend", 1),))        # 128-row chunks, 256-row tiles
    with pytest.raises(csg.CsgError) as e:
        make(kernel)
    assert e.value.status == csg.CSG_ERR_UNSUPPORTED
    p = make(tune.Candidate(None, (("copy_backend", 1),)))   # default Q = 1: 256-row chunks
    assert p.info.n_chunks == 4
    p.close()
    perm_make = tune.uniform_plan_factory("ag", 1024, 64, 64, "bf16", "bf16", world=4, rank=0, shard_rows=256,
                                          order="permutation", default_q=2,
                                          perm_for=lambda q: list(reversed(range(3 * q))),
                                          delays_for=lambda q: [1.0] * (3 * q), device=-1)
    p = perm_make(tune.Candidate(4, ()))
    assert p.info.n_chunks == 16
    p.close()


def test_search_space_grid_dimension():
    """Grid sizes are a search dimension; 0 keeps the library's default grid, which
    stays the first candidate."""
    base = tune.search_space("ag", kernel_copies=False)
    grids = tune.search_space("ag", kernel_copies=False, grids=(0, 224))
    assert grids[0] == base[0]
    assert len(grids) == 2 * len(base)
    assert sum(1 for c in grids if ("num_workgroups", 224) in c.cfg) == len(base)


def test_search_space_intra_order_and_wave_tail_dimensions():
    """The intra-chunk order and the wave-tail split are search dimensions; the default
    candidate stays first, and the wave-tail split is only combined with per-die
    dispatch and no other split. Every candidate builds a host plan whose map equals
    the oracle's for its intra order."""
    base = tune.search_space("ag", kernel_copies=False)
    sp = tune.search_space("ag", kernel_copies=False, intra=((0, 0), (1, 2), (1, 8)), tail_wave=(0, 2))
    assert sp[0] == base[0]
    # every other combination comes once in raster order and once per band height
    assert sum(1 for c in sp if ("intra_order", 1) in c.cfg) == 2 * sum(1 for c in sp if ("intra_order", 1) not in c.cfg)
    for c in sp:
        d = c.cfg_dict()
        if d.get("tail_wave"):
            assert d.get("tile_dispatch", 1) != 2 and "split_k" not in d and "tail_split" not in d
    make = tune.uniform_plan_factory("ag", 4 * 512, 768, 256, "bf16", "bf16", 4, 1, 512, "ring", 2, device=-1)
    chunks, order = oracle.uniform_schedule(4, 1, 512, 2, "ring")
    for c in sp:
        p = make(c)
        d = c.cfg_dict()
        dm = oracle.dep_map(chunks, order, 2048, 768, 256, 256, intra_order=d.get("intra_order", 0),
                            group_m=d.get("group_m", 8))
        assert np.array_equal(p.get_map()["tile_order"], dm.order), c.label()
        p.close()


def test_bench_tuned_plan_configurations_are_accepted():
    """Every plan configuration bench.py measures as a workload's tuned plan is one the
    library accepts for that workload's shape and schedule (host-only plans)."""
    import bench
    import paper_2601_20595_amd as csg
    import seeded_inputs as si
    for cid, cfg in bench.TUNED_PLAN_CFG.items():
        w = si.WORKLOADS[cid]
        d = si.draw(w) if w.op == "grouped" or w.order == "permutation" else None
        if w.op == "grouped":
            s = csg.Schedule.grouped(w.world, w.rank, d.counts)
            gr = [int(x) for x in d.counts.sum(axis=0)]
        else:
            s = csg.Schedule.uniform(w.world, w.rank, w.shard_rows, w.chunks_per_shard, w.order,
                                     d.perm if d is not None else None)
            gr = None
        p = csg.Plan(w.op, w.M, w.N, w.K, w.dtype, w.out_dtype, s, group_rows=gr, cfg=dict(cfg), device=-1)
        assert (p.info.bm, p.info.bn) == (cfg.get("bm", 256), cfg.get("bn", 256))
        p.close()
        s.close()


def test_search_space_copy_split_dimension():
    """Cutting chunk copies into pieces is a dimension of the copy-engine candidates only;
    the default candidate stays first and every copy-engine candidate comes once whole
    and once per piece count."""
    base = tune.search_space("rs")
    sp = tune.search_space("rs", copy_split=(0, 2, 4))
    assert sp[0] == base[0]
    sdma = [c for c in sp if ("copy_backend", 1) not in c.cfg]
    for c in sp:
        d = c.cfg_dict()
        if d.get("copy_split"):
            assert d.get("copy_backend", 0) == 0
    assert len(sdma) == 3 * sum(1 for c in sdma if "copy_split" not in c.cfg_dict())
    assert len(sp) - len(sdma) == len(base) - sum(1 for c in base if ("copy_backend", 1) not in c.cfg)


def test_search_space_tail_taper_dimension():
    """The tapered tail split is a dimension only of candidates with a tail split."""
    tails = ((0, 0), (2, 4), (4, 12))
    base = tune.search_space("ag", kernel_copies=False, tail=tails)
    sp = tune.search_space("ag", kernel_copies=False, tail=tails, tail_taper=(0, 1))
    assert sp[0] == base[0]
    tapered = [c for c in sp if c.cfg_dict().get("tail_taper")]
    assert all(c.cfg_dict().get("tail_split", 0) > 1 for c in tapered)
    assert len(tapered) == sum(1 for c in base if c.cfg_dict().get("tail_split", 0) > 1)
    assert len(sp) == len(base) + len(tapered)

