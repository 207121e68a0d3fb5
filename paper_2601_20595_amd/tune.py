"""Enumerate-and-measure autotuner for chunk-scheduled GEMM plans.

The paper's compiler generates every valid implementation of an operator (the
chunk split factor, the tile configuration, the intra-chunk and dispatch order, and
the communication realization), measures each end to end and keeps the fastest
(Section 5.2, communication code generation; Evaluation, the chunk-size and
tile-order ablations). This module does the same over the knobs this library
exposes, for one operator at one shape:

  - chunks per shard (the chunk split factor; only for uniform schedules): every
    split gives the bit-identical product, as each output row depends on one chunk
    and each tile's K order is fixed;
  - tile dispatch (per-die tickets, or a static deal that gives each die consecutive
    entries of every round);
  - the intra-chunk tile order (raster, or bands of group_m row tiles visited
    column by column; Section 5.2, intra-chunk swizzle; Section 5.3, intra-tile
    orders);
  - the wave-tail split (each die's last partial wave of tiles split along K);
  - split-K for every tile, or for the tiles on the overlap's critical path;
  - the copy realization: copy engines, or the kernel's own workgroups with a
    given number of copy workgroups;
  - the tile shape (bf16 consumers: 256x256, 256x128, 128x256, 128x128), off by
    default: smaller tiles finish a chunk sooner after it lands, at a lower MFMA
    efficiency per tile.

Each candidate is timed as back-to-back calls in overlap mode (the steady state
of a loop over layers), bracketed by csg_plan_check, which waits for the plan's
last kernel and every copy. Candidates the library rejects (CsgError at plan
creation, e.g. GEMM-RS sends from the epilogue with chunks not aligned to the
tile) are recorded with their error and skipped. Host logic only: every step of
the measured path runs in the library's kernels and copies.
"""
from __future__ import annotations

import itertools
import time
from dataclasses import dataclass, field
from typing import Callable, Dict, List, Optional, Sequence, Tuple

from . import CsgError, Plan, Schedule


@dataclass(frozen=True)
class Candidate:
    """One point of the search space: a chunk split (None: the caller's schedule)
    and a plan configuration (csg_plan_cfg fields)."""
    chunks_per_shard: Optional[int]
    cfg: Tuple[Tuple[str, int], ...]

    def cfg_dict(self) -> dict:
        return dict(self.cfg)

    def label(self) -> str:
        parts = [] if self.chunks_per_shard is None else ["Q=%d" % self.chunks_per_shard]
        parts += ["%s=%s" % kv for kv in self.cfg]
        return " ".join(parts) or "defaults"


@dataclass
class Trial:
    candidate: Candidate
    ms_per_step: Optional[float]  # None if the candidate could not run
    status: str                   # "ok", or why it was skipped


@dataclass
class TuneResult:
    best: Candidate
    best_ms: float
    trials: List[Trial] = field(default_factory=list)

    def table(self) -> List[dict]:
        return [{"candidate": t.candidate.label(), "ms_per_step": t.ms_per_step, "status": t.status}
                for t in self.trials]


def _cfg(**kw) -> Tuple[Tuple[str, int], ...]:
    return tuple(sorted((k, int(v)) for k, v in kw.items() if v is not None))


def search_space(op: str, chunk_splits: Sequence[Optional[int]] = (None,), dispatch: Sequence[int] = (1, 2),
                 split_k: Sequence[int] = (1, 2), tail: Sequence[Tuple[int, int]] = ((0, 0), (2, 8)),
                 copy_workgroups: Sequence[int] = (32, 64, 128), sdma: bool = True,
                 kernel_copies: bool = True, tiles: Sequence[Optional[Tuple[int, int]]] = (None,),
                 grids: Sequence[int] = (0,), intra: Sequence[Tuple[int, int]] = ((0, 0),),
                 tail_wave: Sequence[int] = (0,), copy_split: Sequence[int] = (0,),
                 tail_taper: Sequence[int] = (0,)) -> List[Candidate]:
    """Candidates in a fixed order (the first one is the library's default plan).

    op: "ag", "rs" or "grouped". GEMM-RS has no copy workgroups (its kernel
    realization sends from the epilogue), so one kernel candidate replaces the
    copy-workgroup sweep. Split-K combined with a tail split is left out (the tail
    split already covers the critical tiles). tiles: (bm, bn) shapes to try, None for
    the library's default tile. grids: persistent grid sizes to try, 0 for one
    workgroup per co-resident slot (the default); a grid that divides the tile count
    into whole waves (224 for 896 tiles on 256 CUs) keeps the waves in step and the
    workgroups sharing a die's L2 at the same K steps. intra: (intra_order, group_m)
    pairs, (0, 0) the raster order. tail_wave: maximum K-slices for each die's last
    partial wave (0 = off); only combined with per-die dispatch and no other split.
    copy_split: the most pieces a chunk copy may be cut into on idle copy engines
    (0 = whole chunks); copy-engine candidates only. tail_taper: 1 = the tail split
    tapers from tail_split to 1 over the tail chunks; only with a tail split."""
    if op not in ("ag", "rs", "grouped"):
        raise ValueError("unknown op %r" % op)
    backends: List[Tuple[int, Optional[int]]] = []
    if sdma:
        backends.append((0, None))
    if kernel_copies:
        if op == "rs":
            backends.append((1, None))
        else:
            backends += [(1, cw) for cw in copy_workgroups]
    out: List[Candidate] = []
    seen = set()
    for q, (be, cw), disp, sk, (ts, tc), tile, grid, (io, gm), tw, cs, tt in itertools.product(
            chunk_splits, backends, dispatch, split_k, tail, tiles, grids, intra, tail_wave, copy_split, tail_taper):
        if tt and not (ts > 1 and tc > 1):
            continue
        if sk > 1 and ts > 1:
            continue
        if tw > 1 and (disp == 2 or sk > 1 or ts > 1):
            continue
        if cs > 1 and be != 0:
            continue
        bm, bn = tile if tile is not None else (None, None)
        c = Candidate(q, _cfg(copy_backend=be or None, copy_workgroups=cw, tile_dispatch=disp if disp != 1 else None,
                              split_k=sk if sk > 1 else None, tail_split=ts or None, tail_chunks=tc or None,
                              bm=bm, bn=bn, bk=64 if tile is not None else None, num_workgroups=grid or None,
                              intra_order=io or None, group_m=gm if io else None, tail_wave=tw if tw > 1 else None,
                              copy_split=cs if cs > 1 else None, tail_taper=tt or None))
        if c not in seen:
            seen.add(c)
            out.append(c)
    return out


def measure(plan: Plan, call: Callable[[Plan, str], None], steps: int, warmup: int) -> float:
    """Steady-state ms per step of `steps` back-to-back overlap calls."""
    for _ in range(warmup):
        call(plan, "overlap")
    plan.check()
    t0 = time.perf_counter()
    for _ in range(steps):
        call(plan, "overlap")
    plan.check()
    return (time.perf_counter() - t0) * 1e3 / steps


def autotune(make_plan: Callable[[Candidate], Plan], call: Callable[[Plan, str], None],
             candidates: Sequence[Candidate], steps: int = 10, warmup: int = 3,
             keep_best: bool = False,
             measure_fn: Optional[Callable[[Plan, Callable[[Plan, str], None], int, int], float]] = None
             ) -> Tuple[TuneResult, Optional[Plan]]:
    """Times every candidate; returns the result and, with keep_best, the best plan
    (the others are destroyed as soon as they are measured).

    make_plan(candidate) builds the plan (and sets its copy delays, if any);
    call(plan, mode) makes one call with the caller's buffers and streams;
    measure_fn(plan, call, steps, warmup) gives the candidate's time in ms (default:
    `measure`, the steady state of back-to-back overlap calls; a caller may time cold
    isolated calls instead, whose end it can see on the device)."""
    measure_fn = measure_fn or measure
    if not candidates:
        raise ValueError("no candidates")
    trials: List[Trial] = []
    best: Optional[Tuple[float, Candidate]] = None
    best_plan: Optional[Plan] = None
    for cand in candidates:
        try:
            plan = make_plan(cand)
        except CsgError as e:
            trials.append(Trial(cand, None, "rejected: %s" % e))
            continue
        try:
            ms = measure_fn(plan, call, steps, warmup)
        except CsgError as e:
            plan.close()
            trials.append(Trial(cand, None, "failed: %s" % e))
            continue
        trials.append(Trial(cand, ms, "ok"))
        if best is None or ms < best[0]:
            best = (ms, cand)
            if keep_best:
                if best_plan is not None:
                    best_plan.close()
                best_plan = plan
                continue
        plan.close()
    if best is None:
        raise RuntimeError("no candidate could run: " + "; ".join(t.status for t in trials))
    return TuneResult(best[1], best[0], trials), best_plan


def uniform_plan_factory(op: str, M: int, N: int, K: int, in_dtype: str, out_dtype: str, world: int, rank: int,
                         shard_rows: int, order: str, default_q: int,
                         perm_for: Optional[Callable[[int], Sequence[int]]] = None,
                         delays_for: Optional[Callable[[int], Sequence[float]]] = None,
                         device: int = 0) -> Callable[[Candidate], Plan]:
    """make_plan for uniform schedules: builds the schedule for the candidate's chunk
    split (default_q when it has none), its permutation (perm_for(q), for the
    permutation order) and its copy delays (delays_for(q))."""
    def make(c: Candidate) -> Plan:
        q = c.chunks_per_shard or default_q
        perm = perm_for(q) if (perm_for is not None and order == "permutation") else None
        sched = Schedule.uniform(world, rank, shard_rows, q, order, perm)
        try:
            plan = Plan(op, M, N, K, in_dtype, out_dtype, sched, cfg=c.cfg_dict(), device=device)
        finally:
            sched.close()
        if delays_for is not None:
            d = delays_for(q)
            if d is not None:
                plan.set_copy_delays(d)
        return plan
    return make
