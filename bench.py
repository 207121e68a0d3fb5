#!/usr/bin/env python3
"""Benchmark: chunk-scheduled GEMM TFLOP/s on one MI355X, with compute/copy overlap.

One step = one call of the whole path on one batch of synthetic input: the SDMA chunk
copies whose completion signals are the per-chunk flags, and the persistent
chunk-ordered GEMM kernel, in overlap mode. The default workload is the largest one:
the all-gather GEMM of 8 simulated ranks with fine chunks (A 16384 x 8192 bf16 in 8
shards of 16 chunks of 128 rows, seeded arrival order, per-chunk release delays drawn
from U[0, 20] us; B 8192 x 3584; fp32 accumulation, bf16 output).

The timed region is `--steps` back-to-back overlap calls that all gather into the same
landing buffer, as consecutive calls of one layer do: a call's copy of a chunk waits
until the previous call's kernel has read that chunk's rows.

Prints ONE JSON line. Besides the contract fields it reports, from separate phases
after the timed region:
- isolated calls, cold: before each one a 512 MiB write evicts the inputs from the
  last-level cache and the L2s; each call is timed on the device, from an event on the
  compute stream before the call to an event after csg_plan_join (the end of the
  call's kernel and of every copy it issued); median, p10 and p90 of overlap,
  compute-only and copy-only calls, and the per-call overlap efficiency
  max(t_compute, t_copy) / t_total;
- the steady state of the same back-to-back loop in compute-only and copy-only mode,
  and the overlap loop gathering into two landing buffers in turn (the next call's
  copies then run under this call's kernel);
- the roofline of the GEMM kernel: its durations in the timed region (timing events
  the library records around each launch) against the nominal bf16 MFMA peak and the
  peak the MFMA microbenchmark measures on the device;
- the CPU oracle timed on a bounded sample.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

MFMA_PEAK_TFLOPS = {"bf16": 2500.0, "f32": 157.3}  # MI355X dense MFMA peaks
HBM_PEAK_GBS = 8000.0
CAL_BYTES = 256 << 20    # bytes read (and written) by the calibration copy
# The operator implementation per workload, as the autotuner selected it with cold
# isolated calls as the objective (`bench.py --config N --tune --objective isolated`),
# among the copy-engine candidates (the copy engines stand in for the links of a real
# collective; the kernel's own copies move chunks inside HBM faster than links would):
# plan configuration fields. GEMM + reduce-scatter and the grouped GEMM keep 256 x 256
# tiles where the tuner's best used 128 x 256 tiles within 1-3 % per cold call: those
# ran the back-to-back loop 4-20 % slower. --default-plan measures the library's
# defaults instead.
TUNED_PLAN_CFG = {
    2: {"bm": 128, "bn": 256, "bk": 64, "tile_dispatch": 2, "tail_split": 2, "tail_chunks": 4},
    3: {"intra_order": 1, "group_m": 4, "tile_dispatch": 2},
    4: {"bm": 128, "bn": 256, "bk": 64, "tile_dispatch": 2, "tail_split": 4, "tail_chunks": 12, "tail_taper": 1,
        "copy_split": 2},
    5: {"intra_order": 1, "group_m": 4, "tile_dispatch": 2, "tail_split": 2, "tail_chunks": 4, "copy_split": 2},
}
FLUSH_BYTES = 512 << 20  # written before each isolated call: more than the last-level cache and every L2


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", type=int, default=4,
                    help="workload id (1..7; 4 = the headline, 6 = GEMM + all-reduce, 7 = ring attention)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0, help="target length of the CPU baseline sample")
    ap.add_argument("--lanes", type=int, default=0, help="SDMA copy lanes (0 = library default)")
    ap.add_argument("--no-kernel-copies", action="store_true",
                    help="skip the comparison with chunks moved by the kernel's own workgroups")
    ap.add_argument("--isolated-reps", type=int, default=0,
                    help="cold isolated calls per mode (0 = as many as --steps)")
    ap.add_argument("--plan-cfg", type=str, default="",
                    help="JSON object of plan configuration fields for the measured plan (e.g. tile order)")
    ap.add_argument("--default-plan", action="store_true",
                    help="measure the library's default plan instead of the workload's tuned plan configuration")
    ap.add_argument("--objective", choices=("steady", "isolated"), default="steady",
                    help="--tune: time each candidate as back-to-back overlap calls (steady) or as cold "
                         "isolated overlap calls (isolated, the median device time per call)")
    ap.add_argument("--tune", action="store_true",
                    help="instead of the bench line, run the autotuner on the workload (chunk split, intra-chunk "
                         "order, dispatch, copy realization) and print its table as one JSON line")
    ap.add_argument("--timeline", action="store_true",
                    help="instead of the bench line, trace the work units of cold isolated overlap calls "
                         "(when each unit was taken, started after its chunk waits, and finished) and print "
                         "their distribution as one JSON line")
    return ap.parse_args()


def pct(a, q):
    return round(float(np.percentile(np.asarray(a), q)), 4)


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py: this build measures one GPU only; --gpus %d is not supported (run with --gpus 1)"
              % args.gpus, file=sys.stderr)
        sys.exit(2)
    import torch

    import paper_2601_20595_amd as csg
    import seeded_inputs as si

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    if args.tune:
        tune_workload(args)
        return
    if args.timeline and si.WORKLOADS[args.config].op == "attn":
        print("bench.py --timeline: the unit trace covers the GEMM operations", file=sys.stderr)
        sys.exit(2)
    dev = "cuda:0"
    arch = csg.csg_device_check(0)
    w = si.WORKLOADS[args.config]
    d = si.draw(w)

    def to_dev(arr):
        if arr.dtype == np.uint16:
            return torch.from_numpy(np.ascontiguousarray(arr).view(np.int16)).to(dev)
        return torch.from_numpy(np.ascontiguousarray(arr)).to(dev)

    if w.op == "grouped":
        sched = csg.Schedule.grouped(w.world, w.rank, d.counts)
        group_rows = [int(x) for x in d.counts.sum(axis=0)]
    else:
        sched = csg.Schedule.uniform(w.world, w.rank, w.shard_rows, w.chunks_per_shard, w.order, d.perm)
        group_rows = None
    tuned = not args.default_plan and args.config in TUNED_PLAN_CFG
    cfg = dict(TUNED_PLAN_CFG[args.config]) if tuned else {}
    if args.lanes:
        cfg["copy_engines"] = args.lanes
    if args.plan_cfg:
        cfg.update(json.loads(args.plan_cfg))
    if args.timeline:
        cfg["trace"] = 1
    cfg = cfg or None
    if w.op == "attn":
        e = w.extras
        plan = csg.AttnPlan(e["heads"], e["kv_heads"], e["head_dim"], w.M, sched, cfg=cfg)
    else:
        plan = csg.Plan(w.op, w.M, w.N, w.K, w.dtype, w.out_dtype, sched, group_rows=group_rows, cfg=cfg)
    if d.delays_us is not None:
        plan.set_copy_delays(d.delays_us)
    chunks, _ = sched.get()
    remote_rows = sum(c[1] - c[0] for c in chunks if not c[4])

    # the MFMA microbenchmark first, on an idle device: a short run and one about as long
    # as the workload's kernel (the clock falls as a longer run heats the device)
    peak_short = csg.csg_measure_mfma_peak(0, 800)
    peak_long = csg.csg_measure_mfma_peak(0, 8000)

    a_full = to_dev(d.A.device_array)
    b = to_dev(d.B.device_array)
    out_t = torch.int16 if w.out_dtype == "bf16" else torch.float32
    c = torch.empty((w.M, w.N), dtype=out_t, device=dev)
    in_bytes = 2 if w.dtype == "bf16" else 4
    out_bytes = 2 if w.out_dtype == "bf16" else 4
    p_stage = p_land = reduced = None
    if w.op == "attn":
        # the other ranks' keys and values arrive; a_full = queries
        e = w.extras
        landing = None
        k_stage, v_stage = to_dev(d.B.device_array), to_dev(d.V.device_array)
        k_land, v_land = k_stage.clone(), v_stage.clone()
        c = torch.empty((w.M, e["heads"], e["head_dim"]), dtype=torch.int16, device=dev)
        lse = torch.empty((e["heads"], w.M), dtype=torch.float32, device=dev)
        outgoing = None
        moved_bytes = 2 * remote_rows * e["kv_heads"] * e["head_dim"] * 2
    elif w.op == "ar":
        # reduce-scatter sends and all-gather arrivals of the non-local chunks, the other
        # ranks' partials of the own shard, and the sends of the reduced own chunks
        landing = None
        outgoing = torch.zeros((w.M, w.N), dtype=out_t, device=dev)
        p_stage = to_dev(d.partials.device_array)
        p_land = p_stage.clone()
        reduced = to_dev(d.reduced.device_array)
        own_rows = w.M - remote_rows
        moved_bytes = (2 * remote_rows + (w.world - 1) * own_rows + own_rows) * w.N * out_bytes
    elif w.op == "rs":
        landing = None
        outgoing = torch.zeros((w.M, w.N), dtype=out_t, device=dev)
        moved_bytes = remote_rows * w.N * out_bytes
    else:
        landing = a_full.clone()
        outgoing = None
        moved_bytes = remote_rows * w.K * in_bytes
    landings = [landing]   # the timed region: every step gathers into the same buffer
    compute = torch.cuda.Stream(device=dev)
    copy = torch.cuda.Stream(device=dev)
    # plain device-to-device copy of known size, run once before the timed region: the
    # reference that turns the FETCH_SIZE / WRITE_SIZE counters of a profile into bytes
    cal_src = torch.empty(CAL_BYTES // 4, dtype=torch.float32, device=dev).fill_(1.0)
    cal_dst = torch.empty_like(cal_src)
    cal_dst.copy_(cal_src)
    del cal_src, cal_dst
    flush_buf = torch.empty(FLUSH_BYTES // 4, dtype=torch.int32, device=dev)
    torch.cuda.synchronize()

    def call(mode, p=None, step=0):
        p = p or plan
        landing = landings[step % len(landings)]
        if w.op == "attn":
            p.ring_attn(a_full, k_land, v_land, k_stage, v_stage, c, lse, mode, compute, copy)
        elif w.op == "ar":
            p.gemm_ar(a_full, b, c, outgoing, p_stage, p_land, reduced, mode, compute, copy)
        elif w.op == "rs":
            p.gemm_rs(a_full, b, c, outgoing, mode, compute, copy)
        elif w.op == "grouped":
            p.grouped_gemm(landing, a_full, b, c, mode, compute, copy)
        else:
            p.ag_gemm(landing, a_full, b, c, mode, compute, copy)

    def timed_loop(mode, steps, warmup, p=None):
        """Back-to-back calls, as a training or serving loop makes them: no event or
        stream dependency between steps beyond what the library itself orders, so the
        copies of one step may start while the previous step's kernel still runs.
        Returns wall seconds for `steps` calls and the kernel durations (ms) the
        library timed on the compute stream."""
        p = p or plan
        for i in range(warmup):
            call(mode, p, i)
        p.check()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(steps):
            call(mode, p, i)
        p.check()                 # every copy the steps issued has completed
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        return wall, p.kernel_times(steps)

    def isolated(mode, reps, warmup, p=None):
        """Cold isolated calls: the caches flushed and the device idle before each one;
        per call, the device time (ms) from an event queued on the compute stream just
        before the call to one queued after csg_plan_join (the call's kernel and every
        copy it issued have completed)."""
        p = p or plan
        for _ in range(warmup):
            call(mode, p)
        p.check()
        ev0 = torch.cuda.Event(enable_timing=True)
        ev1 = torch.cuda.Event(enable_timing=True)
        tot = []
        for i in range(reps):
            with torch.cuda.stream(compute):
                flush_buf.fill_(i)
            torch.cuda.synchronize()
            ev0.record(compute)
            call(mode, p)
            p.join(compute)
            ev1.record(compute)
            ev1.synchronize()
            p.check()
            tot.append(ev0.elapsed_time(ev1))
        return np.array(tot)

    if args.timeline:
        print(json.dumps(timeline(w, plan, call, isolated, args, cfg, tuned)), flush=True)
        return

    # ---- the timed region: overlap steps ------------------------------------------
    wall, ker = timed_loop("overlap", args.steps, args.warmup)
    ms_per_step = wall * 1e3 / args.steps
    value = w.flops * args.steps / wall / 1e12
    # ---- reference phases (not part of the timed region) ---------------------------
    # the same back-to-back loop without copies, and with copies only
    wall_c, ker_c = timed_loop("compute_only", args.steps, args.warmup)
    wall_x, _ = timed_loop("copy_only", args.steps, args.warmup)
    ms_comp = wall_c * 1e3 / args.steps
    ms_copy = wall_x * 1e3 / args.steps
    ms_two_landing = None
    if landing is not None:
        # the overlap loop gathering into two landing buffers in turn: the next step's
        # copies may run under this step's kernel (a pipeline a dependent layer chain
        # cannot build)
        landings.append(landing.clone())
        wall_2, _ = timed_loop("overlap", args.steps, args.warmup)
        del landings[1:]
        ms_two_landing = wall_2 * 1e3 / args.steps
    # cold isolated calls, each mode alike
    reps = args.isolated_reps or max(args.steps, 10)
    tot = isolated("overlap", reps, args.warmup)
    tot_c = isolated("compute_only", reps, args.warmup)
    tot_x = isolated("copy_only", reps, args.warmup)
    t_total = float(np.median(tot))
    t_comp = float(np.median(tot_c))
    t_copy = float(np.median(tot_x))
    overlap_eff = max(t_comp, t_copy) / t_total
    default_iso = None
    if tuned:
        # the same cold isolated calls on the library's default plan, for comparison
        if w.op == "attn":
            p0 = csg.AttnPlan(e["heads"], e["kv_heads"], e["head_dim"], w.M, sched)
        else:
            p0 = csg.Plan(w.op, w.M, w.N, w.K, w.dtype, w.out_dtype, sched, group_rows=group_rows)
        if d.delays_us is not None:
            p0.set_copy_delays(d.delays_us)
        d_tot = float(np.median(isolated("overlap", reps, args.warmup, p0)))
        d_comp = float(np.median(isolated("compute_only", reps, args.warmup, p0)))
        d_copy = float(np.median(isolated("copy_only", reps, args.warmup, p0)))
        _, d_ker_c = timed_loop("compute_only", args.steps, args.warmup, p0)
        p0.close()
        d_kc = float(np.mean(d_ker_c))
        default_iso = {"plan_cfg": {}, "t_total_ms": round(d_tot, 4), "t_compute_only_ms": round(d_comp, 4),
                       "t_copy_only_ms": round(d_copy, 4), "overlap_eff": round(max(d_comp, d_copy) / d_tot, 4),
                       "e2e_tflops_isolated": round(w.flops / (d_tot * 1e-3) / 1e12, 2),
                       "compute_only_kernel_ms_mean": round(d_kc, 4),
                       "roofline_compute_only_frac": round(w.flops / (d_kc * 1e-3) / 1e12 / MFMA_PEAK_TFLOPS[w.dtype], 4)}

    peak = MFMA_PEAK_TFLOPS[w.dtype]
    k_overlap = float(np.mean(ker))
    k_comp = float(np.mean(ker_c))
    kernel_name = "ring_attn" if w.op == "attn" else "chunk_gemm"
    tf_overlap = w.flops / (k_overlap * 1e-3) / 1e12
    tf_comp = w.flops / (k_comp * 1e-3) / 1e12
    measured = {"short": {"tflops": round(peak_short[0], 1), "ms": round(peak_short[1], 4),
                          "ghz": round(peak_short[2], 3)},
                "sustained": {"tflops": round(peak_long[0], 1), "ms": round(peak_long[1], 4),
                              "ghz": round(peak_long[2], 3)}}
    mpeak = peak_long[0] if w.dtype == "bf16" else None
    rec = {
        "metric": "chunk-scheduled GEMM TFLOP/s @1 GPU; overlap eff = max(comp,copy)/total",
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic (seeded %s values)" % w.dist,
        "config": {"workload": w.name, "op": w.op, "M": w.M, "N": w.N, "K": w.K, "world": w.world,
                   "chunks": len(chunks), "moved_bytes": moved_bytes, "arch": arch,
                   "copy_delays": "cumulative release times, U[0,20] us each" if d.delays_us is not None else None,
                   "num_workgroups": plan.info.num_workgroups,
                   "tile": [plan.info.bm, plan.info.bn, plan.info.bk],
                   "plan_cfg": cfg or {},
                   "plan_cfg_source": ("autotuner, cold isolated calls (bench.py --tune --objective isolated)"
                                       if tuned else "library defaults" if not cfg else "command line"),
                   "landing_buffers": 1 if landing is not None else None},
        # cold isolated calls (device events; caches flushed before each)
        "overlap_eff": round(overlap_eff, 4),
        "t_total_ms": {"median": round(t_total, 4), "p10": pct(tot, 10), "p90": pct(tot, 90)},
        "t_compute_only_ms": {"median": round(t_comp, 4), "p10": pct(tot_c, 10), "p90": pct(tot_c, 90)},
        "t_copy_only_ms": {"median": round(t_copy, 4), "p10": pct(tot_x, 10), "p90": pct(tot_x, 90)},
        "isolated": {"reps": reps, "cache_flush_bytes": FLUSH_BYTES,
                     "timing": "device events: compute stream before the call .. after csg_plan_join"},
        "e2e_tflops_isolated": round(w.flops / (t_total * 1e-3) / 1e12, 2),
        "copy_GBps_isolated": round(moved_bytes / (t_copy * 1e-3) / 1e9, 2),
        # steady state: ms per step of back-to-back loops in each mode
        "ms_per_step_compute_only": round(ms_comp, 4),
        "ms_per_step_copy_only": round(ms_copy, 4),
        "overlap_eff_steady": round(max(ms_comp, ms_copy) / ms_per_step, 4),
        "ms_per_step_two_landing_buffers": None if ms_two_landing is None else round(ms_two_landing, 4),
        "overlap_eff_steady_two_landing_buffers":
            None if ms_two_landing is None else round(max(ms_comp, ms_copy) / ms_two_landing, 4),
        "compute_only_tflops": round(w.flops / (ms_comp * 1e-3) / 1e12, 2),
        "roofline": {"bound": "mfma", "achieved": round(tf_overlap, 2), "peak": peak,
                     "unit": "TFLOP/s", "frac": round(tf_overlap / peak, 4),
                     "traffic": kernel_traffic(w.name, kernel_name, cfg), "kernel": kernel_name,
                     "phase": "overlap (timed region)",
                     "kernel_ms_mean": round(k_overlap, 4),
                     "frac_of_measured_peak": round(tf_overlap / mpeak, 4) if mpeak else None},
        "roofline_compute_only": {"bound": "mfma", "achieved": round(tf_comp, 2),
                                  "peak": peak, "unit": "TFLOP/s",
                                  "frac": round(tf_comp / peak, 4),
                                  "kernel_ms_mean": round(k_comp, 4),
                                  "frac_of_measured_peak": round(tf_comp / mpeak, 4) if mpeak else None},
        "mfma_peak_measured": measured,
    }
    if default_iso is not None:
        rec["default_plan_isolated"] = default_iso
    if not args.no_kernel_copies and w.op not in ("ar", "attn"):  # these copy with the engines only
        rec["kernel_copy_backend"] = kernel_copy_sweep(w, sched, group_rows, d, timed_loop, moved_bytes, args)
    if not args.no_cpu_baseline:
        rec["cpu_baseline"] = cpu_baseline(w, d, chunks, args.cpu_seconds)
        if w.op != "attn":
            rec["cpu_baseline"]["torch_cpu_fp32"] = torch_cpu_reference(w, d, rec["cpu_baseline"])
    if w.op in ("ag", "rs", "ar"):
        rec["hipblaslt_reference"] = hipblaslt_reference(w, a_full, b, compute)
    print(json.dumps(rec), flush=True)


def timeline(w, plan, call, isolated, args, cfg, tuned):
    """The work-unit trace of cold isolated overlap calls: per call, the device time
    around the call (ms), and, in microseconds from the first unit's take (the kernel's
    start), when the units were taken, started (after waiting for their chunks) and
    finished, as percentiles over the call's units; wait = start - take; tail = the
    kernel's end - the last start. The per-call lists hold one entry per call."""
    reps = args.isolated_reps or 10
    tot = isolated("overlap", reps, 3)            # warm-up calls included; the trace holds the last call
    calls = []
    qs = (0, 10, 25, 50, 75, 90, 100)
    for i in range(reps):
        t = isolated("overlap", 1, 0)
        tr = plan.trace()
        t0 = int(tr["t_take"].min())
        take = (tr["t_take"].astype(np.int64) - t0) / 100.0
        start = (tr["t_start"].astype(np.int64) - t0) / 100.0
        end = (tr["t_end"].astype(np.int64) - t0) / 100.0
        wait = start - take
        calls.append({
            "t_total_ms": round(float(t[0]), 4), "units": int(len(tr)), "kernel_us": round(float(end.max()), 1),
            "start_us_pctl": [round(float(np.percentile(start, q)), 1) for q in qs],
            "end_us_pctl": [round(float(np.percentile(end, q)), 1) for q in qs],
            "unit_us_p10_p50_p90": [round(float(np.percentile(end - start, q)), 1) for q in (10, 50, 90)],
            "wait_us_mean_p90_max": [round(float(wait.mean()), 1), round(float(np.percentile(wait, 90)), 1),
                                     round(float(wait.max()), 1)],
            "tail_us": round(float(end.max() - start.max()), 1),
        })
    return {"timeline": {"workload": w.name, "plan_cfg": cfg, "plan": "tuned" if tuned else "default",
                         "calls": len(calls), "percentiles": list(qs),
                         "t_total_ms_median_of_isolated_calls": round(float(np.median(tot)), 4),
                         "per_call": calls}}


def kernel_copy_sweep(w, sched, group_rows, d, timed_loop, moved_bytes, args, sweep=(32, 64, 128)):
    """The same workload with the chunks moved by the GEMM kernel's own workgroups
    (CSG_COPY_KERNEL: copy workgroups for AG / grouped, sends from the tile epilogue
    for GEMM-RS), per number of copy workgroups: steady-state ms per step in each
    mode, as for the copy-engine path above. Outside the timed region; a comparison
    of two realizations of the same chunk schedule, not the headline."""
    import paper_2601_20595_amd as csg
    out = {"note": "chunks moved by the kernel's workgroups instead of SDMA; steady-state ms per step",
           "copy_workgroups": {}}
    for cw in sweep:
        p = csg.Plan(w.op, w.M, w.N, w.K, w.dtype, w.out_dtype, sched, group_rows=group_rows,
                     cfg={"copy_backend": "kernel", "copy_workgroups": cw})
        if d.delays_us is not None:
            p.set_copy_delays(d.delays_us)
        ms = {}
        for mode in ("overlap", "compute_only", "copy_only"):
            wall, _ = timed_loop(mode, args.steps, args.warmup, p)
            ms[mode] = wall * 1e3 / args.steps
        p.close()
        out["copy_workgroups"][str(cw)] = {
            "ms_per_step": round(ms["overlap"], 4), "ms_per_step_compute_only": round(ms["compute_only"], 4),
            "ms_per_step_copy_only": round(ms["copy_only"], 4),
            "overlap_eff": round(max(ms["compute_only"], ms["copy_only"]) / ms["overlap"], 4),
            "tflops": round(w.flops / (ms["overlap"] * 1e-3) / 1e12, 2),
            "copy_only_GBps": round(moved_bytes / (ms["copy_only"] * 1e-3) / 1e9, 2)}
    return out


def tune_workload(args):
    """The enumerate-and-measure autotuner on one workload: chunk splits (uniform
    schedules), intra-chunk tile order, tile dispatch and copy realization, each
    candidate timed as back-to-back overlap calls. Prints one JSON line with every
    candidate's ms per step, the best one, and whether the best plan's product equals
    the default plan's bit for bit."""
    import torch
    import paper_2601_20595_amd as csg
    import seeded_inputs as si
    from paper_2601_20595_amd import tune

    dev = "cuda:0"
    w = si.WORKLOADS[args.config]
    if w.op not in ("ag", "rs", "grouped"):
        print("bench.py --tune: the tuner covers the all-gather, reduce-scatter and grouped GEMMs", file=sys.stderr)
        sys.exit(2)
    d = si.draw(w)

    def to_dev(arr):
        if arr.dtype == np.uint16:
            return torch.from_numpy(np.ascontiguousarray(arr).view(np.int16)).to(dev)
        return torch.from_numpy(np.ascontiguousarray(arr)).to(dev)

    A, B = to_dev(d.A.device_array), to_dev(d.B.device_array)
    out_t = torch.int16 if w.out_dtype == "bf16" else torch.float32
    C = torch.empty((w.M, w.N), dtype=out_t, device=dev)
    comp, cp = torch.cuda.Stream(device=dev), torch.cuda.Stream(device=dev)
    if w.op == "rs":
        outgoing = torch.zeros((w.M, w.N), dtype=out_t, device=dev)
        call = lambda p, m: p.gemm_rs(A, B, C, outgoing, m, comp, cp)
    else:
        landing = A.clone()
        if w.op == "grouped":
            call = lambda p, m: p.grouped_gemm(landing, A, B, C, m, comp, cp)
        else:
            call = lambda p, m: p.ag_gemm(landing, A, B, C, m, comp, cp)
    if w.op == "grouped":
        group_rows = [int(x) for x in d.counts.sum(axis=0)]

        def make(c):
            s = csg.Schedule.grouped(w.world, w.rank, d.counts)
            try:
                return csg.Plan(w.op, w.M, w.N, w.K, w.dtype, w.out_dtype, s, group_rows=group_rows,
                                cfg=c.cfg_dict())
            finally:
                s.close()
        splits = (None,)
    else:
        make = tune.uniform_plan_factory(w.op, w.M, w.N, w.K, w.dtype, w.out_dtype, w.world, w.rank,
                                         w.shard_rows, w.order, w.chunks_per_shard,
                                         perm_for=lambda q: d.perm, delays_for=lambda q: d.delays_us)
        # the workload's own split first: the first candidate is the library's default plan
        splits = (w.chunks_per_shard,) + tuple(q for q in (1, 2, 4, 8) if q != w.chunks_per_shard and
                                               w.shard_rows % q == 0 and (w.shard_rows // q) % 128 == 0)
        if d.delays_us is not None:
            splits = (None,)  # the release delays are drawn per chunk of the workload's own split
    measure_fn = None
    if args.objective == "isolated":
        # cold isolated calls: a 512 MiB write evicts the inputs from every cache, then
        # the device time from an event before the call to one after csg_plan_join
        flush = torch.empty(FLUSH_BYTES // 4, dtype=torch.int32, device=dev)
        ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

        def measure_fn(plan, call_, steps, warmup):
            for _ in range(warmup):
                call_(plan, "overlap")
            plan.check()
            ts = []
            for i in range(steps):
                with torch.cuda.stream(comp):
                    flush.fill_(i)
                torch.cuda.synchronize()
                ev0.record(comp)
                call_(plan, "overlap")
                plan.join(comp)
                ev1.record(comp)
                ev1.synchronize()
                plan.check()
                ts.append(ev0.elapsed_time(ev1))
            return float(np.median(ts))

        # the chunk split stays the workload's; the tile shape, the tail splits (even or
        # tapered) and the pieces of a chunk copy join the space (they decide how much
        # work is left when the last chunk lands)
        cands = tune.search_space(w.op, chunk_splits=splits[:1], split_k=(1,),
                                  tail=((0, 0), (2, 4), (2, 8), (2, 16), (4, 12), (6, 12)), copy_workgroups=(64,),
                                  tiles=(None, (128, 256)), intra=((0, 0), (1, 4)), copy_split=(0, 2),
                                  tail_taper=(0, 1))
    else:
        cands = tune.search_space(w.op, chunk_splits=splits, split_k=(1,), tail=((0, 0),), copy_workgroups=(64,),
                                  intra=((0, 0), (1, 1), (1, 2), (1, 4)), copy_split=(0, 2))
    res, best = tune.autotune(make, call, cands, steps=args.steps, warmup=args.warmup, keep_best=True,
                              measure_fn=measure_fn)
    call(best, "overlap")
    best.check()
    torch.cuda.synchronize()
    got = C.clone()
    p0 = make(cands[0])
    call(p0, "overlap")
    p0.check()
    torch.cuda.synchronize()
    same = bool(torch.equal(got, C))
    p0.close()
    best.close()
    ran = [t for t in res.trials if t.ms_per_step]
    print(json.dumps({
        "tune": {"workload": w.name, "candidates": len(cands), "ran": len(ran), "steps": args.steps,
                 "warmup": args.warmup,
                 "objective": ("median ms of cold isolated overlap calls" if args.objective == "isolated"
                               else "ms per step of back-to-back overlap calls"),
                 "default": cands[0].label(), "default_ms": next((round(t.ms_per_step, 4) for t in res.trials
                                                                   if t.candidate == cands[0] and t.ms_per_step), None),
                 "best": res.best.label(), "best_ms": round(res.best_ms, 4),
                 "best_tflops": round(w.flops / (res.best_ms * 1e-3) / 1e12, 2),
                 "worst_ms": round(max(t.ms_per_step for t in ran), 4),
                 "best_equals_default_product": same,
                 "table": [[t.candidate.label(), round(t.ms_per_step, 4) if t.ms_per_step else t.status]
                           for t in res.trials]}}), flush=True)


# Per measured kernel: its committed HBM-traffic summary and the sources it was taken from.
KERNEL_TRAFFIC = {
    "chunk_gemm": (os.path.join(ROOT, "profiles", "chunk_gemm_traffic.json"),
                   ("paper_2601_20595_amd/csrc/chunk_gemm.hip", "paper_2601_20595_amd/csrc/kernels.hpp")),
    "ring_attn": (os.path.join(ROOT, "profiles", "ring_attn_traffic.json"),
                  ("paper_2601_20595_amd/csrc/chunk_attn.hip", "paper_2601_20595_amd/csrc/attn.hpp")),
}


def kernel_sources_sha256(kernel: str = "chunk_gemm") -> str:
    import hashlib
    h = hashlib.sha256()
    for rel in KERNEL_TRAFFIC[kernel][1]:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def kernel_traffic(workload: str, kernel: str = "chunk_gemm", plan_cfg=None):
    """HBM bytes per launch of the kernel (FETCH_SIZE + WRITE_SIZE, scaled by the
    calibration copy) from the committed counter summary, or None when that summary is
    missing, covers another workload or plan configuration, or was taken from a
    different kernel source."""
    try:
        with open(KERNEL_TRAFFIC[kernel][0]) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    entry = t.get("workloads", {}).get(workload)
    if not entry or t.get("source_sha256") != kernel_sources_sha256(kernel):
        return None
    if entry.get("plan_cfg", {}) != (plan_cfg or {}):
        return None
    return entry.get("bytes_per_launch")


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def hipblaslt_reference(w, a, b, stream, reps=20):
    """Context, not part of any figure above: the same product as one library GEMM
    (torch.matmul, which runs hipBLASLt), A (M x K) times B^T with B^T made contiguous,
    bf16 in and out, timed warm on the device (median of `reps` launches)."""
    import torch
    bt = b.view(torch.bfloat16).t().contiguous()
    x = a.view(torch.bfloat16)
    with torch.cuda.stream(stream):
        for _ in range(3):
            y = torch.matmul(x, bt)
        ts = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            y = torch.matmul(x, bt)
            e1.record(stream)
            ts.append((e0, e1))
    torch.cuda.synchronize()
    ms = float(np.median([e0.elapsed_time(e1) for e0, e1 in ts]))
    del y, bt
    return {"ms": round(ms, 4), "tflops": round(w.flops / (ms * 1e-3) / 1e12, 2),
            "what": "torch.matmul (hipBLASLt), one GEMM of the whole M x N x K, warm, no communication"}


def torch_cpu_reference(w, d, base):
    """Context beside the oracle: torch's fp32 CPU matmul (its BLAS) over as many
    output rows as the oracle's sample, all columns, on the same cores."""
    import torch
    rows = int(base["sample"].split(" of ")[0])
    A = torch.from_numpy(np.ascontiguousarray(d.A.values[:rows], dtype=np.float32))
    B = d.B.values if w.op != "grouped" else d.B.values[0]
    Bt = torch.from_numpy(np.ascontiguousarray(np.asarray(B, dtype=np.float32).T))
    torch.matmul(A[:64], Bt)
    t0 = time.perf_counter()
    torch.matmul(A, Bt)
    t = time.perf_counter() - t0
    return {"value": round(2.0 * rows * w.N * w.K / t / 1e12, 4), "unit": "TFLOP/s", "threads": torch.get_num_threads(),
            "seconds": round(t, 3), "what": "torch.matmul fp32 on the CPU, as many output rows as the oracle's sample"}


def cpu_baseline(w, d, chunks, target_s):
    """The oracle as it stands, timed on a bounded sample of the same workload: whole
    output rows of the chunks in arrival order, grown until about target_s seconds."""
    import oracle

    rows_all = []
    for ch in chunks:
        rows_all.extend(range(ch[0], ch[1]))
    B = d.B.device_array
    A = d.A.device_array

    if w.op == "attn":
        # queries of the first rows, all heads, against every key (fp64 plain attention)
        Q, K, V = d.A.values, d.B.values, d.V.values
        e = w.extras
        n = 8
        t0 = time.perf_counter()
        oracle.attention(Q[:n], K, V)
        t = time.perf_counter() - t0
        n = int(min(w.M, max(n, n * target_s / max(t, 1e-6))))
        t0 = time.perf_counter()
        oracle.attention(Q[:n], K, V)
        t = time.perf_counter() - t0
        flops = 4.0 * n * K.shape[0] * e["head_dim"] * e["heads"]
        try:  # numpy's products run on its BLAS thread pool
            from threadpoolctl import threadpool_info
            cores = max(int(i.get("num_threads", 1)) for i in threadpool_info() if i.get("user_api") == "blas")
        except Exception:
            cores = 1
        return {"value": round(flops / t / 1e12, 6), "unit": "TFLOP/s", "cores": cores,
                "affinity_cores": len(os.sched_getaffinity(0)), "cpu_model": cpu_model(),
                "kind": "oracle", "seconds": round(t, 3),
                "sample": "%d of %d query rows, all %d heads, all %d keys, fp64 numpy attention"
                          % (n, w.M, e["heads"], K.shape[0])}

    def run(rows):
        t0 = time.perf_counter()
        if w.op == "grouped":
            groups = {}
            for ch in chunks:
                for r in range(ch[0], ch[1]):
                    groups[r] = ch[3]
            by_e = {}
            for r in rows:
                by_e.setdefault(groups[r], []).append(r)
            for e, rs in by_e.items():
                oracle.gemm_rows(A, B[e], rs)
        else:
            oracle.gemm_rows(A, B, rows)
        return time.perf_counter() - t0

    n = 32
    t = run(rows_all[:n])
    n = int(min(len(rows_all), max(n, n * target_s / max(t, 1e-6))))
    t = run(rows_all[:n])
    flops = 2.0 * n * w.N * w.K
    return {"value": round(flops / t / 1e12, 6), "unit": "TFLOP/s", "cores": oracle.num_threads(),
            "affinity_cores": len(os.sched_getaffinity(0)), "cpu_model": cpu_model(),
            "kind": "oracle", "seconds": round(t, 3),
            "sample": "%d of %d output rows (first rows in chunk row order), all %d columns, K=%d, fp64 plain loops"
                      % (n, w.M, w.N, w.K)}


if __name__ == "__main__":
    main()
