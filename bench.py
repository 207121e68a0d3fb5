#!/usr/bin/env python3
"""Benchmark: chunk-scheduled GEMM TFLOP/s on one MI355X, with compute/copy overlap.

One step = one call of the whole path on one batch of synthetic input: the
prologue, the SDMA chunk copies whose completion signals are the per-chunk flags,
and the persistent chunk-ordered GEMM kernel, in overlap mode. Steps run back to
back, as in a layer loop where each layer gathers into its own activation: the
all-gather and grouped workloads alternate between two landing buffers
(--landing-buffers), so a step's copies wait only for the kernel two steps back to
have read the rows they overwrite (the library tracks that per buffer), and the same
loop with one landing buffer is reported beside it. The default workload is the
all-gather GEMM of 8 simulated ranks (A 8192 x 4096 bf16 in 8 shards of 4
chunks, ring arrival; B 4096 x 1792; fp32 accumulation, bf16 output).

Prints ONE JSON line. Besides the contract fields it reports, from separate
phases after the timed region, isolated-call times of the overlap, compute-only
and copy-only modes of the same workload and the overlap efficiency
max(t_compute, t_copy) / t_total; the roofline of the GEMM kernel (its durations
in the timed region, from timing events the library records around each launch);
and the CPU oracle timed on a bounded sample.
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
CAL_BYTES = 256 << 20  # bytes read (and written) by the calibration copy


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", type=int, default=2, help="workload id (1..7; 6 = GEMM + all-reduce, 7 = ring attention)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0, help="target length of the CPU baseline sample")
    ap.add_argument("--lanes", type=int, default=0, help="SDMA copy lanes (0 = library default)")
    ap.add_argument("--no-kernel-copies", action="store_true",
                    help="skip the comparison with chunks moved by the kernel's own workgroups")
    ap.add_argument("--landing-buffers", type=int, default=2,
                    help="all-gather and grouped workloads: consecutive steps gather into this many landing "
                         "buffers in turn (as consecutive layers gather into their own activations); 1 = every "
                         "step into the same buffer")
    return ap.parse_args()


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
    cfg = {"copy_engines": args.lanes} if args.lanes else None
    if w.op == "attn":
        e = w.extras
        plan = csg.AttnPlan(e["heads"], e["kv_heads"], e["head_dim"], w.M, sched, cfg=cfg)
    else:
        plan = csg.Plan(w.op, w.M, w.N, w.K, w.dtype, w.out_dtype, sched, group_rows=group_rows, cfg=cfg)
    if d.delays_us is not None:
        plan.set_copy_delays(d.delays_us)
    chunks, _ = sched.get()
    remote_rows = sum(c[1] - c[0] for c in chunks if not c[4])

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
    # landing buffers used in turn by consecutive steps (all-gather and grouped)
    landings = [landing] + [landing.clone() for _ in range(max(args.landing_buffers, 1) - 1)] if landing is not None \
        else [None]
    compute = torch.cuda.Stream(device=dev)
    copy = torch.cuda.Stream(device=dev)
    # plain device-to-device copy of known size, run once before the timed region: the
    # reference that turns the FETCH_SIZE / WRITE_SIZE counters of a profile into bytes
    cal_src = torch.empty(CAL_BYTES // 4, dtype=torch.float32, device=dev).fill_(1.0)
    cal_dst = torch.empty_like(cal_src)
    cal_dst.copy_(cal_src)
    del cal_src, cal_dst
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

    def bracketed(mode, reps, warmup):
        """Isolated calls (the GPU idle before each): per call, the wall time from the
        call to its kernel and every copy having completed (ms)."""
        for _ in range(warmup):
            call(mode)
        plan.check()
        tot = []
        for _ in range(reps):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            call(mode)
            plan.check()
            torch.cuda.synchronize()
            tot.append((time.perf_counter() - t0) * 1e3)
        ker = plan.kernel_times(reps) if mode != "copy_only" else np.array([])
        return np.array(tot), ker

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
    overlap_eff = max(ms_comp, ms_copy) / ms_per_step
    ms_one_landing = None
    if len(landings) > 1:
        # the same overlap loop with every step gathering into one landing buffer: a
        # step's copy of a chunk then waits for the previous step's kernel to have read it
        kept = list(landings)
        landings[:] = kept[:1]
        wall_1, _ = timed_loop("overlap", args.steps, args.warmup)
        landings[:] = kept
        ms_one_landing = wall_1 * 1e3 / args.steps
    # isolated calls: each mode timed alike (the call until its kernel and copies are
    # done, GPU idle before)
    tot, _ = bracketed("overlap", args.steps, args.warmup)
    tot_c, _ = bracketed("compute_only", args.steps, args.warmup)
    tot_x, _ = bracketed("copy_only", args.steps, args.warmup)
    t_total = float(np.median(tot))
    t_comp = float(np.median(tot_c))
    t_copy = float(np.median(tot_x))
    overlap_eff_isolated = max(t_comp, t_copy) / t_total

    peak = MFMA_PEAK_TFLOPS[w.dtype]
    k_overlap = float(np.mean(ker))
    k_comp = float(np.mean(ker_c))
    kernel_name = "ring_attn" if w.op == "attn" else "chunk_gemm"
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
                   "num_workgroups": plan.info.num_workgroups,
                   "tile": [plan.info.bm, plan.info.bn, plan.info.bk],
                   "landing_buffers": len(landings) if landing is not None else None},
        # steady state: ms per step of back-to-back loops in each mode
        "ms_per_step_compute_only": round(ms_comp, 4),
        "ms_per_step_copy_only": round(ms_copy, 4),
        "overlap_eff": round(overlap_eff, 4),
        "ms_per_step_one_landing_buffer": None if ms_one_landing is None else round(ms_one_landing, 4),
        "compute_only_tflops": round(w.flops / (ms_comp * 1e-3) / 1e12, 2),
        "copy_only_GBps": round(moved_bytes / (ms_copy * 1e-3) / 1e9, 2),
        # one isolated call per mode (median)
        "t_total_ms_median": round(t_total, 4),
        "t_compute_only_ms_median": round(t_comp, 4),
        "t_copy_only_ms_median": round(t_copy, 4),
        "overlap_eff_isolated": round(overlap_eff_isolated, 4),
        "roofline": {"bound": "mfma", "achieved": round(w.flops / (k_overlap * 1e-3) / 1e12, 2), "peak": peak,
                     "unit": "TFLOP/s", "frac": round(w.flops / (k_overlap * 1e-3) / 1e12 / peak, 4),
                     "traffic": kernel_traffic(w.name, kernel_name), "kernel": kernel_name,
                     "phase": "overlap (timed region)",
                     "kernel_ms_mean": round(k_overlap, 4)},
        "roofline_compute_only": {"bound": "mfma", "achieved": round(w.flops / (k_comp * 1e-3) / 1e12, 2),
                                  "peak": peak, "unit": "TFLOP/s",
                                  "frac": round(w.flops / (k_comp * 1e-3) / 1e12 / peak, 4),
                                  "kernel_ms_mean": round(k_comp, 4)},
    }
    if not args.no_kernel_copies and w.op not in ("ar", "attn"):  # these copy with the engines only
        rec["kernel_copy_backend"] = kernel_copy_sweep(w, sched, group_rows, d, timed_loop, moved_bytes, args)
    if not args.no_cpu_baseline:
        rec["cpu_baseline"] = cpu_baseline(w, d, chunks, args.cpu_seconds)
    print(json.dumps(rec), flush=True)


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


def kernel_traffic(workload: str, kernel: str = "chunk_gemm"):
    """HBM bytes per launch of the kernel (FETCH_SIZE + WRITE_SIZE, scaled by the
    calibration copy) from the committed counter summary, or None when that summary is
    missing, covers another workload, or was taken from a different kernel source."""
    try:
        with open(KERNEL_TRAFFIC[kernel][0]) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    entry = t.get("workloads", {}).get(workload)
    if not entry or t.get("source_sha256") != kernel_sources_sha256(kernel):
        return None
    return entry.get("bytes_per_launch")


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
            "kind": "oracle", "seconds": round(t, 3),
            "sample": "%d of %d output rows (first rows in chunk row order), all %d columns, K=%d, fp64 plain loops"
                      % (n, w.M, w.N, w.K)}


if __name__ == "__main__":
    main()
