"""Benchmark of the recomputation DP on one MI355X.

One step is one pass of the whole path over one synthetic graph: build the
lower-set family (rc_build_family), fill the DP table and select t*
(rc_solve), trace the schedule back and re-evaluate it (rc_reconstruct).
The graph itself is handed over (rc_graph_create) before the timed
region, so the inputs are resident in HBM when timing starts.

Prints one JSON line.  `value` is DP relaxations per second of wall time
per step; `roofline` rates the wavefront fill kernel against the packed
16-bit VALU peak of MI355X (the table holds 16-bit cells and the kernel
relaxes two cells per lane and instruction), with the kernel time taken
from HIP events that the library records around that one launch on the
fill's stream; `cpu_baseline` times the CPU oracle on the same graph on
this host.  `--copy-calibration BYTES` instead runs one device-to-device
copy of BYTES bytes (the reference kernel that scales rocprofv3's
FETCH_SIZE / WRITE_SIZE counters to bytes) and exits.
"""

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

# MI355X: 256 CUs, 4 SIMDs of 16 lanes each per CU (64 lane-ops per clock),
# 2.4 GHz peak engine clock.  Packed 16-bit integer VALU instructions do two
# operations per lane.
VALU_INT32_PEAK_TOPS = 256 * 64 * 2.4e9 / 1e12
VALU_U16_PEAK_TOPS = 2 * VALU_INT32_PEAK_TOPS
OPS_PER_RELAXATION = 3          # compare with tau, add dm, min into the target
# The sources that shape each wavefront fill kernel and its traffic: the
# kernel, its record preparation, the shared helpers and constants.
_CSRC = "paper_1905_11722_amd/csrc/"
FILL_SOURCES = {
    "k_fill_blocked": [_CSRC + "blocked.hip", _CSRC + "blocks.hip", _CSRC + "wavefront.h",
                       _CSRC + "rc_internal.h"],
    "k_fill_wide": [_CSRC + "wide.hip", _CSRC + "blocks.hip", _CSRC + "wavefront.h",
                    _CSRC + "rc_internal.h"],
    "k_fill_ghost": [_CSRC + "ghost.hip", _CSRC + "blocks.hip", _CSRC + "wavefront.h",
                     _CSRC + "rc_internal.h", _CSRC + "ghost_cut.h"],
    "k_fill_level_vec": [_CSRC + "fill.hip", _CSRC + "wavefront.h", _CSRC + "rc_internal.h"],
    "k_fill_level": [_CSRC + "fill.hip", _CSRC + "rc_internal.h"],
}


def fill_source_hash(kernel):
    h = hashlib.sha256()
    for rel in FILL_SOURCES[kernel]:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def read_traffic(kernel, workload):
    """HBM traffic of the fill kernel from committed rocprofv3 PMC runs, if
    they were taken on the current source of that kernel; else None."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload}_traffic.txt")
    if not os.path.exists(path):
        return None
    rec = {}
    with open(path) as f:
        for line in f:
            if "=" in line and not line.startswith((" ", "#", "`")):
                k, v = line.split("=", 1)
                rec[k.strip()] = v.strip()
    if rec.get("fill_source_sha256_16") != fill_source_hash(kernel):
        return None
    try:
        return int(rec["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def run_step(rcdp, g, case):
    fam = g.build_family(case.mode)
    sol = fam.solve(case.B, case.objective)
    sched = sol.reconstruct() if sol.feasible else None
    fill_ms = sol.fill_ms()
    kernel_ms = sol.fill_kernel_ms()
    kernel = sol.fill_kernel()
    info = fam.info
    t_star = sol.t_star
    m_star = sol.m_star
    sol.free()
    fam.free()
    return info, fill_ms, kernel_ms, (t_star, m_star), sched, kernel


def time_phases(rcdp, torch, case, steps):
    """Per-phase host wall time of `steps` whole solves including the graph's
    hand-over: rc_graph_create, rc_build_family, rc_solve, rc_reconstruct
    (each returns after its results reached the host)."""
    acc = {"graph_create_ms": [], "build_family_ms": [], "solve_ms": [], "reconstruct_ms": [],
           "wall_ms": []}
    for _ in range(steps):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        g = rcdp.Graph.create(case.graph)
        t1 = time.perf_counter()
        fam = g.build_family(case.mode)
        t2 = time.perf_counter()
        sol = fam.solve(case.B, case.objective)
        t3 = time.perf_counter()
        if sol.feasible:
            sol.reconstruct()
        t4 = time.perf_counter()
        for k, a, b in (("graph_create_ms", t0, t1), ("build_family_ms", t1, t2),
                        ("solve_ms", t2, t3), ("reconstruct_ms", t3, t4), ("wall_ms", t0, t4)):
            acc[k].append((b - a) * 1e3)
        sol.free()
        fam.free()
        g.free()
    return {k: round(sorted(v)[len(v) // 2], 4) for k, v in acc.items()}


def time_case(rcdp, torch, case, steps, warmup):
    g = rcdp.Graph.create(case.graph)
    for _ in range(warmup):
        run_step(rcdp, g, case)
    torch.cuda.synchronize()
    fills, kernels = [], []
    t0 = time.perf_counter()
    for _ in range(steps):
        info, fill_ms, kernel_ms, (t_star, m_star), sched, kernel = run_step(rcdp, g, case)
        fills.append(fill_ms)
        kernels.append(kernel_ms)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    g.free()
    phases = time_phases(rcdp, torch, case, steps)
    return {
        "phases": phases,
        "ms_per_step": (t1 - t0) * 1e3 / steps,
        "fill_ms": sum(fills) / len(fills),
        "fill_ms_min": min(fills),
        "kernel_ms": sum(kernels) / len(kernels),
        "kernel_ms_min": min(kernels),
        "kernel_ms_median": sorted(kernels)[len(kernels) // 2],
        "kernel_ms_max": max(kernels),
        "info": info,
        "t_star": t_star,
        "m_star": m_star,
        "schedule": sched,
        "k": None if sched is None else int(len(sched.chain)),
        "kernel": kernel,
    }


def mc_sweep(rcdp, torch, name="resnet50", count=32, reps=2):
    """The memory-centric sweep of the ResNet-50-shaped graph: the smallest
    feasible budget (rc_min_budget), then `count` budgets from it to 2 M(V),
    solved in one batched fill (rc_solve_batch) and each traced; the same
    budgets solved one by one are timed beside it."""
    case = workloads_case(name)
    g = rcdp.Graph.create(case.graph)
    fam = g.build_family(case.mode)
    top = 2 * sum(case.graph.M)
    best = None
    for _ in range(reps):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        b_min = fam.min_budget()
        t1 = time.perf_counter()
        budgets = [b_min + (j * (top - b_min)) // (count - 1) for j in range(count)]
        sols = fam.sweep(budgets, "mc")
        for _, sol in sols:
            sol.reconstruct()
        torch.cuda.synchronize()
        t2 = time.perf_counter()
        t_mc = [sol.t_star for _, sol in sols]
        batch_fill = sols[0][1].fill_ms()
        for _, sol in sols:
            sol.free()
        t3 = time.perf_counter()
        fills = []
        for B in budgets:
            sol = fam.solve(B, "mc")
            sol.reconstruct()
            fills.append(round(sol.fill_ms(), 4))
            sol.free()
        torch.cuda.synchronize()
        t4 = time.perf_counter()
        res = {"workload": name, "budgets": count, "B_min": b_min, "B_max": top,
               "min_budget_ms": (t1 - t0) * 1e3, "batched_sweep_ms": (t2 - t1) * 1e3,
               "batched_fill_ms": batch_fill,
               "batched_fill_per_budget_ms": batch_fill / count,
               "one_by_one_ms": (t4 - t3) * 1e3, "one_by_one_fill_ms": fills,
               "t_mc_first_last": [t_mc[0], t_mc[-1]]}
        if best is None or res["batched_sweep_ms"] < best["batched_sweep_ms"]:
            best = res
    fam.free()
    g.free()
    return best


def dual_tables(rcdp, torch, reps=5, names=None):
    """rc_solve_dual on every workload: t*, opt[V, t*] and a schedule from
    the table indexed by cached memory.  step_ms = rc_build_family +
    rc_solve_dual with its schedule (the same outputs as a step of the
    time-indexed path: t*, chain, Eq. 1 / Eq. 2), fill_ms = its table
    kernels; `agrees` records that (t*, opt[V, t*]) equals rc_solve's on the
    same family and that the schedule re-evaluates to them."""
    from paper_1905_11722_amd import workloads
    out = {}
    for name in names or workloads.CASES:
        case = workloads.case(name)
        g = rcdp.Graph.create(case.graph)
        steps, fills = [], []
        fam = None
        for r in range(reps + 1):
            if fam is not None:
                fam.free()
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            fam = g.build_family(case.mode)
            t, m, ms, sched = fam.solve_dual(case.B, case.objective, schedule=True)
            torch.cuda.synchronize()
            t1 = time.perf_counter()
            if r > 0:
                steps.append((t1 - t0) * 1e3)
                fills.append(ms)
        sol = fam.solve(case.B, case.objective)
        agrees = (t, m) == (sol.t_star, sol.m_star) and (
            sched is None or (sched.overhead, sched.cache_mem) == (t, m))
        sol.free()
        width = min(case.B, 2 * sum(case.graph.M), sum(case.graph.M)) + 1
        out[name] = {"step_ms": round(sorted(steps)[len(steps) // 2], 4),
                     "fill_ms": round(sorted(fills)[len(fills) // 2], 4),
                     "cells": fam.info["num_sets"] * width, "t_star": t, "m_star": m,
                     "agrees": agrees}
        fam.free()
        g.free()
    return out


def dominance_fills(rcdp, torch, reps=5, names=None):
    """rc_solve_dominance (the skip of Section 4.2 on the level fill) against
    rc_solve on the same family, with its default fill and with the level
    fill forced (RCDP_FILL=level: the skip's own cost and gain): fill_ms of
    each (median of reps), and `agrees` = equal (t*, opt[V, t*])."""
    from paper_1905_11722_amd import workloads
    out = {}
    for name in names or ("resnet50", "unet", "densenet121"):
        case = workloads.case(name)
        g = rcdp.Graph.create(case.graph)
        fam = g.build_family(case.mode)
        dom, plain, level = [], [], []
        agrees = True
        for r in range(reps + 1):
            a = fam.solve_dominance(case.B)
            b = fam.solve(case.B, "tc")
            os.environ["RCDP_FILL"] = "level"
            try:
                c = fam.solve(case.B, "tc")
            finally:
                os.environ.pop("RCDP_FILL", None)
            if r > 0:
                dom.append(a.fill_ms())
                plain.append(b.fill_ms())
                level.append(c.fill_ms())
            agrees = agrees and (a.t_star, a.m_star) == (b.t_star, b.m_star) == (c.t_star, c.m_star)
            a.free()
            b.free()
            c.free()
        out[name] = {"fill_ms": round(sorted(dom)[len(dom) // 2], 4),
                     "rc_solve_fill_ms": round(sorted(plain)[len(plain) // 2], 4),
                     "rc_solve_level_fill_ms": round(sorted(level)[len(level) // 2], 4),
                     "agrees": agrees}
        fam.free()
        g.free()
    return out


def workloads_case(name):
    from paper_1905_11722_amd import workloads
    return workloads.case(name)


def host_description():
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        usable = len(os.sched_getaffinity(0))
    except AttributeError:
        usable = os.cpu_count()
    return {"nproc": usable, "cpu_count": os.cpu_count(), "cpu_model": model,
            "omp_num_threads": os.environ.get("OMP_NUM_THREADS")}


def cpu_baseline(case, relaxations):
    """The oracle (Algorithm 1 as printed, t over 0..T(V)) on this host: one
    full solve of the workload with the all-cores OpenMP build (the reported
    value) and one with the single-threaded build, both rated against the
    same relaxation count as the GPU.  Their tables are identical
    (tests/test_oracle_parallel.py)."""
    from oracle import oracle
    legs = {}
    ref = None
    for parallel in (True, False):
        # the single-threaded leg runs pinned to one core of the allowed set
        keep = os.sched_getaffinity(0) if hasattr(os, "sched_getaffinity") else None
        if not parallel and keep:
            os.sched_setaffinity(0, {min(keep)})
        try:
            t0 = time.perf_counter()
            r = oracle.solve(case.graph, case.mode, case.B, case.objective, parallel=parallel)
            dt = time.perf_counter() - t0
        finally:
            if not parallel and keep:
                os.sched_setaffinity(0, keep)
        legs[parallel] = (dt, r.t_star, r.num_sets, oracle.threads(parallel))
        if parallel:
            ref = r
        else:
            del r
    dt, t_star, num_sets, cores = legs[True]
    dt1, t_star1, _, _ = legs[False]
    assert t_star1 == t_star
    return ref, {
        "value": relaxations / dt,
        "unit": "relaxations/s",
        "cores": cores,
        "kind": "oracle",
        "sample": (f"one full {case.objective.upper()} solve of {case.name} "
                   f"(Algorithm 1 over all {num_sets} sets, t over 0..T(V)) with the "
                   f"OpenMP build on {cores} threads, {dt:.2f} s; t*={t_star}"),
        "seconds": dt,
        "t_star": t_star,
        "one_core": {"value": relaxations / dt1, "seconds": dt1, "cores": 1,
                     "pinned": hasattr(os, "sched_setaffinity")},
        "host": host_description(),
    }


def same_run_parity(ref, res):
    """The GPU's last timed step against the oracle's solve of the same
    workload in this run: t*, opt[V, t*], the traced chain, seg, cached and
    the Eq. 1 / Eq. 2 re-evaluation (the whole tables are compared in the GPU
    tests)."""
    out = {"t_star": res["t_star"] == ref.t_star, "m_star": res["m_star"] == ref.m_star}
    sched = res["schedule"]
    if sched is not None and ref.t_star >= 0:
        chain, seg, cached = ref.schedule()
        out["chain"] = list(map(int, sched.chain)) == list(map(int, chain))
        out["seg"] = list(map(int, sched.seg)) == list(map(int, seg))
        out["cached"] = list(map(bool, sched.cached)) == list(map(bool, cached))
        out["overhead_peak_cache"] = (sched.overhead, sched.peak, sched.cache_mem) == (
            ref.overhead, ref.peak, ref.cache_mem)
    out["all_equal"] = all(out.values())
    return out


def measured_peaks(torch, copy_bytes=2 << 30):
    """The chip's integer VALU rates and HBM copy bandwidth, measured now by
    the microbenchmarks of libpeak.so (best of a few launches)."""
    import ctypes

    from paper_1905_11722_amd import build as hip_build
    lib = ctypes.CDLL(hip_build.PEAK_LIB)
    lib.peak_valu.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_void_p,
                              ctypes.POINTER(ctypes.c_float), ctypes.POINTER(ctypes.c_double)]
    lib.peak_copy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int,
                              ctypes.POINTER(ctypes.c_float)]
    blocks = 256 * 16
    out = torch.empty(blocks * 256, dtype=torch.int32, device="cuda")
    res = {}
    for kind, key in ((0, "valu_int32_tops"), (1, "valu_pk_u16_tops")):
        best = 0.0
        for rep in range(4):
            ms, ops = ctypes.c_float(), ctypes.c_double()
            assert lib.peak_valu(kind, blocks, 200, ctypes.c_void_p(out.data_ptr()),
                                 ctypes.byref(ms), ctypes.byref(ops)) == 0
            if rep:
                best = max(best, ops.value / (ms.value / 1e3) / 1e12)
        res[key] = best
    src = torch.ones(copy_bytes // 4, dtype=torch.int32, device="cuda")
    dst = torch.empty_like(src)
    best = 0.0
    for rep in range(4):
        ms = ctypes.c_float()
        assert lib.peak_copy(ctypes.c_void_p(src.data_ptr()), ctypes.c_void_p(dst.data_ptr()),
                             copy_bytes, 256 * 64, ctypes.byref(ms)) == 0
        if rep:
            best = max(best, 2 * copy_bytes / (ms.value / 1e3) / 1e9)
    torch.cuda.synchronize()
    assert bool((dst[-8:] == 1).all())
    res["hbm_copy_gbs"] = best
    res["copy_bytes"] = copy_bytes
    res["note"] = ("independent add/min chains (32-bit and packed 16-bit), 4096 workgroups "
                   "of 256; HBM: read + write bytes of a device-to-device copy")
    del src, dst, out
    return res


def copy_calibration(nbytes):
    """One device-to-device copy of nbytes: reads and writes nbytes of HBM."""
    import torch
    assert torch.cuda.is_available(), "the copy calibration needs a GPU"
    n = nbytes // 4
    src = torch.arange(n, dtype=torch.int32, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    dst.copy_(src)
    torch.cuda.synchronize()
    assert bool((dst[-16:] == src[-16:]).all())
    print(json.dumps({"copy_calibration_bytes": n * 4}), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="densenet121")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-other-graphs", action="store_true")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES")
    ap.add_argument("--dominance", action="store_true",
                    help="time only the level fill with the dominance skip (rc_solve_dominance) "
                         "against rc_solve on --workload")
    ap.add_argument("--dual", action="store_true",
                    help="time only the memory-indexed table (rc_solve_dual) on --workload")
    args = ap.parse_args()
    if args.copy_calibration:
        copy_calibration(args.copy_calibration)
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (--gpus {args.gpus} requested): the DP of one "
              "graph does not shard across GPUs; independent solves would.", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_1905_11722_amd import rcdp, workloads

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    rcdp.load_library()
    if args.dominance:
        res = dominance_fills(rcdp, torch, reps=max(3, args.steps), names=[args.workload])
        print(json.dumps({"dominance": res}), flush=True)
        return
    if args.dual:
        res = dual_tables(rcdp, torch, reps=max(3, args.steps), names=[args.workload])
        print(json.dumps({"dual": res}), flush=True)
        return

    case = workloads.case(args.workload)
    main_res = time_case(rcdp, torch, case, args.steps, args.warmup)
    info = main_res["info"]
    W = info["relaxations"]
    step_s = main_res["ms_per_step"] / 1e3
    fill_s = main_res["fill_ms"] / 1e3
    kernel_s = main_res["kernel_ms"] / 1e3
    achieved = OPS_PER_RELAXATION * W / kernel_s / 1e12

    per_graph = {}
    if not args.no_other_graphs:
        for name in workloads.CASES:
            if name == args.workload:
                r = main_res
            else:
                r = time_case(rcdp, torch, workloads.case(name), max(3, args.steps // 4), 1)
            per_graph[name] = {
                "wall_ms": r["phases"]["wall_ms"],
                "step_ms": round(r["ms_per_step"], 4),
                "phases": r["phases"],
                "fill_ms": round(r["fill_ms"], 4),
                "relaxations": r["info"]["relaxations"],
                "relax_per_s_fill": r["info"]["relaxations"] / (r["fill_ms"] / 1e3)
                if r["fill_ms"] > 0 else None,
                "t_star": r["t_star"],
                "k": r["k"],
            }

    peaks = measured_peaks(torch)
    sweep = None if args.no_other_graphs else mc_sweep(rcdp, torch)
    dual = None if args.no_other_graphs else dual_tables(rcdp, torch)
    dominance = None if args.no_other_graphs else dominance_fills(rcdp, torch, reps=3)

    out = {
        "metric": "DP cell relaxations/sec (whole step: family + fill + traceback)",
        "value": W / step_s,
        "unit": "relaxations/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": main_res["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u16",
        "data": "synthetic",
        "config": {
            "workload": case.name,
            "description": case.note,
            "nodes": info["n"],
            "family": case.mode,
            "B": case.B,
            "objective": case.objective,
            "sets": info["num_sets"],
            "pairs": info["num_pairs"],
            "levels": info["num_levels"],
            "T_total": info["T_total"],
            "table_cells": info["table_cells"],
            "relaxations": W,
            "t_star": main_res["t_star"],
        },
        "phases": main_res["phases"],
        "step_ms_with_graph_create": main_res["phases"]["wall_ms"],
        "fill_ms": main_res["fill_ms"],
        "fill_relax_per_s": W / fill_s,
        "fill_kernel_ms": {k: main_res[f"kernel_ms{s}"] for k, s in
                           (("mean", ""), ("median", "_median"), ("min", "_min"),
                            ("max", "_max"))},
        "roofline": {
            "bound": "alu",
            "achieved": achieved,
            "peak": VALU_U16_PEAK_TOPS,
            "unit": "TOP/s (packed 16-bit integer VALU)",
            "frac": achieved / VALU_U16_PEAK_TOPS,
            "traffic": read_traffic(main_res["kernel"], case.name),
            "traffic_unit": "HBM bytes per launch (rocprofv3 FETCH_SIZE + WRITE_SIZE)",
            "kernel": main_res["kernel"],
            "kernel_ms": main_res["kernel_ms"],
            "ops_per_relaxation": OPS_PER_RELAXATION,
            "frac_of_int32_peak": achieved / VALU_INT32_PEAK_TOPS,
            "measured_peak_pk_u16": peaks["valu_pk_u16_tops"],
            "frac_of_measured_pk_u16": achieved / peaks["valu_pk_u16_tops"],
            "measured_peak_int32": peaks["valu_int32_tops"],
            "frac_of_measured_int32": achieved / peaks["valu_int32_tops"],
        },
        "peaks": peaks,
        "per_graph": per_graph,
        "mc_sweep": sweep,
        "dual": dual,
        "dominance": dominance,
    }
    if not args.no_cpu_baseline:
        ref, out["cpu_baseline"] = cpu_baseline(case, W)
        out["parity"] = same_run_parity(ref, main_res)
        assert out["parity"]["all_equal"], f"oracle and GPU disagree: {out['parity']}"
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
