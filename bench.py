"""Benchmark: candidate plans scored per second on one MI355X.

A step is one dy_plan_select over the workload's whole plan set: the seeding
pre-pass, the fp32 scoring pass over every plan, certification of the
candidates in fp64 and the copy of the K winners back to the host.  The
problem tables are staged once (dy_plan_create) before timing; their staging
time is reported separately as "stage_ms".

Default workload: forkjoin8 (8-node fork-join DAG, 12 implementations per
node, 12^8 = 429,981,696 plans, 8 pressure levels).  --workload picks another
(chain4, layered10, batch6, stream24) for profiling; --objective scores it
under the paper's additive objective J_L instead (levels L in {0, 1.5, 3},
call cost c = tau * size), a separate measurement of that mode.

Two timed loops of the same K calls: the first, as a caller runs them
(repeated calls replay one HIP graph), gives "value" and "ms_per_step"; the
second runs with the library's timing option, which records HIP events around
the scoring kernel on the call's stream (timed calls launch directly, since
events inside a graph are not updated by its replays), and gives the
roofline's kernel duration ("ms_per_step_timed" is that loop's step time).

Prints one JSON line (rank 0).  The roofline object describes the dominant
kernel; "traffic" is the HBM traffic per launch from stored rocprofv3
FETCH_SIZE / WRITE_SIZE counters (calibrated on a device copy), reported only
while the kernel sources are the ones the counters were taken on.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "candidate plans scored/sec on 1 MI355X; % of FP32 VALU (or HBM) roofline"
# MI355X: 256 CUs x 4 SIMDs x 16 lanes at 2.4 GHz; a SIMD completes one 64-lane
# VALU instruction every 4 cycles (the SQ counters count one quad-cycle of
# SQ_ACTIVE_INST_VALU per instruction), so unpacked fp32 / integer operations
# peak at 256 x 4 x 16 x 2.4e9 = 39.3e12 lane-ops/s.  The vendor's 157.3
# TFLOP/s counts packed fp32 FMA (two lanes' worth of FMA per lane-instruction,
# 2 flops each); packed fp32 instructions are disabled in this build and this
# op mix has no FMA, so 39.3e12 is the ceiling; the packed-equivalent 78.6e12
# is reported beside it.
PEAK_VALU = 256 * 4 * 16 * 2.4e9
PEAK_VALU_PACKED = 2 * PEAK_VALU
PEAK_HBM = 8.0e12                 # bytes/s

# Kernel sources whose hash keys the stored HBM-traffic counters: a stored
# figure is reported only while these files are unchanged.
KERNEL_SOURCES = ("paper_2607_02942_amd/csrc/kernels.hip", "paper_2607_02942_amd/csrc/jit_rows.cpp",
                  "paper_2607_02942_amd/csrc/dyplan_internal.h")
DOMINANT = {"stream24": "dy_rows_scan_a", "stream24_obj": "dy_rows_scan_a",
            "stream24_perclass": "dy_rows_scan_a", "forkjoin8": "dy_sweep", "forkjoin8_obj": "dy_sweep",
            "layered10": "dy_sweep", "forkjoin8_perclass": "dy_sweep",
            "layered10_perclass": "dy_sweep"}  # else the library's sweep kernel


def score_kernel(prob, per_class):
    """The kernel dy_plan_score runs for a 2^26-plan range of `prob`."""
    if per_class:
        return "k_score"
    return "dy_score_range" if prob.n_nodes > 16 else "k_score_fast"
OBJ_SWEEP = "k_sweep_obj"


def kernel_source_sha():
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def traffic_path(workload):
    return os.path.join(ROOT, "profiles", f"traffic_{workload}.json")


def stored_traffic(workload):
    """HBM bytes per launch of the dominant kernel, from the counters stored
    for the current kernel sources (None when absent or stale)."""
    try:
        with open(traffic_path(workload)) as fh:
            t = json.load(fh)
    except (OSError, ValueError):
        return None
    return t["traffic_bytes_per_launch"] if t.get("source_sha") == kernel_source_sha() else None


def _pmc_means(db, counter):
    """{kernel name: mean per dispatch of `counter`} from a rocprofv3 counter database."""
    import sqlite3
    con = sqlite3.connect(db)
    per = {}
    for name, disp, val in con.execute(
            "select kernel_name, dispatch_id, sum(value) from counters_collection where counter_name = ? "
            "group by dispatch_id", (counter,)):
        per.setdefault(name, []).append(val)
    return {k: sum(v) / len(v) for k, v in per.items()}


def ingest_pmc(workload, fetch_db, write_db, calib_fetch_db, calib_write_db, calib_bytes, commands):
    """Store the dominant kernel's HBM traffic per launch: FETCH_SIZE and
    WRITE_SIZE (KiB per dispatch), each scaled by bytes / counter of a plain
    device copy of known size."""
    def pick(means, key):
        hits = [(k, v) for k, v in means.items() if key in k]
        if not hits:
            raise SystemExit(f"no kernel matching {key!r} in {sorted(means)}")
        return hits[0]
    if workload.endswith("_score"):
        import paper_2607_02942_amd.workload as wlm
        kern = score_kernel(wlm.by_name(workload.split("_")[0]), "_perclass" in workload)
    else:
        kern = DOMINANT.get(workload, OBJ_SWEEP if workload.endswith("_obj") else "k_sweep")
    kname, fetch = pick(_pmc_means(fetch_db, "FETCH_SIZE"), kern)
    _, write = pick(_pmc_means(write_db, "WRITE_SIZE"), kern)
    _, cf = pick(_pmc_means(calib_fetch_db, "FETCH_SIZE"), "copyBuffer")
    _, cw = pick(_pmc_means(calib_write_db, "WRITE_SIZE"), "copyBuffer")
    ff, fw = calib_bytes / (cf * 1024.0), calib_bytes / (cw * 1024.0)
    rec = {"workload": workload, "kernel": kname, "source_sha": kernel_source_sha(),
           "fetch_kib_per_dispatch": fetch, "write_kib_per_dispatch": write,
           "calib_copy_bytes": calib_bytes, "calib_fetch_kib": cf, "calib_write_kib": cw,
           "fetch_factor": ff, "write_factor": fw,
           "traffic_bytes_per_launch": fetch * 1024.0 * ff + write * 1024.0 * fw,
           "commands": commands}
    with open(traffic_path(workload), "w") as fh:
        json.dump(rec, fh, indent=1)
    print(json.dumps(rec), flush=True)


def edge_count(prob):
    return len({(int(u), int(v)) for u, v in prob.edges})


def sweep_work_per_plan(prob):
    """Algorithmic fp32 operations per plan of the prefix-shared sweep.

    Per plan: 1 multiply (corr), 1 add (CP), 1 compare (prefilter); per row of
    the inner sweep (R_y plans): the add and multiply of node x and the max of
    y's predecessors; per block (R_x R_y plans): the prefix products and one
    max/add per prefix edge.  Counted like the full recurrence, operation by
    operation, so the figure never exceeds the work actually done.
    """
    n = prob.n_nodes
    rx = int(prob.radix[n - 2]) if n >= 2 else 1
    ry = int(prob.radix[n - 1])
    edges = {(int(u), int(v)) for u, v in prob.edges}
    npre = max(n - 2, 0)
    pre_edges = sum(1 for u, v in edges if v < npre)
    x_pred = sum(1 for u, v in edges if v == n - 2)
    y_pred = sum(1 for u, v in edges if v == n - 1 and u != n - 2)
    per_plan = 3.0
    per_row = 2.0 + (1.0 if (n - 2, n - 1) in edges and y_pred > 0 else 0.0)
    per_block = max(npre - 1, 0) + pre_edges + x_pred + y_pred
    return per_plan + per_row / ry + per_block / (rx * ry)


def obj_sweep_work_per_plan(prob):
    """Algorithmic fp32 operations per plan of the objective-mode sweep.

    Per plan: the add of y's duration (T), the max with the prefix sinks' path
    when there is one, the adds of y's utility (U) and d (D), the fused
    multiply-add G = U - lambda_l T and the prefilter compare; per row: the
    adds of node x (its path, utility and d) and the max of y's predecessors;
    per block: the prefix sums of u and d and one max/add per prefix edge.
    """
    n = prob.n_nodes
    rx = int(prob.radix[n - 2]) if n >= 2 else 1
    ry = int(prob.radix[n - 1])
    edges = {(int(u), int(v)) for u, v in prob.edges}
    npre = max(n - 2, 0)
    pre_edges = sum(1 for u, v in edges if v < npre)
    x_pred = sum(1 for u, v in edges if v == n - 2)
    y_pred = sum(1 for u, v in edges if v == n - 1 and u != n - 2)
    pre_sinks = any(all(u != m for u, v in edges) for m in range(npre))
    has_s2 = pre_sinks or (n - 2, n - 1) not in edges
    per_plan = 5.0 + (1.0 if has_s2 else 0.0)
    per_row = 3.0 + (1.0 if (n - 2, n - 1) in edges and y_pred > 0 else 0.0)
    per_block = 2 * max(npre - 1, 0) + pre_edges + x_pred + y_pred
    return per_plan + per_row / ry + per_block / (rx * ry)


def full_work_per_plan(prob, K):
    """The per-plan count of the full recurrence: (N-1) mul + E max/add + K compares."""
    return (prob.n_nodes - 1) + edge_count(prob) + K


def cpu_baseline(prob, sample_plans=None, rows=None, obj=None):
    from oracle import oracle as orc
    t0 = time.perf_counter()
    if rows is not None:
        if obj is None:
            orc.select_rows(prob, rows, 0)
        else:
            orc.obj_select_rows(prob, obj, rows, 0)
        n = rows.shape[0]
        what = f"first {n} rows"
    else:
        if obj is None:
            orc.select_range(prob, 0, sample_plans)
        else:
            orc.obj_select_range(prob, obj, 0, sample_plans)
        n = sample_plans
        what = f"plan indices [0, {sample_plans})"
    dt = time.perf_counter() - t0
    return {"value": n / dt, "unit": "plans/s", "cores": 1, "kind": "oracle",
            "sample": f"{prob.name}: {what}, single-threaded fp64 oracle, {dt:.1f} s"}


def score_bench(args, torch, D, wl, stream, tkey):
    """Per-plan scores of a forkjoin8 range into device buffers: corr, CP at each
    level, demand and feasibility bits, 4 (3 + K) bytes per plan, write-bound."""
    prob = wl.by_name(args.workload if args.workload != "batch6" else "forkjoin8")
    if args.pressure == "per-class":
        prob = wl.per_class(prob)
    K = prob.n_levels
    n = min(1 << 26, prob.n_plans() if args.workload != "layered10" else 1 << 32)
    corr = torch.empty(n, dtype=torch.float32, device="cuda")
    cp = torch.empty(n, K, dtype=torch.float32, device="cuda")
    dem = torch.empty(n, dtype=torch.float32, device="cuda")
    feas = torch.empty(n, dtype=torch.int32, device="cuda")
    with D.Plan(prob) as plan:
        src = D.range_source(0, 0, n)
        for _ in range(args.warmup):
            plan.score(src, corr, cp, dem, feas, stream=stream)
        ev0 = torch.cuda.Event(enable_timing=True)
        ev1 = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        ev0.record(stream)
        for i in range(args.steps):
            plan.score(src, corr, cp, dem, feas, stream=stream)
        ev1.record(stream)
        torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1) / args.steps
    per_plan = 4.0 * (3 + K)
    achieved = n * per_plan / (ms / 1e3)
    res = {"metric": "plans scored/sec by dy_plan_score on 1 MI355X (per-plan outputs)", "value": n / (ms / 1e3),
           "unit": "plans/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms,
           "higher_is_better": True, "dtype": "f32", "data": "synthetic",
           "config": {"workload": prob.name, "plans": n, "levels": K, "outputs": "corr, cp[K], demand, feas"},
           "roofline": {"bound": "hbm", "kernel": score_kernel(prob, args.pressure == "per-class"),
                        "achieved": achieved / 1e9, "peak": PEAK_HBM / 1e9,
                        "unit": "GB/s", "frac": achieved / PEAK_HBM, "per_unit": f"{per_plan:.0f} B written per plan",
                        "traffic": stored_traffic(tkey)}}
    print(json.dumps(res), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="forkjoin8",
                    choices=["chain4", "forkjoin8", "layered10", "batch6", "stream24"])
    ap.add_argument("--objective", action="store_true",
                    help="the paper's additive objective J_L (levels 0, 1.5, 3) instead of corr / SLO")
    ap.add_argument("--pressure", choices=["level", "per-class"], default="level",
                    help="per-class: the second backend pressed at half the level's rho (per-backend pressure)")
    ap.add_argument("--score", action="store_true",
                    help="time dy_plan_score (per-plan corr, CP per level, demand, feasibility bits) instead")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample", type=int, default=1 << 26)
    ap.add_argument("--sample-stride", type=int, default=0)
    ap.add_argument("--calib-copy", type=int, default=0, help="MiB: run one device copy (counter calibration)")
    ap.add_argument("--ingest-pmc", nargs=4, metavar=("FETCH_DB", "WRITE_DB", "CALIB_FETCH_DB", "CALIB_WRITE_DB"),
                    help="store the dominant kernel's traffic from rocprofv3 --pmc databases (no GPU needed)")
    ap.add_argument("--calib-bytes", type=int, default=1 << 30)
    ap.add_argument("--pmc-command", action="append", default=[], help="command that produced a database")
    args = ap.parse_args()
    tkey = args.workload + ("_obj" if args.objective else "") + ("_perclass" if args.pressure == "per-class" else "")
    if args.score:
        tkey = args.workload + ("_perclass" if args.pressure == "per-class" else "") + "_score"
    if args.ingest_pmc:
        ingest_pmc(tkey, *args.ingest_pmc, args.calib_bytes, args.pmc_command)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(the work would shard by plan range or row range, one shard per GPU)", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2607_02942_amd import dyplan as D
    from paper_2607_02942_amd import workload as wl

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream()

    if args.calib_copy:
        n = args.calib_copy << 20
        a = torch.empty(n, dtype=torch.uint8, device="cuda")
        b = torch.empty(n, dtype=torch.uint8, device="cuda")
        a.fill_(1)
        torch.cuda.synchronize()
        b.copy_(a)
        torch.cuda.synchronize()
        print(json.dumps({"calib_copy_bytes": n}), flush=True)
        return

    if args.score:
        score_bench(args, torch, D, wl, stream, tkey)
        return

    name = args.workload
    rows_dev = None
    rows_host = None
    if name == "batch6":
        probs = wl.batch6()
        sources = [D.range_source(r, 0, 12 ** 6) for r in range(len(probs))]
        plans = len(probs) * 12 ** 6
    else:
        probs = [wl.by_name(name)]
        if name == "stream24":
            plans = wl.STREAM_ROWS
            rows_host = wl.make_rows(plans, 24, 36)
            rows_dev = torch.from_numpy(rows_host).cuda()
            sources = [D.rows_source(0, rows_dev, plans, 24, 0)]
        else:
            plans = wl.LAYERED_RANGE if name == "layered10" else probs[0].n_plans()
            sources = [D.range_source(0, 0, plans)]
    if args.pressure == "per-class":
        probs = [wl.per_class(p) for p in probs]
    prob = probs[0]
    K = prob.n_levels
    objs = None
    if args.objective:
        objs = [wl.paper_objective(p) for p in probs]
        K = objs[0].n_levels
    else:
        for p in probs:
            assert np.isfinite(p.slo), f"stored SLO missing for {p.name}"

    t0 = time.perf_counter()
    plan = D.Plan(list(zip(probs, objs)) if objs else probs, device=0)
    stage_ms = (time.perf_counter() - t0) * 1e3
    if args.sample_stride:
        plan.set_option(D.DY_OPT_SAMPLE_STRIDE, args.sample_stride)
    srcs = (D.DySource * len(sources))(*sources)
    out = (D.DyChoice * (len(sources) * plan.kmax))()

    def step():
        st = plan.select_raw(srcs, len(sources), out, stream)
        if st != 0:
            raise RuntimeError(f"select failed {st}: {D.last_error(plan._h)}")

    def timed_loop(tag, collect):
        # collect: read the library's per-call statistics after every step
        # (the caller-side loop does not, as a caller needs only the choices)
        cands, main_ms, gen = [], [], []
        ev0 = torch.cuda.Event(enable_timing=True)
        ev1 = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        ev0.record(stream)
        for i in range(args.steps):
            step()
            if collect:
                s = plan.stats()
                main_ms.append(s.main_ms)
                cands.append(s.candidates)
                gen.append(s.generated_jobs)
            if i == 0 or (i + 1) % max(1, args.steps // 4) == 0:
                print(f"[bench] {tag} step {i + 1}/{args.steps}", file=sys.stderr, flush=True)
        ev1.record(stream)
        torch.cuda.synchronize()
        return ev0.elapsed_time(ev1) / args.steps, main_ms, cands, gen

    # 1) the steps as a caller runs them: repeated calls replay one HIP graph
    for _ in range(args.warmup):
        step()
    ms_per_step, _, _, _ = timed_loop("step", False)
    value = plans / (ms_per_step / 1e3)
    # 2) the same calls with the library's HIP events around the scoring kernel
    #    (on the call's stream; timed calls launch directly, not from a graph)
    plan.set_option(D.DY_OPT_TIMING, 1)
    for _ in range(max(1, args.warmup // 2)):
        step()
    ms_per_step_timed, main_ms, cands, gen = timed_loop("timed", True)
    generated = bool(gen) and max(gen) > 0  # the library ran a kernel generated for the problem
    kern_ms = float(np.mean(main_ms))
    kern_plans_s = plans / (kern_ms / 1e3)

    if name == "stream24":
        bytes_per_plan = 24.0
        achieved = kern_plans_s * bytes_per_plan
        kname = "dy_rows_scan_a (rows, generated for the DAG" + (", objective)" if objs else ")")
        roof = {"bound": "hbm", "kernel": kname, "achieved": achieved / 1e9,
                "peak": PEAK_HBM / 1e9, "unit": "GB/s", "frac": achieved / PEAK_HBM,
                "traffic": stored_traffic(tkey), "per_unit": "24 B of row per plan", "kernel_ms": kern_ms}
    else:
        f = obj_sweep_work_per_plan(prob) if objs else sweep_work_per_plan(prob)
        achieved = kern_plans_s * f
        if generated:
            kname = "dy_sweep (generated for the DAG" + (", objective)" if objs else ")")
        else:
            kname = OBJ_SWEEP if objs else "k_sweep"
        roof = {"bound": "alu", "kernel": kname, "achieved": achieved / 1e12,
                "peak": PEAK_VALU / 1e12, "unit": "TFLOP/s", "frac": achieved / PEAK_VALU,
                "peak_packed_fp32": PEAK_VALU_PACKED / 1e12, "frac_vs_packed_fp32": achieved / PEAK_VALU_PACKED,
                "traffic": stored_traffic(tkey),
                "per_unit": f"{f:.4f} fp32 ops per plan (prefix-shared sweep{', objective' if objs else ''})",
                "kernel_ms": kern_ms}
        if not objs:
            roof["full_recurrence_ops_per_plan"] = full_work_per_plan(prob, K)

    res = {
        "metric": METRIC, "value": value, "unit": "plans/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms_per_step, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": name, "plans": plans, "nodes": prob.n_nodes, "edges": edge_count(prob),
                   "impls_per_node": int(prob.radix[0]), "levels": K,
                   "problems": len(probs), "parallelism": "single GPU",
                   "selection": "paper objective J_L, L in {0, 1.5, 3}" if objs else "max corr s.t. CP_k <= SLO",
                   "pressure": "per-class (backend 1 at rho_k / 2)" if args.pressure == "per-class" else "per level"},
        "roofline": roof,
        "stage_ms": stage_ms,
        "ms_per_step_timed": ms_per_step_timed,
        "candidates_per_step": float(np.mean(cands)),
    }
    if not args.no_cpu_baseline:
        o0 = objs[0] if objs else None
        if name == "stream24":
            res["cpu_baseline"] = cpu_baseline(prob, rows=rows_host[: 1 << 22], obj=o0)
        elif name == "batch6":
            res["cpu_baseline"] = cpu_baseline(prob, sample_plans=12 ** 6, obj=o0)
        else:
            res["cpu_baseline"] = cpu_baseline(prob, sample_plans=min(args.cpu_sample, plans), obj=o0)
    plan.close()
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
