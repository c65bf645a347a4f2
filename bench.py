"""Benchmark: candidate plans scored per second on one MI355X.

A step is one dy_plan_select over the workload's whole plan set: the seeding
pre-pass, the fp32 scoring pass over every plan, certification of the
candidates in fp64 and the copy of the K winners back to the host.  The
problem tables are staged once (dy_plan_create) before timing; their staging
time is reported separately as "stage_ms".

Default workload: batch6, the largest single-GPU configuration: 4,096
requests, each its own random 6-node DAG with 12 implementations per node,
every request's 12^6 = 2,985,984 plans scored at 4 pressure levels
(12,230,590,464 plans per step).  --workload picks another (chain4, forkjoin8,
layered10, stream24); --objective scores it under the paper's additive
objective J_L instead (levels L in {0, 1.5, 3}, call cost c = tau * size);
--pressure per-class presses the second backend at half the level's rho.

Two timed loops of the same K calls: the first, as a caller runs them
(repeated calls replay one HIP graph), gives "value" and "ms_per_step"; the
second runs with the library's timing option, which records HIP events around
the scoring kernel on the call's stream (timed calls launch directly, since
events inside a graph are not updated by its replays), and gives the
roofline's kernel duration ("ms_per_step_timed" is that loop's step time).
The choices of the last call are compared with the oracle's stored selections
(tests/golden/select_<workload>.json, written by oracle/golden.py) where the
mode has them; a mismatch exits non-zero after the JSON line.

The CPU baseline (the fp64 oracle, single-threaded) runs first, in a child
process pinned to one core with taskset, before the GPU is touched.

Prints one JSON line.  The roofline object describes the dominant kernel;
"traffic" is its HBM traffic per step (every launch of it in a step) from
stored rocprofv3 FETCH_SIZE / WRITE_SIZE counters (calibrated on a device
copy), reported only while the kernel sources are the ones the counters were
taken on.

Modes that need no GPU turn rocprofv3 output into the summaries kept under
profiles/: --trace-summary (kernel trace), --pmc-summary (SQ counters),
--ingest-pmc (HBM traffic record).
"""
from __future__ import annotations

import argparse
import json
import os
import subprocess
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "candidate plans scored/sec on 1 MI355X; % of FP32 VALU (or HBM) roofline"
# MI355X: 256 CUs x 4 SIMDs x 16 lanes at 2.4 GHz; a SIMD completes one 64-lane
# VALU instruction every 4 cycles, so unpacked fp32 / integer operations peak
# at 256 x 4 x 16 x 2.4e9 = 39.3e12 lane-ops/s.  The vendor's 157.3 TFLOP/s
# counts packed fp32 FMA (two lanes' worth of FMA per lane-instruction, 2
# flops each); packed fp32 instructions are disabled in this build and this op
# mix has no FMA, so 39.3e12 is the ceiling; the packed-equivalent 78.6e12 is
# reported beside it.
N_CU = 256
CLOCK_HZ = 2.4e9
PEAK_VALU = N_CU * 4 * 16 * CLOCK_HZ
PEAK_VALU_PACKED = 2 * PEAK_VALU
PEAK_HBM = 8.0e12                 # bytes/s

# Sources whose hash keys a kernel's stored HBM-traffic counters: the file
# that defines it (the library's kernels, or the generator of the per-problem
# "dy_*" kernels), the device layout they share, and the host code that sizes
# and launches them.  A stored figure is reported only while these files are
# unchanged.
CSRC = "paper_2607_02942_amd/csrc/"


def kernel_sources(kernel):
    own = CSRC + ("jit_rows.cpp" if kernel.startswith("dy_") else "kernels.hip")
    return (own, CSRC + "dyplan_internal.h", CSRC + "host.cpp")


GOLDEN_DIR = os.path.join(ROOT, "tests", "golden")
WORKLOADS = ["chain4", "forkjoin8", "layered10", "batch6", "stream24"]


# ---------------------------------------------------------------------------
# kernel names
# ---------------------------------------------------------------------------

def kernel_base(name):
    """Base name of a (demangled) kernel name: 'void dyp::k_sweep<false, 12, 4>(...)' -> 'k_sweep'."""
    depth, out = 0, []
    for ch in name.split("(")[0]:  # drop template arguments
        if ch == "<":
            depth += 1
        elif ch == ">":
            depth -= 1
        elif depth == 0:
            out.append(ch)
    toks = "".join(out).split()
    return toks[-1].split("::")[-1] if toks else name


def match_kernel(names, base):
    """The names whose base name is exactly `base`."""
    return [n for n in names if kernel_base(n) == base]


def score_kernel(prob, per_class):
    """The kernel dy_plan_score runs for a 2^26-plan range of `prob`."""
    return "k_score" if per_class else "k_score_row"


def kernel_source_sha(kernel):
    import hashlib
    h = hashlib.sha256()
    for f in kernel_sources(kernel):
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def traffic_path(key):
    return os.path.join(ROOT, "profiles", f"traffic_{key}.json")


def stored_traffic(key, kernel):
    """HBM bytes per step of `kernel`, from the counters stored for the
    current kernel sources (None when absent, stale or of another kernel)."""
    try:
        with open(traffic_path(key)) as fh:
            t = json.load(fh)
    except (OSError, ValueError):
        return None
    if t.get("kernel_base") != kernel or t.get("source_sha") != kernel_source_sha(kernel):
        return None
    return t["traffic_bytes_per_step"]


# ---------------------------------------------------------------------------
# rocprofv3 databases -> summaries (no GPU needed)
# ---------------------------------------------------------------------------

def _pmc_per_dispatch(db, counter):
    """{kernel name: [value per dispatch]} of `counter` from a rocprofv3 counter database."""
    import sqlite3
    con = sqlite3.connect(db)
    per = {}
    for name, disp, val in con.execute(
            "select kernel_name, dispatch_id, sum(value) from counters_collection where counter_name = ? "
            "group by dispatch_id", (counter,)):
        per.setdefault(name, []).append(val)
    return per


def _steps(counts, hits):
    """Steps in a profiled run: every selection call certifies once (one
    k_certify dispatch for up to 65,535 sources); without it (the score
    bench) each step launches each matched kernel once.  A step may launch
    a kernel several times: one instantiation per group of sources (k_sweep
    with and without prefix sinks), or one launch per share of a rows source
    scored in two shares."""
    cert = match_kernel(counts.keys(), "k_certify")
    if cert:
        return counts[cert[0]]
    return max(counts[h] for h in hits)


def _one_kernel(per, base, db):
    """(names, per-step value, steps) of the dispatches of the kernels whose
    base name is `base`: the sum over the matched dispatches divided by the
    number of steps."""
    hits = match_kernel(per.keys(), base)
    if not hits:
        raise SystemExit(f"{db}: no kernel named {base!r} among {sorted(per)}")
    steps = _steps({k: len(v) for k, v in per.items()}, hits)
    return hits, sum(sum(per[h]) for h in hits) / steps, steps


def ingest_pmc(key, kernel, fetch_db, write_db, calib_fetch_db, calib_write_db, calib_bytes, commands):
    """Store `kernel`'s HBM traffic per step: FETCH_SIZE and WRITE_SIZE (KiB,
    summed over that kernel's dispatches of a step, every instantiation of it,
    mean over the steps), each scaled by bytes / counter of a plain device
    copy of known size."""
    knames, fetch, nf = _one_kernel(_pmc_per_dispatch(fetch_db, "FETCH_SIZE"), kernel, fetch_db)
    _, write, nw = _one_kernel(_pmc_per_dispatch(write_db, "WRITE_SIZE"), kernel, write_db)
    _, cf, _ = _one_kernel(_pmc_per_dispatch(calib_fetch_db, "FETCH_SIZE"), "__amd_rocclr_copyBuffer", calib_fetch_db)
    _, cw, _ = _one_kernel(_pmc_per_dispatch(calib_write_db, "WRITE_SIZE"), "__amd_rocclr_copyBuffer", calib_write_db)
    ff, fw = calib_bytes / (cf * 1024.0), calib_bytes / (cw * 1024.0)
    rec = {"workload": key, "kernels": knames, "kernel_base": kernel, "source_sha": kernel_source_sha(kernel),
           "sources": list(kernel_sources(kernel)),
           "steps": [nf, nw],
           "fetch_kib_per_step": fetch, "write_kib_per_step": write,
           "calib_copy_bytes": calib_bytes, "calib_fetch_kib": cf, "calib_write_kib": cw,
           "fetch_factor": ff, "write_factor": fw,
           "traffic_bytes_per_step": fetch * 1024.0 * ff + write * 1024.0 * fw,
           "commands": commands}
    with open(traffic_path(key), "w") as fh:
        json.dump(rec, fh, indent=1)
    print(json.dumps(rec), flush=True)


def _bench_line(path):
    lines = [l for l in open(path) if l.startswith('{"metric"')]
    return json.loads(lines[-1]) if lines else None


def trace_summary(db, title, command, kernel, bench_log=None, plain_log=None, plain_command=None):
    """Markdown summary of a rocprofv3 kernel trace: per-kernel statistics,
    then `kernel`'s own dispatches (matched by exact base name)."""
    import sqlite3
    con = sqlite3.connect(db)
    rows = list(con.execute("select name, count(*), sum(duration), avg(duration), min(duration), max(duration) "
                            "from kernels group by name order by sum(duration) desc"))
    tot = sum(r[2] for r in rows)
    out = [f"# {title}", "", "Command (on the MI355X machine; `<repo>` is the repository root):", "", "```", command, "```", "",
           "rocprofv3 kernel trace, per-kernel statistics (durations in microseconds):", "",
           "| kernel | calls | total us | avg us | min us | max us | % |", "|---|---|---|---|---|---|---|"]
    for n, c, s, a, mn, mx in rows:
        out.append(f"| `{n}` | {c} | {s / 1e3:.1f} | {a / 1e3:.2f} | {mn / 1e3:.2f} | {mx / 1e3:.2f} | "
                   f"{100 * s / tot:.1f} |")
    names = [r[0] for r in rows]
    hits = match_kernel(names, kernel)
    if not hits:
        raise SystemExit(f"no kernel named {kernel!r} in {names}")
    per = {h: [r[0] for r in con.execute("select duration from kernels where name = ? order by start", (h,))]
           for h in hits}
    steps = _steps({r[0]: r[1] for r in rows}, hits)
    step_us = sum(sum(v) for v in per.values()) / steps / 1e3
    desc = ", ".join(f"`{h}` ({len(v)} dispatches, average {sum(v) / len(v) / 1e3:.2f} us)" for h, v in per.items())
    out += ["", f"Dominant kernel `{kernel}`: {desc}; {steps} steps (calls), {step_us:.2f} us of `{kernel}` per "
                "step (trace average)."]
    if bench_log:
        d = _bench_line(bench_log)
        if d:
            r = d["roofline"]
            out += ["", "The same run's bench line (`kernel_ms` comes from the library's HIP events around the "
                        "scoring kernel on the call's stream, in the second, timed loop):", "", "```",
                    json.dumps(d), "```", "",
                    f"Key figures: {d['value']:.4g} plans/s, step {d['ms_per_step']:.4f} ms; `{kernel}` "
                    f"{r['kernel_ms'] * 1e3:.1f} us per step (events) -> roofline frac {r['frac']:.3f} "
                    f"({r['bound']})."]
            if r["bound"] in ("alu", "hbm") and "achieved_units_per_step" in r:
                fr = r["achieved_units_per_step"] / (step_us / 1e6) / (r["peak"] * r["peak_scale"])
                out.append(f"From the trace's per-step average instead: frac {fr:.3f}.")
    if plain_log:
        p = _bench_line(plain_log)
        if p:
            pr = p["roofline"]
            out += ["", f"The same command without the profiler (`{plain_command or ''}`), run just before on the "
                        f"same machine: {p['value']:.4g} plans/s, step {p['ms_per_step']:.4f} ms, `{kernel}` "
                        f"{pr['kernel_ms'] * 1e3:.1f} us per step (events) -> roofline frac {pr['frac']:.3f}. "
                        "Bench line:", "", "```", json.dumps(p), "```"]
    print("\n".join(out))


def pmc_summary(dbs, kernel, title, commands, trace_db=None):
    """Markdown summary of SQ counters of `kernel` (exact base name) from
    several rocprofv3 --pmc databases.  Rates use the kernel's average trace
    duration (from `trace_db`) times the 2.4 GHz clock as the denominator, so
    a rate cannot exceed what 256 CUs can issue in that time."""
    import sqlite3
    vals = {}
    for db in dbs:
        con = sqlite3.connect(db)
        names = [r[0] for r in con.execute("select distinct counter_name from counters_collection")]
        for cn in names:
            per = _pmc_per_dispatch(db, cn)
            knames, v, nsteps = _one_kernel(per, kernel, db)
            vals[cn] = (v, nsteps, knames)
    kn = ", ".join(f"`{k}`" for k in next(iter(vals.values()))[2])
    out = [f"# {title}", "", "Commands (on the MI355X machine; `<repo>` is the repository root), one counter pass each:", "",
           "```"] + commands + ["```", "",
                                f"Per-step values of `{kernel}` (summed over a step's dispatches of {kn}, "
                                "mean over the steps):", "",
                                "| counter | value per step | steps |", "|---|---|---|"]
    for cn in sorted(vals):
        out.append(f"| `{cn}` | {vals[cn][0]:.0f} | {vals[cn][1]} |")
    g = lambda c: vals[c][0] if c in vals else None
    out += ["", "Derived:", ""]
    if g("SQ_WAVES"):
        w = g("SQ_WAVES")
        for c, lab in (("SQ_INSTS_VALU", "VALU"), ("SQ_INSTS_SALU", "SALU"), ("SQ_INSTS_LDS", "LDS"),
                       ("SQ_INSTS_SMEM", "SMEM")):
            if g(c) is not None:
                out.append(f"- {lab} instructions per wave: {g(c) / w:.1f}")
    if trace_db:
        con = sqlite3.connect(trace_db)
        names = [r[0] for r in con.execute("select distinct name from kernels")]
        hits = match_kernel(names, kernel)
        per = {h: [r[0] for r in con.execute("select duration from kernels where name = ?", (h,))] for h in hits}
        counts = {r[0]: r[1] for r in con.execute("select name, count(*) from kernels group by name")}
        dur = sum(sum(v) for v in per.values()) / _steps(counts, hits) / 1e9
        cyc = dur * CLOCK_HZ
        out.append(f"- duration per step in the kernel trace: {dur * 1e6:.2f} us = {cyc:.0f} cycles at 2.4 GHz")
        if g("SQ_INSTS_VALU") is not None:
            out.append(f"- VALU issue: {g('SQ_INSTS_VALU') / (cyc * N_CU):.3f} wave-instructions per CU per cycle "
                       "(nominal rate 1: four SIMDs, each one 64-lane instruction per 4 cycles; readings at or "
                       "slightly above it, as some instruction forms issue faster, mean the VALU pipes are "
                       "saturated)")
        if g("SQ_WAVE_CYCLES") is not None:
            out.append(f"- mean resident waves per CU: {4 * g('SQ_WAVE_CYCLES') / (cyc * N_CU):.2f} of at most 32 "
                       "(SQ_WAVE_CYCLES counts quad-cycles: 4 SQ_WAVE_CYCLES / (duration x clock x CUs))")
        if g("SQ_ACTIVE_INST_LDS") is not None:
            out.append(f"- LDS issue: {g('SQ_ACTIVE_INST_LDS') / (cyc * N_CU):.3f} per CU per cycle")
    if g("SQ_LDS_BANK_CONFLICT") is not None and g("SQ_ACTIVE_INST_LDS"):
        out.append(f"- LDS bank-conflict cycles / LDS-active cycles: "
                   f"{g('SQ_LDS_BANK_CONFLICT') / g('SQ_ACTIVE_INST_LDS'):.3f}")
    print("\n".join(out))


# ---------------------------------------------------------------------------
# work counts
# ---------------------------------------------------------------------------

def edge_count(prob):
    return len({(int(u), int(v)) for u, v in prob.edges})


def sweep_work_per_plan(prob, ydiv=False):
    """Algorithmic fp32 operations per plan of the prefix-shared sweep.

    Per plan: 1 multiply (corr), 1 add (CP), 1 compare (prefilter); per row of
    the inner sweep (R_y plans): the add and multiply of node x and the max of
    y's predecessors; per block (R_x R_y plans): the prefix products and one
    max/add per prefix edge.  Counted like the full recurrence, operation by
    operation, so the figure never exceeds the work actually done.

    ydiv: the sweep compares x's product (the rest of a plan's corr) with
    thresholds divided ahead by each implementation of y's factor, so a plan
    costs 1 add (CP) and 1 selection operation (the min of its CP bin's
    threshold into its row's least threshold; the row's last one is the
    compare with x's product) and no multiply.  The bin's address (an AND of
    the CP's pattern) is addressing, not counted.
    """
    n = prob.n_nodes
    rx = int(prob.radix[n - 2]) if n >= 2 else 1
    ry = int(prob.radix[n - 1])
    edges = {(int(u), int(v)) for u, v in prob.edges}
    npre = max(n - 2, 0)
    pre_edges = sum(1 for u, v in edges if v < npre)
    x_pred = sum(1 for u, v in edges if v == n - 2)
    y_pred = sum(1 for u, v in edges if v == n - 1 and u != n - 2)
    per_plan = 2.0 if ydiv else 3.0
    per_row = 2.0 + (1.0 if (n - 2, n - 1) in edges and y_pred > 0 else 0.0)
    per_block = max(npre - 1, 0) + pre_edges + x_pred + y_pred
    return per_plan + per_row / ry + per_block / (rx * ry)


def obj_sweep_work_per_plan(prob, yshift=False):
    """Algorithmic fp32 operations per plan of the objective-mode sweep.

    Per plan: the add of y's duration (T), the max with the prefix sinks' path
    when there is one, the adds of y's utility (U) and d (D), the fused
    multiply-add G = U - lambda_l T and the prefilter compare; per row: the
    adds of node x (its path, utility and d) and the max of y's predecessors;
    per block: the prefix sums of u and d and one max/add per prefix edge.

    yshift: the sweep compares the row's R = ux - lambda_l M (one fused
    multiply-add per row) with bin thresholds lowered ahead by each
    implementation of y's utility and latency term, so a plan costs the add of
    its D and 1 selection operation (the min of its D bin's threshold into the
    row's least threshold; the row's last one is the compare with R).
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
    per_plan = 2.0 if yshift else 5.0 + (1.0 if has_s2 else 0.0)
    per_row = (4.0 if yshift else 3.0) + (1.0 if (n - 2, n - 1) in edges and y_pred > 0 else 0.0)
    per_block = 2 * max(npre - 1, 0) + pre_edges + x_pred + y_pred
    return per_plan + per_row / ry + per_block / (rx * ry)


def full_work_per_plan(prob, K):
    """The per-plan count of the full recurrence: (N-1) mul + E max/add + K compares."""
    return (prob.n_nodes - 1) + edge_count(prob) + K


# ---------------------------------------------------------------------------
# inputs
# ---------------------------------------------------------------------------

def make_workload(name, objective, pressure):
    """(problems, objectives or None, [(kind, problem, begin, count)], plans)."""
    from paper_2607_02942_amd import workload as wl
    if name == "batch6":
        probs = wl.batch6()
        specs = [("range", r, 0, 12 ** 6) for r in range(len(probs))]
    else:
        probs = [wl.by_name(name)]
        if name == "stream24":
            specs = [("rows", 0, 0, wl.STREAM_ROWS)]
        else:
            n = wl.LAYERED_RANGE if name == "layered10" else probs[0].n_plans()
            specs = [("range", 0, 0, n)]
    if pressure == "per-class":
        probs = [wl.per_class(p) for p in probs]
    objs = [wl.paper_objective(p) for p in probs] if objective else None
    return probs, objs, specs, sum(s[3] for s in specs)


def cpu_info():
    model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return model, os.cpu_count(), len(os.sched_getaffinity(0))


def cpu_baseline_child(args):
    """Time the fp64 oracle (single-threaded) on a bounded sample of the
    workload; runs in a child process pinned to one core, without the GPU."""
    from oracle import oracle as orc
    from paper_2607_02942_amd import workload as wl
    probs, objs, specs, _ = make_workload(args.workload, args.objective, args.pressure)
    t0 = time.perf_counter()
    if args.workload == "stream24":
        n = args.cpu_rows
        rows = wl.make_rows(n, 24, 36, threads=1)
        t0 = time.perf_counter()
        if objs:
            orc.obj_select_rows(probs[0], objs[0], rows, 0)
        else:
            orc.select_rows(probs[0], rows, 0)
        what = f"the first {n} rows of the 2^28"
    elif args.workload == "batch6":
        nreq = args.cpu_requests
        n = 0
        for r in range(nreq):
            cnt = specs[r][3]
            if objs:
                orc.obj_select_range(probs[r], objs[r], 0, cnt)
            else:
                orc.select_range(probs[r], 0, cnt)
            n += cnt
        what = f"the first {nreq} of the 4,096 requests, every plan of each ({n} plans)"
    else:
        n = min(args.cpu_sample, specs[0][3])
        if objs:
            orc.obj_select_range(probs[0], objs[0], 0, n)
        else:
            orc.select_range(probs[0], 0, n)
        what = f"plan indices [0, {n})"
    dt = time.perf_counter() - t0
    model, ncpu, naff = cpu_info()
    print(json.dumps({"value": n / dt, "unit": "plans/s", "cores": 1, "kind": "oracle",
                      "sample": f"{args.workload}: {what}; single-threaded fp64 oracle (gcc -O2 -ffp-contract=off), "
                                f"{dt:.1f} s",
                      "cpu_model": model, "nproc": ncpu, "pinned_core": sorted(os.sched_getaffinity(0))}),
          flush=True)


def run_cpu_baseline(args):
    """The oracle leg in a child process pinned with taskset to the last core
    this process may use (the GPU work has not started yet)."""
    core = sorted(os.sched_getaffinity(0))[-1]
    cmd = [sys.executable, os.path.abspath(__file__), "--cpu-baseline-child", "--workload", args.workload,
           "--pressure", args.pressure, "--cpu-sample", str(args.cpu_sample), "--cpu-rows", str(args.cpu_rows),
           "--cpu-requests", str(args.cpu_requests)] + (["--objective"] if args.objective else [])
    try:
        cmd = ["taskset", "-c", str(core)] + cmd
        res = subprocess.run(cmd, capture_output=True, text=True, timeout=600,
                             env=dict(os.environ, OMP_NUM_THREADS="1"))
    except (OSError, subprocess.TimeoutExpired) as e:
        return {"error": str(e)}
    lines = [l for l in res.stdout.splitlines() if l.startswith("{")]
    if res.returncode != 0 or not lines:
        return {"error": f"rc {res.returncode}: {res.stderr[-400:]}"}
    d = json.loads(lines[-1])
    d["pinning"] = f"taskset -c {core}"
    return d


def golden_check(name, mode_tag, got, n_levels):
    """Compare the choices with the oracle's stored full-size selections."""
    if mode_tag:
        path = os.path.join(GOLDEN_DIR, f"select_{name}_{mode_tag}.json")
    else:
        path = os.path.join(GOLDEN_DIR, f"select_{name}.json")
    if not os.path.exists(path):
        return "no stored selection for this mode", True
    g = json.load(open(path))
    want = g["choices"] if name == "batch6" else [g["choices"]]
    f32 = lambda x: float(np.float32(float(x)))
    bad = 0
    for r, (gs, ws) in enumerate(zip(got, want)):
        for k, w in enumerate(ws):
            c = gs[k]
            if (c[0], c[1]) != (int(w[0]), int(w[1])):
                bad += 1
            elif int(w[1]) and (c[2] != f32(w[2]) or c[3] != f32(w[3]) or c[4] != f32(w[4])):
                bad += 1
    rel = os.path.relpath(path, ROOT)
    if bad:
        return f"MISMATCH: {bad} (source, level) choices differ from {rel}", False
    return f"every choice equals {rel} ({sum(len(w) for w in want)} (source, level) pairs)", True


# ---------------------------------------------------------------------------
# GPU runs
# ---------------------------------------------------------------------------

def score_bench(args, torch, D, wl, stream, tkey):
    """Per-plan scores of a 2^26-plan range into device buffers: corr, CP at each
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
    kern = score_kernel(prob, args.pressure == "per-class")
    res = {"metric": "plans scored/sec by dy_plan_score on 1 MI355X (per-plan outputs)", "value": n / (ms / 1e3),
           "unit": "plans/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms,
           "higher_is_better": True, "dtype": "f32", "data": "synthetic",
           "config": {"workload": prob.name, "plans": n, "levels": K, "outputs": "corr, cp[K], demand, feas"},
           "roofline": {"bound": "hbm", "kernel": kern, "achieved": achieved / 1e9, "peak": PEAK_HBM / 1e9,
                        "unit": "GB/s", "frac": achieved / PEAK_HBM, "per_unit": f"{per_plan:.0f} B written per plan",
                        "traffic": stored_traffic(tkey, kern), "kernel_ms": ms,
                        "achieved_units_per_step": n * per_plan, "peak_scale": 1e9}}
    print(json.dumps(res), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="batch6", choices=WORKLOADS)
    ap.add_argument("--objective", action="store_true",
                    help="the paper's additive objective J_L (levels 0, 1.5, 3) instead of corr / SLO")
    ap.add_argument("--pressure", choices=["level", "per-class"], default="level",
                    help="per-class: the second backend pressed at half the level's rho (per-backend pressure)")
    ap.add_argument("--score", action="store_true",
                    help="time dy_plan_score (per-plan corr, CP per level, demand, feasibility bits) instead")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample", type=int, default=1 << 26, help="oracle plans timed (range workloads)")
    ap.add_argument("--cpu-rows", type=int, default=1 << 24, help="oracle rows timed (stream24)")
    ap.add_argument("--cpu-requests", type=int, default=64, help="oracle requests timed (batch6)")
    ap.add_argument("--cpu-baseline-child", action="store_true", help=argparse.SUPPRESS)
    ap.add_argument("--sample-stride", type=int, default=0)
    ap.add_argument("--calib-copy", type=int, default=0, help="MiB: run one device copy (counter calibration)")
    ap.add_argument("--ingest-pmc", nargs=4, metavar=("FETCH_DB", "WRITE_DB", "CALIB_FETCH_DB", "CALIB_WRITE_DB"),
                    help="store a kernel's traffic from rocprofv3 --pmc databases (no GPU needed)")
    ap.add_argument("--kernel", help="kernel base name for --ingest-pmc / --trace-summary / --pmc-summary")
    ap.add_argument("--calib-bytes", type=int, default=1 << 30)
    ap.add_argument("--pmc-command", action="append", default=[], help="command that produced a database")
    ap.add_argument("--trace-summary", metavar="DB", help="markdown summary of a rocprofv3 kernel trace")
    ap.add_argument("--pmc-summary", nargs="+", metavar="DB", help="markdown summary of rocprofv3 --pmc databases")
    ap.add_argument("--trace-db", help="kernel trace giving durations for --pmc-summary")
    ap.add_argument("--title", default="")
    ap.add_argument("--command", default="")
    ap.add_argument("--bench-log", help="log holding the profiled run's bench line")
    ap.add_argument("--plain-log", help="log holding the same command's bench line without the profiler")
    ap.add_argument("--plain-command", default="")
    args = ap.parse_args()
    tkey = args.workload + ("_obj" if args.objective else "") + ("_perclass" if args.pressure == "per-class" else "")
    if args.score:
        tkey = args.workload + ("_perclass" if args.pressure == "per-class" else "") + "_score"
    if args.ingest_pmc:
        ingest_pmc(tkey, args.kernel, *args.ingest_pmc, args.calib_bytes, args.pmc_command)
        return
    if args.trace_summary:
        trace_summary(args.trace_summary, args.title, args.command, args.kernel, args.bench_log, args.plain_log,
                      args.plain_command)
        return
    if args.pmc_summary:
        pmc_summary(args.pmc_summary, args.kernel, args.title, args.pmc_command, args.trace_db)
        return
    if args.cpu_baseline_child:
        cpu_baseline_child(args)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(the work would shard by plan range, request or row range, one shard per GPU)", file=sys.stderr)
        sys.exit(2)

    cpu = None
    if not args.no_cpu_baseline and not args.score and not args.calib_copy:
        print("[bench] cpu baseline (oracle, one pinned core)", file=sys.stderr, flush=True)
        cpu = run_cpu_baseline(args)

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
    probs, objs, specs, plans = make_workload(name, args.objective, args.pressure)
    rows_dev = None
    sources = []
    for kind, p, b, c in specs:
        if kind == "rows":
            rows_host = wl.make_rows(c, probs[p].n_nodes, int(probs[p].radix[0]))
            rows_dev = torch.from_numpy(rows_host).cuda()
            del rows_host
            sources.append(D.rows_source(p, rows_dev, c, probs[p].n_nodes, 0))
        else:
            sources.append(D.range_source(p, b, c))
    prob = probs[0]
    K = objs[0].n_levels if objs else prob.n_levels
    if not objs:
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
        cands, main_ms, gen, ydiv = [], [], [], []
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
                ydiv.append(s.ydiv_jobs)
            if i == 0 or (i + 1) % max(1, args.steps // 4) == 0:
                print(f"[bench] {tag} step {i + 1}/{args.steps}", file=sys.stderr, flush=True)
        ev1.record(stream)
        torch.cuda.synchronize()
        return ev0.elapsed_time(ev1) / args.steps, main_ms, cands, gen, ydiv

    # 1) the steps as a caller runs them: repeated calls replay one HIP graph
    for _ in range(args.warmup):
        step()
    ms_per_step, _, _, _, _ = timed_loop("step", False)
    value = plans / (ms_per_step / 1e3)
    got_graph = [[out[j * plan.kmax + k].as_tuple() for k in range(K)] for j in range(len(sources))]
    # 2) the same calls with the library's HIP events around the scoring kernel
    #    (on the call's stream; timed calls launch directly, not from a graph)
    plan.set_option(D.DY_OPT_TIMING, 1)
    for _ in range(max(1, args.warmup // 2)):
        step()
    ms_per_step_timed, main_ms, cands, gen, ydiv = timed_loop("timed", True)
    got_timed = [[out[j * plan.kmax + k].as_tuple() for k in range(K)] for j in range(len(sources))]
    generated = bool(gen) and max(gen) > 0  # the library ran a kernel generated for the problem
    kern_ms = float(np.mean(main_ms))

    if name == "stream24":
        kbase = "dy_rows_scan_a"
        units = plans * 24.0
        achieved = units / (kern_ms / 1e3)
        roof = {"bound": "hbm", "kernel": kbase + " (rows, generated for the DAG" + (", objective)" if objs else ")"),
                "achieved": achieved / 1e9, "peak": PEAK_HBM / 1e9, "unit": "GB/s", "frac": achieved / PEAK_HBM,
                "traffic": stored_traffic(tkey, kbase), "per_unit": "24 B of row per plan", "kernel_ms": kern_ms,
                "achieved_units_per_step": units, "peak_scale": 1e9}
    else:
        # sources whose sweep took the pre-divided thresholds (every one or none
        # in these workloads: one DAG, or requests of one shape)
        yd = max(ydiv) if ydiv else 0
        if yd not in (0, len(sources)):
            raise RuntimeError(f"{yd} of {len(sources)} sources took the pre-divided thresholds")
        if objs:
            units = sum(obj_sweep_work_per_plan(probs[p], yd > 0) * c for _, p, _, c in specs)
        else:
            units = sum(sweep_work_per_plan(probs[p], yd > 0) * c for _, p, _, c in specs)
        f = units / plans
        achieved = units / (kern_ms / 1e3)
        if generated:
            kbase = "dy_sweep"
            kname = "dy_sweep (generated for the DAG" + (", objective)" if objs else ")")
        else:
            kbase = "k_sweep_obj" if objs else "k_sweep"
            kname = kbase
        roof = {"bound": "alu", "kernel": kname, "achieved": achieved / 1e12,
                "peak": PEAK_VALU / 1e12, "unit": "TFLOP/s", "frac": achieved / PEAK_VALU,
                "peak_packed_fp32": PEAK_VALU_PACKED / 1e12, "frac_vs_packed_fp32": achieved / PEAK_VALU_PACKED,
                "traffic": stored_traffic(tkey, kbase),
                "per_unit": f"{f:.4f} fp32 ops per plan (prefix-shared sweep{', objective' if objs else ''}"
                            + ((", thresholds lowered ahead by y's terms" if objs else
                                ", thresholds divided ahead by y's factor") if yd else "")
                            + (", mean over the requests' DAGs" if len(specs) > 1 else "") + ")",
                "kernel_ms": kern_ms, "achieved_units_per_step": units, "peak_scale": 1e12}
        if not objs:
            roof["full_recurrence_ops_per_plan"] = sum(full_work_per_plan(probs[p], K) * c
                                                       for _, p, _, c in specs) / plans
    mode_tag = "_".join(t for t in (("objective" if objs else ""), ("perclass" if args.pressure == "per-class"
                                                                     else "")) if t)
    check, ok = golden_check(name, mode_tag, got_timed, K)
    same = lambda a, b: all(x == y or (x != x and y != y) for ra, rb in zip(a, b) for ca, cb in zip(ra, rb)
                            for x, y in zip(ca, cb))
    if not same(got_graph, got_timed):
        check, ok = "MISMATCH: the graph-replayed and the direct calls chose differently", False

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
        "candidates_min_max": [int(min(cands)), int(max(cands))],
        "golden_check": check,
    }
    if name == "batch6":
        res["config"]["edges"] = "per request (random DAG, p = 0.35)"
    if cpu is not None:
        res["cpu_baseline"] = cpu
    plan.close()
    print(json.dumps(res), flush=True)
    if not ok:
        sys.exit(3)


if __name__ == "__main__":
    main()
