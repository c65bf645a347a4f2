"""Write the stored workload SLOs and full-size expected selections.

The SLO table goes beside the generator (paper_2607_02942_amd/workload_slo.json,
a workload parameter); the expected selections go to tests/golden/.

TEST INFRASTRUCTURE ONLY.  Every stored number is produced here by the fp64
oracle (oracle.c) on inputs from the seeded workload generator; nothing comes
from the GPU library.

  SLO = 1.5 x the exact lower median (0-based rank floor((n-1)/2)) of the
        unpressured critical path over the workload's scored plan set,
        computed in fp64 and rounded to the nearest fp32.
  select_<workload>.json = the oracle's per-level winners over the full
        plan set, computed as independent single-threaded chunks merged by
        the exact rule (greatest correctness, then lowest index).

Usage:  python -m oracle.golden [--procs P] [--only name,...] [--skip-select]
                                [--mode level|perclass|objective]
"""
from __future__ import annotations

import argparse
import json
import multiprocessing as mp
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from oracle import oracle as orc  # noqa: E402
from paper_2607_02942_amd import workload as wl  # noqa: E402

GOLDEN_DIR = os.path.join(ROOT, "tests", "golden")
HIST_BITS = 24

# workload -> (source kind, plan count)
SOURCES = {
    "chain4": ("range", 12 ** 4),
    "forkjoin8": ("range", 12 ** 8),
    "layered10": ("range", wl.LAYERED_RANGE),
    "stream24": ("rows", wl.STREAM_ROWS),
}


def _problem(name, r=None):
    if name == "batch6":
        return wl.batch6_request(r, slo=0.0)
    return {"chain4": wl.chain4, "forkjoin8": wl.forkjoin8, "layered10": wl.layered10,
            "stream24": wl.stream24}[name](slo=0.0)


def _rows(prob, begin, count):
    return wl.make_rows(count, prob.n_nodes, int(prob.radix[0]), row_begin=begin, threads=1)


def _chunks(total, size):
    return [(b, min(size, total - b)) for b in range(0, total, size)]


# ---- median ------------------------------------------------------------------
#
# The lower median of ~1e10 values does not fit in memory, so it is found in
# two passes over the plan set: a histogram of the top HIST_BITS bits of each
# fp64 value's bit pattern (non-negative doubles order like their patterns),
# then the values of the one bucket that holds the wanted rank, sorted.

def _hist_task(args):
    prob, kind, begin, count, bits = args
    op = orc.OracleProblem(prob, 0.0)
    hist = np.zeros(1 << bits, np.uint64)
    if kind == "rows":
        rows = _rows(prob, begin, count)
        orc.lib().or_cp0_hist(op.ref, 1, rows.ctypes.data, rows.shape[1], 0, count, bits, hist.ctypes.data)
    else:
        orc.lib().or_cp0_hist(op.ref, 0, None, 0, begin, count, bits, hist.ctypes.data)
    nz = np.nonzero(hist)[0]
    return nz, hist[nz]


def _collect_task(args):
    prob, kind, begin, count, bits, bucket, cap = args
    op = orc.OracleProblem(prob, 0.0)
    out = np.zeros(cap, np.float64)
    if kind == "rows":
        rows = _rows(prob, begin, count)
        got = orc.lib().or_cp0_collect(op.ref, 1, rows.ctypes.data, rows.shape[1], 0, count, bits,
                                       bucket, out.ctypes.data, cap)
    else:
        got = orc.lib().or_cp0_collect(op.ref, 0, None, 0, begin, count, bits, bucket, out.ctypes.data, cap)
    assert got <= cap, "bucket larger than the collection buffer"
    return out[:got]


class SerialPool:
    """The two pool methods lower_median_cp0 uses, run in this process."""

    def imap_unordered(self, fn, tasks, chunksize=1):
        return map(fn, tasks)

    def imap(self, fn, tasks, chunksize=1):
        return map(fn, tasks)


def lower_median_cp0(prob, kind, total, pool, chunk, bits=HIST_BITS):
    """Lower median (0-based rank floor((total-1)/2)) of the fp64 unpressured
    CP over plan indices [0, total) (kind "range") or the first `total` rows
    of the workload's row stream (kind "rows")."""
    tasks = [(prob, kind, b, c, bits) for b, c in _chunks(total, chunk)]
    hist = np.zeros(1 << bits, np.uint64)
    for nz, v in pool.imap_unordered(_hist_task, tasks):
        hist[nz] += v
    rank = (total - 1) // 2
    cum = np.cumsum(hist)
    bucket = int(np.searchsorted(cum, rank + 1))
    below = int(cum[bucket - 1]) if bucket > 0 else 0
    cap = int(hist[bucket])
    vals = np.concatenate(list(pool.imap(_collect_task, [t + (bucket, cap) for t in tasks])))
    assert vals.size == cap
    vals.sort()
    return float(vals[rank - below])


def _batch_slo_task(r):
    prob = _problem("batch6", r)
    vals = orc.cp0_values(prob, 0, prob.n_plans())
    rank = (vals.size - 1) // 2
    med = np.partition(vals, rank)[rank]
    return r, float(np.float32(1.5 * med))


# ---- selection -----------------------------------------------------------------
#
# mode "level": the recipes' pressure (every backend at the level's rho);
# "perclass": workload.per_class (the second backend at half the level's rho),
# the same SLO; "objective": the paper's additive objective J_L
# (workload.paper_objective), every plan admissible.

def _moded(prob, mode):
    if mode == "perclass":
        return wl.per_class(prob), None
    if mode == "objective":
        return prob, wl.paper_objective(prob)
    return prob, None


def _select_part(prob, obj, kind, begin, count, slo):
    if kind == "rows":
        rows = _rows(prob, begin, count)
        if obj is not None:
            return orc.obj_select_rows(prob, obj, rows, begin)
        return orc.select_rows(prob, rows, begin, slo=slo)
    if obj is not None:
        return orc.obj_select_range(prob, obj, begin, count)
    return orc.select_range(prob, begin, count, slo=slo)


def _select_task(args):
    name, kind, begin, count, slo, mode = args
    prob, obj = _moded(_problem(name), mode)
    return begin, _select_part(prob, obj, kind, begin, count, slo)


def full_select(name, slo, pool, chunk, mode="level"):
    kind, total = SOURCES[name]
    tasks = [(name, kind, b, c, slo, mode) for b, c in _chunks(total, chunk)]
    parts = sorted(pool.imap_unordered(_select_task, tasks))
    return orc.merge_choices([p for _, p in parts])


def _batch_select_task(args):
    r, slo, mode = args
    prob, obj = _moded(_problem("batch6", r), mode)
    return r, _select_part(prob, obj, "range", 0, prob.n_plans(), slo)


def _fmt_choices(ch):
    return [[int(c[0]), int(c[1]), repr(float(c[2])), repr(float(c[3])), repr(float(c[4]))] for c in ch]


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--procs", type=int, default=os.cpu_count() or 1)
    ap.add_argument("--only", default="chain4,forkjoin8,batch6,layered10,stream24")
    ap.add_argument("--skip-select", action="store_true")
    ap.add_argument("--mode", choices=["level", "perclass", "objective"], default="level",
                    help="selections under per-class pressure or the paper's objective (the stored SLOs are kept)")
    args = ap.parse_args()
    names = args.only.split(",")
    os.makedirs(GOLDEN_DIR, exist_ok=True)
    slo_path = wl.SLO_FILE
    slos = json.load(open(slo_path)) if os.path.exists(slo_path) else {}
    chunk = {"chain4": 1 << 20, "forkjoin8": 1 << 22, "layered10": 1 << 24, "stream24": 1 << 22}
    ctx = mp.get_context("fork")
    with ctx.Pool(args.procs) as pool:
        for name in names:
            t0 = time.time()
            if args.mode != "level":
                pass
            elif name == "batch6":
                res = sorted(pool.imap_unordered(_batch_slo_task, range(wl.N_BATCH), chunksize=8))
                slos["batch6"] = [s for _, s in res]
            else:
                kind, total = SOURCES[name]
                med = lower_median_cp0(_problem(name), kind, total, pool, chunk[name])
                slos[name] = float(np.float32(1.5 * med))
            if args.mode == "level":
                json.dump(slos, open(slo_path, "w"), indent=1)
                print(f"[golden] slo {name}: {slos[name] if name != 'batch6' else '4096 values'} "
                      f"({time.time() - t0:.1f}s)", flush=True)
            if args.skip_select:
                continue
            t0 = time.time()
            out = {"workload": name, "generator": "paper_2607_02942_amd.workload",
                   "oracle": "oracle/objective.c" if args.mode == "objective" else "oracle/oracle.c"}
            if args.mode != "level":
                out["mode"] = {"perclass": "workload.per_class: backend 1 at half the level's rho",
                               "objective": "workload.paper_objective: J_L, L in {0, 1.5, 3}"}[args.mode]
            if name == "batch6":
                res = sorted(pool.imap_unordered(_batch_select_task,
                                                 [(r, slos["batch6"][r], args.mode) for r in range(wl.N_BATCH)],
                                                 chunksize=8))
                out["source"] = {"kind": "range", "begin": 0, "count": 12 ** 6, "requests": wl.N_BATCH}
                out["choices"] = [_fmt_choices(ch) for _, ch in res]
            else:
                kind, total = SOURCES[name]
                out["source"] = {"kind": kind, "begin": 0, "count": total}
                out["slo"] = slos[name]
                out["choices"] = _fmt_choices(full_select(name, slos[name], pool, chunk[name], args.mode))
            tag = "" if args.mode == "level" else "_" + args.mode
            path = os.path.join(GOLDEN_DIR, f"select_{name}{tag}.json")
            with open(path, "w") as f:
                if name == "batch6":
                    f.write("{\n")
                    for key in [k for k in ("workload", "generator", "oracle", "mode", "source") if k in out]:
                        f.write(f" {json.dumps(key)}: {json.dumps(out[key])},\n")
                    f.write(' "choices": [\n')
                    f.write(",\n".join(json.dumps(c, separators=(",", ":")) for c in out["choices"]))
                    f.write("\n ]\n}\n")
                else:
                    json.dump(out, f, indent=1)
            print(f"[golden] select {name} ({time.time() - t0:.1f}s)", flush=True)


if __name__ == "__main__":
    main()
