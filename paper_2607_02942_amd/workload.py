"""Seeded synthetic planning workloads shaped like the paper's agentic workflows.

This module only *generates inputs*: workflow DAGs, per-implementation profile
tables (success probability, nominal duration, model-size factor, backend),
per-node vulnerability, pressure levels and, for the streamed workload, rows of
candidate implementation ids.  It holds none of the scoring or selection
arithmetic, so both the product path and the CPU oracle can consume its output.

Problem structure follows the paper's statement: a materialised DAG whose LLM
nodes each pick a (model x verification policy x backend) implementation
(Sec. 3.1, eq. physical-plan), a backend-independent quality profile
(Sec. 4.1), a nominal service time per implementation (Sec. 4.2, eq. tau),
a per-node vulnerability (Sec. 4.3) and a bounded set of pressure levels
(Sec. 4.4).  The concrete distributions are the five workload recipes:

  chain4   4-node chain, 12 impls (3 models x {none, verify} x 2 backends),
           levels {0, .3, .6, .85}, seed 0
  forkjoin8  1 -> 3 branches of 2 nodes -> 1 join, 12 impls, 8 levels on
           [0, .9], seed 1
  batch6   4096 requests, each a random 6-node DAG (edge prob .35), 12 impls,
           levels as chain4, seed 2 + request id
  layered10  layers 1-3-3-2-1 fully connected between adjacent layers,
           36 impls (6 models x {none, self, cross} x 2 backends),
           16 levels on [0, .95], seed 3, plan range [0, 2^32)
  stream24 random 24-node DAG (edge prob .15), 36 impls, 8 levels on
           [0, .95], 2^28 rows of uniform ids, seed 4

Random numbers are SplitMix64 outputs (Steele, Lea & Flood, OOPSLA 2014) used
as a counter-based generator: draw(key, c) is output number c+1 of a
SplitMix64 stream seeded with `key`.  U[0,1) = (x >> 11) * 2^-53, normals by
Box-Muller, row ids by (x_hi32 * R) >> 32.
"""
from __future__ import annotations

import ctypes
import dataclasses
import json
import os
from typing import Optional

import numpy as np

GOLDEN_GAMMA = np.uint64(0x9E3779B97F4A7C15)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)

# stream tags
TAG_DAG = 1
TAG_W = 2
TAG_LAT = 3
TAG_P = 4
TAG_GAIN = 5
TAG_PHI = 6
TAG_ROWS = 7

SIZES_3 = (1.0, 2.5, 6.0)
SIZES_6 = (0.5, 1.0, 2.0, 4.0, 8.0, 16.0)
# verification latency factor ranges per policy (index 0 = no verification)
PHI_2 = ((1.0, 1.0), (1.3, 2.0))
PHI_3 = ((1.0, 1.0), (1.3, 2.0), (1.8, 3.0))

WORKLOADS = ("chain4", "forkjoin8", "batch6", "layered10", "stream24")
N_BATCH = 4096
STREAM_ROWS = 1 << 28
LAYERED_RANGE = 1 << 32

_HERE = os.path.dirname(os.path.abspath(__file__))
# Stored SLOs of the five workloads (1.5 x the lower median of the unpressured
# critical path over the scored plan set, a workload parameter that needs
# ~1e10 fp64 evaluations for the largest sets), written by oracle/golden.py.
SLO_FILE = os.path.join(_HERE, "workload_slo.json")


def _mix(z: np.ndarray) -> np.ndarray:
    z = (z ^ (z >> np.uint64(30))) * _M1
    z = (z ^ (z >> np.uint64(27))) * _M2
    return z ^ (z >> np.uint64(31))


def draw(key: int, ctr) -> np.ndarray:
    """Counter-based SplitMix64: output number ctr+1 of the stream seeded with key."""
    c = np.asarray(ctr, dtype=np.uint64)
    with np.errstate(over="ignore"):
        return _mix(np.uint64(key) + (c + np.uint64(1)) * GOLDEN_GAMMA)


def stream_key(cfg: int, seed: int, tag: int) -> int:
    assert 0 <= cfg < (1 << 16) and 0 <= seed < (1 << 32) and 0 <= tag < (1 << 16)
    return int(draw(0, (cfg << 48) ^ (seed << 16) ^ tag))


def u01(x: np.ndarray) -> np.ndarray:
    return (x >> np.uint64(11)).astype(np.float64) * (2.0 ** -53)


def _pair_ctr(a, b):
    return (np.asarray(a, dtype=np.uint64) << np.uint64(32)) | np.asarray(b, dtype=np.uint64)


# ----------------------------------------------------------------------------
# DAG shapes (nodes numbered in a topological order: every edge is u < v)
# ----------------------------------------------------------------------------

def dag_chain(n: int) -> np.ndarray:
    return np.array([[i, i + 1] for i in range(n - 1)], dtype=np.int32).reshape(-1, 2)


def dag_forkjoin(branches: int = 3, depth: int = 2) -> np.ndarray:
    """Source 0 -> `branches` parallel chains of `depth` nodes -> join.

    Nodes are numbered layer by layer: branch b occupies 1+b, 1+branches+b, ...
    """
    e = []
    for b in range(branches):
        e.append((0, 1 + b))
        for d in range(depth - 1):
            e.append((1 + d * branches + b, 1 + (d + 1) * branches + b))
    join = 1 + depth * branches
    for b in range(branches):
        e.append((1 + (depth - 1) * branches + b, join))
    return np.array(sorted(e), dtype=np.int32)


def dag_layered(widths) -> np.ndarray:
    e = []
    start = 0
    layers = []
    for wd in widths:
        layers.append(list(range(start, start + wd)))
        start += wd
    for la, lb in zip(layers[:-1], layers[1:]):
        for u in la:
            for v in lb:
                e.append((u, v))
    return np.array(e, dtype=np.int32)


def dag_random(n: int, edge_p: float, key: int) -> np.ndarray:
    """Edges i<j drawn with probability edge_p in (i, j) lexicographic order, then
    0 -> j for every j without a predecessor and i -> n-1 for every i without a
    successor, which leaves a single source (0) and a single sink (n-1)."""
    edges = set()
    for i in range(n):
        for j in range(i + 1, n):
            if u01(draw(key, _pair_ctr(i, j)))[()] < edge_p:
                edges.add((i, j))
    for j in range(1, n):
        if not any(v == j for (_, v) in edges):
            edges.add((0, j))
    for i in range(n - 1):
        if not any(u == i for (u, _) in edges):
            edges.add((i, n - 1))
    return np.array(sorted(edges), dtype=np.int32).reshape(-1, 2)


# ----------------------------------------------------------------------------
# Problem container
# ----------------------------------------------------------------------------

@dataclasses.dataclass
class Problem:
    """One planning problem in the layout the C-ABI and the oracle both take.

    Tables are row-major [n_nodes][max_radix]; entry (n, i) describes
    implementation i of node n; entries with i >= radix[n] are padding.
    """
    n_nodes: int
    edges: np.ndarray      # int32 [E, 2], u < v
    radix: np.ndarray      # int32 [N]
    p: np.ndarray          # float32 [N, R] success probability
    tau: np.ndarray        # float32 [N, R] nominal duration
    size: np.ndarray       # float32 [N, R] model-size factor
    backend: np.ndarray    # int32   [N, R] backend id
    w: np.ndarray          # float32 [N] vulnerability
    rho: np.ndarray        # float32 [K, B] pressure per level and backend
    slo: float = float("nan")
    name: str = ""

    @property
    def max_radix(self) -> int:
        return int(self.p.shape[1])

    @property
    def n_levels(self) -> int:
        return int(self.rho.shape[0])

    @property
    def n_backends(self) -> int:
        return int(self.rho.shape[1])

    @property
    def n_edges(self) -> int:
        return int(self.edges.shape[0])

    def n_plans(self) -> int:
        return int(np.prod(self.radix.astype(object)))

    def copy(self) -> "Problem":
        return dataclasses.replace(
            self, edges=self.edges.copy(), radix=self.radix.copy(), p=self.p.copy(),
            tau=self.tau.copy(), size=self.size.copy(), backend=self.backend.copy(),
            w=self.w.copy(), rho=self.rho.copy())


@dataclasses.dataclass
class Objective:
    """The paper's additive objective J_L (Sec. 4.3 eq. admission-objective,
    Sec. 4.4 eq. variant-objective) for a Problem: quality q = Problem.p,
    vulnerability v = Problem.w, nominal durations Problem.tau.

    cost: float32 [N, R] call cost c_{n,i}; is_tool: int32 [N] (1 = tool node:
    no quality or cost term, not in D_tau, duration kept in T) or None;
    levels: float32 [K] the specialisation levels L_k.
    """
    cost: np.ndarray
    levels: np.ndarray
    lambda_f: float = 1.0
    lambda_c: float = 0.01
    lambda_l: float = 0.05
    lambda_ld: float = 0.05
    beta: float = 1.0
    effort: float = 0.5
    is_tool: Optional[np.ndarray] = None

    @property
    def n_levels(self) -> int:
        return int(self.levels.shape[0])


PAPER_LEVELS = (0.0, 1.5, 3.0)  # L in {0, 1.5, 3} (balanced trace, Sec. 7)


def paper_objective(prob: Problem, levels=PAPER_LEVELS, **weights) -> Objective:
    """Objective for `prob` with call cost c = tau * size (duration times model
    size, computed in fp32) and the given levels and weights."""
    cost = (prob.tau.astype(np.float32) * prob.size.astype(np.float32)).astype(np.float32)
    return Objective(cost=cost, levels=np.asarray(levels, np.float32), **weights)


def levels(k: int, lo: float, hi: float) -> np.ndarray:
    """k pressure levels evenly spaced on [lo, hi], endpoints included."""
    if k == 1:
        return np.array([lo], dtype=np.float64)
    return np.array([lo + (hi - lo) * i / (k - 1) for i in range(k)], dtype=np.float64)


def make_tables(cfg: int, seed: int, n: int, sizes, phis, n_backends: int):
    """Profile tables for every node of one problem.

    impl id = (m * V + v) * B + b  (model-major, backend-minor).
    p for an unverified impl is drawn per (node, model, backend) from U[0.6, 0.95];
    a verified impl raises that p to p + (1 - p) * U[0.3, 0.7] with its own draw.
    tau = l_n * size_m * phi, l_n ~ LogNormal(0, 0.5) per node, phi = 1 for no
    verification and U[lo_v, hi_v] drawn per verified impl.
    """
    n_models, n_pol, B = len(sizes), len(phis), n_backends
    R = n_models * n_pol * B
    kw = stream_key(cfg, seed, TAG_W)
    kl = stream_key(cfg, seed, TAG_LAT)
    kp = stream_key(cfg, seed, TAG_P)
    kg = stream_key(cfg, seed, TAG_GAIN)
    kf = stream_key(cfg, seed, TAG_PHI)
    nodes = np.arange(n)
    w = u01(draw(kw, nodes))
    u1 = 1.0 - u01(draw(kl, 2 * nodes))          # (0, 1]
    u2 = u01(draw(kl, 2 * nodes + 1))
    z = np.sqrt(-2.0 * np.log(u1)) * np.cos(2.0 * np.pi * u2)
    lat = np.exp(0.0 + 0.5 * z)
    p = np.zeros((n, R), np.float64)
    tau = np.zeros((n, R), np.float64)
    size = np.zeros((n, R), np.float64)
    backend = np.zeros((n, R), np.int32)
    for m in range(n_models):
        for v in range(n_pol):
            for b in range(B):
                i = (m * n_pol + v) * B + b
                base_id = (m * n_pol + 0) * B + b
                pb = 0.6 + 0.35 * u01(draw(kp, _pair_ctr(nodes, base_id)))
                if v == 0:
                    p[:, i] = pb
                    phi = np.ones(n)
                else:
                    gain = 0.3 + 0.4 * u01(draw(kg, _pair_ctr(nodes, i)))
                    p[:, i] = pb + (1.0 - pb) * gain
                    lo, hi = phis[v]
                    phi = lo + (hi - lo) * u01(draw(kf, _pair_ctr(nodes, i)))
                tau[:, i] = lat * sizes[m] * phi
                size[:, i] = sizes[m]
                backend[:, i] = b
    return (p.astype(np.float32), tau.astype(np.float32), size.astype(np.float32),
            backend, w.astype(np.float32))


def _slo_table() -> dict:
    if not os.path.exists(SLO_FILE):
        return {}
    with open(SLO_FILE) as f:
        return json.load(f)


def _with_slo(prob: Problem, key: str, slo: Optional[float]) -> Problem:
    if slo is not None:
        prob.slo = float(np.float32(slo))
        return prob
    t = _slo_table()
    if key in t:
        prob.slo = float(np.float32(t[key]))
    return prob


def _build(cfg, seed, edges, n, sizes, phis, lv, name, B=2):
    p, tau, size, backend, w = make_tables(cfg, seed, n, sizes, phis, B)
    R = p.shape[1]
    rho = np.repeat(lv[:, None], B, axis=1).astype(np.float32)
    return Problem(n_nodes=n, edges=np.ascontiguousarray(edges, np.int32),
                   radix=np.full(n, R, np.int32), p=p, tau=tau, size=size,
                   backend=backend, w=w, rho=rho, name=name)


def chain4(slo: Optional[float] = None) -> Problem:
    prob = _build(0, 0, dag_chain(4), 4, SIZES_3, PHI_2, np.array([0.0, 0.3, 0.6, 0.85]), "chain4")
    return _with_slo(prob, "chain4", slo)


def forkjoin8(slo: Optional[float] = None) -> Problem:
    prob = _build(1, 1, dag_forkjoin(3, 2), 8, SIZES_3, PHI_2, levels(8, 0.0, 0.9), "forkjoin8")
    return _with_slo(prob, "forkjoin8", slo)


def batch6_request(r: int, slo: Optional[float] = None) -> Problem:
    seed = 2 + r
    edges = dag_random(6, 0.35, stream_key(2, seed, TAG_DAG))
    prob = _build(2, seed, edges, 6, SIZES_3, PHI_2, np.array([0.0, 0.3, 0.6, 0.85]), f"batch6[{r}]")
    if slo is None:
        t = _slo_table().get("batch6")
        if t is not None and r < len(t):
            slo = t[r]
    return _with_slo(prob, f"batch6[{r}]", slo)


def batch6(n_requests: int = N_BATCH):
    t = _slo_table().get("batch6")
    out = []
    for r in range(n_requests):
        s = t[r] if (t is not None and r < len(t)) else None
        out.append(batch6_request(r, s))
    return out


def layered10(slo: Optional[float] = None) -> Problem:
    prob = _build(3, 3, dag_layered((1, 3, 3, 2, 1)), 10, SIZES_6, PHI_3, levels(16, 0.0, 0.95), "layered10")
    return _with_slo(prob, "layered10", slo)


def stream24(slo: Optional[float] = None) -> Problem:
    edges = dag_random(24, 0.15, stream_key(4, 4, TAG_DAG))
    prob = _build(4, 4, edges, 24, SIZES_6, PHI_3, levels(8, 0.0, 0.95), "stream24")
    return _with_slo(prob, "stream24", slo)


# ----------------------------------------------------------------------------
# Candidate rows (uint8 implementation ids), generated natively
# ----------------------------------------------------------------------------

_rows_lib = None


def _load_rows_lib():
    global _rows_lib
    if _rows_lib is None:
        path = os.path.join(_HERE, "libdyworkload.so")
        if not os.path.exists(path):
            raise RuntimeError(f"{path} is not built; run __graft_entry__.build()")
        lib = ctypes.CDLL(path)
        lib.dw_rows.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_uint64,
                                ctypes.c_int32, ctypes.c_int32, ctypes.c_uint64,
                                ctypes.c_void_p, ctypes.c_int32]
        lib.dw_rows.restype = ctypes.c_int32
        lib.dw_draw.argtypes = [ctypes.c_uint64, ctypes.c_uint64]
        lib.dw_draw.restype = ctypes.c_uint64
        _rows_lib = lib
    return _rows_lib


def rows_key(cfg: int = 4, seed: int = 4) -> int:
    return stream_key(cfg, seed, TAG_ROWS)


def make_rows(n_rows: int, n_nodes: int, radix: int, row_begin: int = 0, key: Optional[int] = None,
              stride: Optional[int] = None, out: Optional[np.ndarray] = None, threads: int = 0) -> np.ndarray:
    """Rows [row_begin, row_begin + n_rows) of uniform ids in [0, radix).

    id(row, n) = (hi32(draw(key, row * n_nodes + n)) * radix) >> 32.
    """
    if key is None:
        key = rows_key()
    stride = n_nodes if stride is None else stride
    if out is None:
        out = np.zeros((n_rows, stride), dtype=np.uint8)
    assert out.dtype == np.uint8 and out.flags.c_contiguous and out.shape == (n_rows, stride)
    lib = _load_rows_lib()
    rc = lib.dw_rows(key, row_begin, n_rows, n_nodes, radix, stride, out.ctypes.data, threads)
    if rc != 0:
        raise RuntimeError(f"dw_rows failed ({rc})")
    return out


def make_rows_numpy(n_rows: int, n_nodes: int, radix: int, row_begin: int = 0,
                    key: Optional[int] = None) -> np.ndarray:
    """Slow pure-numpy twin of make_rows, for cross-checking the native generator."""
    if key is None:
        key = rows_key()
    ctr = (np.arange(row_begin, row_begin + n_rows, dtype=np.uint64)[:, None] * np.uint64(n_nodes)
           + np.arange(n_nodes, dtype=np.uint64)[None, :])
    hi = draw(key, ctr) >> np.uint64(32)
    with np.errstate(over="ignore"):
        ids = (hi * np.uint64(radix)) >> np.uint64(32)
    return ids.astype(np.uint8)


def by_name(name: str) -> Problem:
    return {"chain4": chain4, "forkjoin8": forkjoin8, "layered10": layered10,
            "stream24": stream24}[name]()


def per_class(prob: Problem, factors=(1.0, 0.5)) -> Problem:
    """The problem under per-backend pressure: at level k backend b gets
    factors[b] * rho_k (rho_k = the level's value, backend 0's column), a
    synthetic stand-in for the per-class load the runtime reads from the
    serving backends (Sec. 5.2).  The default presses the second backend half
    as hard as the first."""
    p = prob.copy()
    base = prob.rho[:, 0].astype(np.float64)
    p.rho = np.stack([base * f for f in factors], axis=1).astype(np.float32)
    return p


def model_table(prob: Problem):
    """(model class of every implementation [N, R] int32, number of classes):
    the recipes give each model class its own size factor, so a class is the
    rank of the implementation's size among the problem's distinct sizes."""
    sizes = np.unique(prob.size)
    return np.searchsorted(sizes, prob.size).astype(np.int32), int(sizes.shape[0])
