"""ctypes binding of the plain fp64 CPU oracle (oracle.c: corr / CP / demand
selection; objective.c: the paper's additive objective J_L).

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the benchmark's
CPU-baseline leg may use this module; the product path never does.  It shares
no code with the GPU library; it takes the same seeded inputs.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import List, Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liboracle.so")
SRC_PATH = os.path.join(_HERE, "oracle.c")
OBJ_PATH = os.path.join(_HERE, "objective.c")
CFLAGS = ["-O2", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared", "-std=c11"]


def build(force: bool = True) -> str:
    """Compile oracle.c and objective.c into liboracle.so (plain gcc, fp64, no FMA contraction)."""
    if force or not os.path.exists(LIB_PATH):
        subprocess.check_call(["gcc", *CFLAGS, "-o", LIB_PATH, SRC_PATH, OBJ_PATH, "-lm"])
    return LIB_PATH


class _Problem(ctypes.Structure):
    _fields_ = [
        ("n_nodes", ctypes.c_int32), ("n_edges", ctypes.c_int32),
        ("edges", ctypes.c_void_p), ("radix", ctypes.c_void_p), ("max_radix", ctypes.c_int32),
        ("p", ctypes.c_void_p), ("tau", ctypes.c_void_p), ("size", ctypes.c_void_p),
        ("backend", ctypes.c_void_p), ("w", ctypes.c_void_p),
        ("n_levels", ctypes.c_int32), ("n_backends", ctypes.c_int32),
        ("rho", ctypes.c_void_p), ("slo", ctypes.c_float),
    ]


class _ObjProblem(ctypes.Structure):
    _fields_ = [
        ("n_nodes", ctypes.c_int32), ("n_edges", ctypes.c_int32),
        ("edges", ctypes.c_void_p), ("radix", ctypes.c_void_p), ("max_radix", ctypes.c_int32),
        ("q", ctypes.c_void_p), ("tau", ctypes.c_void_p), ("cost", ctypes.c_void_p),
        ("v", ctypes.c_void_p), ("is_tool", ctypes.c_void_p),
        ("lambda_f", ctypes.c_float), ("lambda_c", ctypes.c_float), ("lambda_l", ctypes.c_float),
        ("lambda_ld", ctypes.c_float), ("beta", ctypes.c_float), ("effort", ctypes.c_float),
        ("n_levels", ctypes.c_int32), ("levels", ctypes.c_void_p),
    ]


class Choice(ctypes.Structure):
    _fields_ = [("index", ctypes.c_int64), ("feasible", ctypes.c_int32),
                ("corr", ctypes.c_double), ("cp", ctypes.c_double), ("demand", ctypes.c_double)]

    def as_tuple(self):
        return (int(self.index), int(self.feasible), float(self.corr), float(self.cp), float(self.demand))


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            build()
        L = ctypes.CDLL(LIB_PATH)
        P = ctypes.POINTER(_Problem)
        vp, u64, i32 = ctypes.c_void_p, ctypes.c_uint64, ctypes.c_int32
        L.or_decode.argtypes = [P, u64, vp]
        L.or_corr.argtypes = [P, vp]
        L.or_corr.restype = ctypes.c_double
        L.or_cp.argtypes = [P, vp, i32]
        L.or_cp.restype = ctypes.c_double
        L.or_demand.argtypes = [P, vp]
        L.or_demand.restype = ctypes.c_double
        L.or_select_range.argtypes = [P, u64, u64, vp]
        L.or_select_rows.argtypes = [P, vp, u64, u64, u64, vp]
        L.or_score_range.argtypes = [P, u64, u64, vp, vp, vp, vp]
        L.or_score_rows.argtypes = [P, vp, u64, u64, vp, vp, vp, vp]
        L.or_score_indices.argtypes = [P, vp, u64, vp, vp, vp, vp]
        L.or_cp0_hist.argtypes = [P, i32, vp, u64, u64, u64, i32, vp]
        L.or_cp0_collect.argtypes = [P, i32, vp, u64, u64, u64, i32, u64, vp, u64]
        L.or_cp0_collect.restype = ctypes.c_int64
        L.or_cp0_range.argtypes = [P, i32, vp, u64, u64, u64, vp]
        for f in ("or_select_range", "or_select_rows", "or_score_range", "or_score_rows",
                  "or_score_indices", "or_cp0_hist", "or_cp0_range"):
            getattr(L, f).restype = ctypes.c_int32
        Q = ctypes.POINTER(_ObjProblem)
        L.op_reach.argtypes = [Q, vp]
        L.op_eval.argtypes = [Q, vp, vp, vp, vp, vp]
        L.op_select_range.argtypes = [Q, u64, u64, vp]
        L.op_select_rows.argtypes = [Q, vp, u64, u64, u64, vp]
        L.op_score.argtypes = [Q, i32, vp, u64, u64, u64, vp, vp, vp, vp]
        for f in ("op_reach", "op_eval", "op_select_range", "op_select_rows", "op_score"):
            getattr(L, f).restype = ctypes.c_int32
        _lib = L
    return _lib


class OracleProblem:
    """Holds contiguous copies of a problem's arrays and the C view of them."""

    def __init__(self, prob, slo: Optional[float] = None):
        self.n_nodes = int(prob.n_nodes)
        self.edges = np.ascontiguousarray(prob.edges, dtype=np.int32).reshape(-1, 2)
        self.radix = np.ascontiguousarray(prob.radix, dtype=np.int32)
        self.p = np.ascontiguousarray(prob.p, dtype=np.float32)
        self.tau = np.ascontiguousarray(prob.tau, dtype=np.float32)
        self.size = np.ascontiguousarray(prob.size, dtype=np.float32)
        self.backend = np.ascontiguousarray(prob.backend, dtype=np.int32)
        self.w = np.ascontiguousarray(prob.w, dtype=np.float32)
        self.rho = np.ascontiguousarray(prob.rho, dtype=np.float32)
        self.slo = float(prob.slo if slo is None else slo)
        self.K = int(self.rho.shape[0])
        self.c = _Problem(
            self.n_nodes, int(self.edges.shape[0]), self.edges.ctypes.data, self.radix.ctypes.data,
            int(self.p.shape[1]), self.p.ctypes.data, self.tau.ctypes.data, self.size.ctypes.data,
            self.backend.ctypes.data, self.w.ctypes.data, self.K, int(self.rho.shape[1]),
            self.rho.ctypes.data, ctypes.c_float(self.slo))

    @property
    def ref(self):
        return ctypes.byref(self.c)


def _op(prob, slo=None) -> OracleProblem:
    return prob if isinstance(prob, OracleProblem) else OracleProblem(prob, slo)


def decode(prob, index: int) -> np.ndarray:
    op = _op(prob)
    impl = np.zeros(op.n_nodes, np.int32)
    lib().or_decode(op.ref, int(index), impl.ctypes.data)
    return impl


def corr(prob, impl) -> float:
    op = _op(prob)
    a = np.ascontiguousarray(impl, dtype=np.int32)
    return lib().or_corr(op.ref, a.ctypes.data)


def cp(prob, impl, level: int) -> float:
    """Critical path at pressure level `level`; level=-1 gives the unpressured CP."""
    op = _op(prob)
    a = np.ascontiguousarray(impl, dtype=np.int32)
    return lib().or_cp(op.ref, a.ctypes.data, int(level))


def demand(prob, impl) -> float:
    op = _op(prob)
    a = np.ascontiguousarray(impl, dtype=np.int32)
    return lib().or_demand(op.ref, a.ctypes.data)


def select_range(prob, begin: int, count: int, slo=None) -> List[tuple]:
    op = _op(prob, slo)
    out = (Choice * op.K)()
    rc = lib().or_select_range(op.ref, int(begin), int(count), out)
    if rc != 0:
        raise ValueError(f"oracle select failed ({rc})")
    return [c.as_tuple() for c in out]


def select_rows(prob, rows: np.ndarray, index_base: int = 0, slo=None) -> List[tuple]:
    op = _op(prob, slo)
    rows = np.ascontiguousarray(rows, dtype=np.uint8)
    out = (Choice * op.K)()
    rc = lib().or_select_rows(op.ref, rows.ctypes.data, rows.shape[0], rows.shape[1], int(index_base), out)
    if rc != 0:
        raise ValueError(f"oracle select failed ({rc})")
    return [c.as_tuple() for c in out]


def score_range(prob, begin: int, count: int, slo=None):
    op = _op(prob, slo)
    corr_ = np.zeros(count, np.float64)
    cp_ = np.zeros((count, op.K), np.float64)
    dem = np.zeros(count, np.float64)
    feas = np.zeros(count, np.uint32)
    rc = lib().or_score_range(op.ref, int(begin), int(count), corr_.ctypes.data, cp_.ctypes.data,
                              dem.ctypes.data, feas.ctypes.data)
    if rc != 0:
        raise ValueError(f"oracle score failed ({rc})")
    return corr_, cp_, dem, feas


def score_rows(prob, rows: np.ndarray, slo=None):
    op = _op(prob, slo)
    rows = np.ascontiguousarray(rows, dtype=np.uint8)
    n = rows.shape[0]
    corr_ = np.zeros(n, np.float64)
    cp_ = np.zeros((n, op.K), np.float64)
    dem = np.zeros(n, np.float64)
    feas = np.zeros(n, np.uint32)
    rc = lib().or_score_rows(op.ref, rows.ctypes.data, n, rows.shape[1], corr_.ctypes.data,
                             cp_.ctypes.data, dem.ctypes.data, feas.ctypes.data)
    if rc != 0:
        raise ValueError(f"oracle score failed ({rc})")
    return corr_, cp_, dem, feas


def score_indices(prob, indices, slo=None):
    op = _op(prob, slo)
    idx = np.ascontiguousarray(indices, dtype=np.uint64)
    n = idx.shape[0]
    corr_ = np.zeros(n, np.float64)
    cp_ = np.zeros((n, op.K), np.float64)
    dem = np.zeros(n, np.float64)
    feas = np.zeros(n, np.uint32)
    rc = lib().or_score_indices(op.ref, idx.ctypes.data, n, corr_.ctypes.data, cp_.ctypes.data,
                                dem.ctypes.data, feas.ctypes.data)
    if rc != 0:
        raise ValueError(f"oracle score failed ({rc})")
    return corr_, cp_, dem, feas


def cp0_values(prob, begin: int = 0, count: Optional[int] = None, rows: Optional[np.ndarray] = None):
    """Unpressured CP for a range of plans (kind 0) or for every row (kind 1)."""
    op = _op(prob, 0.0)
    if rows is not None:
        rows = np.ascontiguousarray(rows, dtype=np.uint8)
        n = rows.shape[0]
        out = np.zeros(n, np.float64)
        lib().or_cp0_range(op.ref, 1, rows.ctypes.data, rows.shape[1], 0, n, out.ctypes.data)
        return out
    out = np.zeros(count, np.float64)
    lib().or_cp0_range(op.ref, 0, None, 0, int(begin), int(count), out.ctypes.data)
    return out


def merge_choices(parts: List[List[tuple]]) -> List[tuple]:
    """Exact merge of per-chunk selections given in increasing index order:
    the greatest correctness wins, ties go to the lowest plan index."""
    K = len(parts[0])
    best = [(-1, 0, float("nan"), float("nan"), float("nan"))] * K
    for part in parts:
        for k in range(K):
            c = part[k]
            if c[0] < 0:
                continue
            b = best[k]
            if b[0] < 0 or c[2] > b[2] or (c[2] == b[2] and c[0] < b[0]):
                best[k] = c
    return best


# ---------------------------------------------------------------------------
# the paper's additive objective (objective.c)
# ---------------------------------------------------------------------------

class ObjectiveProblem:
    """C view of a problem under the additive objective: quality q = p, vulnerability
    v = w, nominal durations tau, and the objective's costs, weights and levels."""

    def __init__(self, prob, obj):
        self.n_nodes = int(prob.n_nodes)
        self.edges = np.ascontiguousarray(prob.edges, dtype=np.int32).reshape(-1, 2)
        self.radix = np.ascontiguousarray(prob.radix, dtype=np.int32)
        self.q = np.ascontiguousarray(prob.p, dtype=np.float32)
        self.tau = np.ascontiguousarray(prob.tau, dtype=np.float32)
        self.cost = np.ascontiguousarray(obj.cost, dtype=np.float32)
        self.v = np.ascontiguousarray(prob.w, dtype=np.float32)
        self.is_tool = None if obj.is_tool is None else np.ascontiguousarray(obj.is_tool, dtype=np.int32)
        self.levels = np.ascontiguousarray(obj.levels, dtype=np.float32)
        self.K = int(self.levels.shape[0])
        self.c = _ObjProblem(
            self.n_nodes, int(self.edges.shape[0]), self.edges.ctypes.data, self.radix.ctypes.data,
            int(self.q.shape[1]), self.q.ctypes.data, self.tau.ctypes.data, self.cost.ctypes.data,
            self.v.ctypes.data, None if self.is_tool is None else self.is_tool.ctypes.data,
            obj.lambda_f, obj.lambda_c, obj.lambda_l, obj.lambda_ld, obj.beta, obj.effort,
            self.K, self.levels.ctypes.data)

    @property
    def ref(self):
        return ctypes.byref(self.c)


class ObjChoice(ctypes.Structure):
    _fields_ = [("index", ctypes.c_int64), ("feasible", ctypes.c_int32),
                ("j", ctypes.c_double), ("t", ctypes.c_double), ("d", ctypes.c_double)]

    def as_tuple(self):
        return (int(self.index), int(self.feasible), float(self.j), float(self.t), float(self.d))


def _oq(prob, obj) -> ObjectiveProblem:
    return prob if isinstance(prob, ObjectiveProblem) else ObjectiveProblem(prob, obj)


def obj_reach(prob, obj) -> np.ndarray:
    q = _oq(prob, obj)
    out = np.zeros(q.n_nodes, np.float64)
    if lib().op_reach(q.ref, out.ctypes.data) != 0:
        raise ValueError("bad problem")
    return out


def obj_eval(prob, obj, impl):
    """(U, T, D, [J_k]) of one plan given by its implementation ids."""
    q = _oq(prob, obj)
    a = np.ascontiguousarray(impl, dtype=np.int32)
    U, T, D = ctypes.c_double(), ctypes.c_double(), ctypes.c_double()
    J = np.zeros(q.K, np.float64)
    if lib().op_eval(q.ref, a.ctypes.data, ctypes.byref(U), ctypes.byref(T), ctypes.byref(D), J.ctypes.data):
        raise ValueError("bad problem")
    return U.value, T.value, D.value, J


def obj_select_range(prob, obj, begin: int, count: int) -> List[tuple]:
    q = _oq(prob, obj)
    out = (ObjChoice * q.K)()
    if lib().op_select_range(q.ref, int(begin), int(count), out) != 0:
        raise ValueError("bad problem")
    return [c.as_tuple() for c in out]


def obj_select_rows(prob, obj, rows: np.ndarray, index_base: int = 0) -> List[tuple]:
    q = _oq(prob, obj)
    rows = np.ascontiguousarray(rows, dtype=np.uint8)
    out = (ObjChoice * q.K)()
    if lib().op_select_rows(q.ref, rows.ctypes.data, rows.shape[0], rows.shape[1], int(index_base), out) != 0:
        raise ValueError("bad problem")
    return [c.as_tuple() for c in out]


def obj_score(prob, obj, begin: int = 0, count: Optional[int] = None, rows: Optional[np.ndarray] = None):
    """Per-plan U, T, D and J[:, k] over a range or over rows."""
    q = _oq(prob, obj)
    if rows is not None:
        rows = np.ascontiguousarray(rows, dtype=np.uint8)
        n, kind, rp, st = rows.shape[0], 1, rows.ctypes.data, rows.shape[1]
    else:
        n, kind, rp, st = int(count), 0, None, 0
    U, T, D = (np.zeros(n, np.float64) for _ in range(3))
    J = np.zeros((n, q.K), np.float64)
    if lib().op_score(q.ref, kind, rp, st, int(begin), n, U.ctypes.data, T.ctypes.data, D.ctypes.data,
                      J.ctypes.data) != 0:
        raise ValueError("bad problem")
    return U, T, D, J
