"""Python binding of the C-ABI plan scorer (libdyplan.so).

Argument marshalling only: every step of scoring and selection runs in the HIP
library.  Host arrays are numpy; device buffers are passed as raw pointers
(ints) or any object with a ``data_ptr()`` method (e.g. torch tensors), and a
stream as a raw ``hipStream_t`` (int), an object with ``cuda_stream``, or None
for the default stream.  The library must be built (``__graft_entry__.build()``);
importing this module never falls back to anything else.
"""
from __future__ import annotations

import ctypes
import os
from typing import List, Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libdyplan.so")

DY_OK, DY_EINVAL, DY_ENOTDAG, DY_ELIMIT, DY_ENOMEM, DY_EDEVICE = 0, -1, -2, -3, -4, -5
DY_SOURCE_RANGE, DY_SOURCE_ROWS = 0, 1
DY_OPT_TIMING, DY_OPT_SAMPLE_STRIDE, DY_OPT_CAND_CAPACITY, DY_OPT_FORCE_FP64, DY_OPT_JIT, DY_OPT_GRAPH = 1, 2, 3, 4, 5, 6
DY_OPT_CLIMB = 7
DY_MAX_NODES, DY_MAX_RADIX, DY_MAX_LEVELS, DY_MAX_BACKENDS = 32, 255, 32, 64

EXPORTED = ("dy_plan_create", "dy_plan_select", "dy_plan_score", "dy_plan_destroy", "dy_plan_max_levels",
            "dy_plan_num_problems", "dy_plan_set_option", "dy_plan_get_stats", "dy_plan_last_error",
            "dy_status_str", "dy_abi_version", "dy_selftest", "dy_suffix_create", "dy_suffix_problem",
            "dy_suffix_nodes", "dy_suffix_merge", "dy_suffix_destroy", "dy_bundle_annotate",
            "dy_switch_simulate", "dy_kernel_source", "dy_plan_select_static")


class DyObjective(ctypes.Structure):
    _fields_ = [
        ("cost", ctypes.c_void_p), ("is_tool", ctypes.c_void_p), ("lambda_f", ctypes.c_float),
        ("lambda_c", ctypes.c_float), ("lambda_l", ctypes.c_float), ("lambda_ld", ctypes.c_float),
        ("beta", ctypes.c_float), ("effort", ctypes.c_float), ("n_levels", ctypes.c_int32),
        ("levels", ctypes.c_void_p),
    ]


class DyProblem(ctypes.Structure):
    _fields_ = [
        ("n_nodes", ctypes.c_int32), ("n_edges", ctypes.c_int32), ("edges", ctypes.c_void_p),
        ("radix", ctypes.c_void_p), ("max_radix", ctypes.c_int32), ("p", ctypes.c_void_p),
        ("tau", ctypes.c_void_p), ("size", ctypes.c_void_p), ("backend", ctypes.c_void_p),
        ("w", ctypes.c_void_p), ("n_levels", ctypes.c_int32), ("n_backends", ctypes.c_int32),
        ("rho", ctypes.c_void_p), ("slo", ctypes.c_float), ("objective", ctypes.POINTER(DyObjective)),
    ]


class DyVariant(ctypes.Structure):
    _fields_ = [("dominant", ctypes.c_int32), ("quality", ctypes.c_double)]


class DySwitchRules(ctypes.Structure):
    _fields_ = [("high", ctypes.c_double), ("low", ctypes.c_double), ("tolerance", ctypes.c_double),
                ("margin", ctypes.c_double), ("dwell", ctypes.c_double)]


class DySource(ctypes.Structure):
    _fields_ = [
        ("kind", ctypes.c_int32), ("problem", ctypes.c_int32), ("begin", ctypes.c_uint64),
        ("count", ctypes.c_uint64), ("rows", ctypes.c_void_p), ("row_stride", ctypes.c_uint64),
        ("index_base", ctypes.c_uint64),
    ]


class DyChoice(ctypes.Structure):
    _fields_ = [("index", ctypes.c_int64), ("feasible", ctypes.c_int32), ("corr", ctypes.c_float),
                ("cp", ctypes.c_float), ("demand", ctypes.c_float)]

    def as_tuple(self):
        return (int(self.index), int(self.feasible), float(self.corr), float(self.cp), float(self.demand))


class DyStats(ctypes.Structure):
    _fields_ = [("plans", ctypes.c_uint64), ("candidates", ctypes.c_uint64), ("fallbacks", ctypes.c_int32),
                ("n_jobs", ctypes.c_int32), ("main_ms", ctypes.c_float), ("total_ms", ctypes.c_float),
                ("generated_jobs", ctypes.c_int32), ("ydiv_jobs", ctypes.c_int32)]


class DyplanError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"dyplan status {status}: {message}")
        self.status = status


_lib = None


def lib():
    """Load libdyplan.so (raises if it has not been built).

    When PyTorch is installed it is imported first: its bundled HIP runtime
    carries this library's runtime soname, so the process then holds one HIP
    runtime.  Loaded the other way round, torch's libraries (which name the
    runtime without the version suffix) would load a second copy beside the
    system one, and the two disagree about the device."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
        try:
            import torch  # noqa: F401
        except ImportError:
            pass
        L = ctypes.CDLL(LIB_PATH)
        vp, i32 = ctypes.c_void_p, ctypes.c_int32
        L.dy_plan_create.argtypes = [ctypes.POINTER(DyProblem), i32, i32, ctypes.POINTER(vp)]
        L.dy_plan_create.restype = ctypes.c_int
        L.dy_plan_select.argtypes = [vp, ctypes.POINTER(DySource), i32, ctypes.POINTER(DyChoice), vp]
        L.dy_plan_select.restype = ctypes.c_int
        L.dy_plan_select_static.argtypes = [vp, ctypes.POINTER(DySource), i32, ctypes.POINTER(DyChoice), vp]
        L.dy_plan_select_static.restype = ctypes.c_int
        L.dy_plan_score.argtypes = [vp, ctypes.POINTER(DySource), vp, vp, vp, vp, vp]
        L.dy_plan_score.restype = ctypes.c_int
        L.dy_plan_destroy.argtypes = [vp]
        L.dy_plan_destroy.restype = None
        L.dy_plan_max_levels.argtypes = [vp]
        L.dy_plan_max_levels.restype = i32
        L.dy_plan_num_problems.argtypes = [vp]
        L.dy_plan_num_problems.restype = i32
        L.dy_plan_set_option.argtypes = [vp, i32, ctypes.c_int64]
        L.dy_plan_set_option.restype = ctypes.c_int
        L.dy_plan_get_stats.argtypes = [vp, ctypes.POINTER(DyStats)]
        L.dy_plan_get_stats.restype = ctypes.c_int
        L.dy_plan_last_error.argtypes = [vp]
        L.dy_plan_last_error.restype = ctypes.c_char_p
        L.dy_status_str.argtypes = [ctypes.c_int]
        L.dy_status_str.restype = ctypes.c_char_p
        L.dy_abi_version.restype = i32
        L.dy_selftest.restype = ctypes.c_int
        L.dy_suffix_create.argtypes = [ctypes.POINTER(DyProblem), vp, ctypes.POINTER(vp)]
        L.dy_suffix_create.restype = ctypes.c_int
        L.dy_suffix_problem.argtypes = [vp]
        L.dy_suffix_problem.restype = ctypes.POINTER(DyProblem)
        L.dy_suffix_nodes.argtypes = [vp, vp]
        L.dy_suffix_nodes.restype = i32
        L.dy_suffix_merge.argtypes = [vp, vp, ctypes.c_int64, vp, ctypes.POINTER(ctypes.c_int64)]
        L.dy_suffix_merge.restype = ctypes.c_int
        L.dy_suffix_destroy.argtypes = [vp]
        L.dy_suffix_destroy.restype = None
        L.dy_bundle_annotate.argtypes = [ctypes.POINTER(DyProblem), vp, i32, vp, vp, ctypes.POINTER(i32),
                                         ctypes.POINTER(ctypes.c_double)]
        L.dy_bundle_annotate.restype = ctypes.c_int
        L.dy_switch_simulate.argtypes = [ctypes.POINTER(DyVariant), i32, i32, vp, vp, i32,
                                         ctypes.POINTER(DySwitchRules), vp, ctypes.POINTER(i32)]
        L.dy_switch_simulate.restype = ctypes.c_int
        L.dy_kernel_source.argtypes = [ctypes.POINTER(DyProblem), ctypes.c_char_p, ctypes.c_uint64,
                                       ctypes.POINTER(ctypes.c_uint64)]
        L.dy_kernel_source.restype = ctypes.c_int
        _lib = L
    return _lib


def _ptr(x) -> Optional[int]:
    if x is None:
        return None
    if isinstance(x, int):
        return x
    if hasattr(x, "data_ptr"):
        return int(x.data_ptr())
    raise TypeError(f"cannot take a device pointer from {type(x)!r}")


def _stream(s) -> Optional[int]:
    if s is None:
        return None
    if isinstance(s, int):
        return s
    if hasattr(s, "cuda_stream"):
        return int(s.cuda_stream)
    raise TypeError(f"cannot take a stream from {type(s)!r}")


def range_source(problem: int, begin: int, count: int) -> DySource:
    return DySource(DY_SOURCE_RANGE, problem, begin, count, None, 0, 0)


def rows_source(problem: int, rows, count: int, row_stride: int, index_base: int = 0) -> DySource:
    """A ROWS source over device memory.  The source keeps a reference to
    `rows`, so a tensor passed as a temporary stays allocated while the source
    object is alive (the library only sees its address)."""
    src = DySource(DY_SOURCE_ROWS, problem, 0, count, _ptr(rows), row_stride, index_base)
    src._keep = rows
    return src


class _Arrays:
    """Contiguous host copies kept alive while dy_plan_create reads them.
    `obj` (a workload.Objective or None) selects the additive objective."""

    def __init__(self, prob, obj=None):
        self.edges = np.ascontiguousarray(prob.edges, dtype=np.int32).reshape(-1, 2)
        self.radix = np.ascontiguousarray(prob.radix, dtype=np.int32)
        self.p = np.ascontiguousarray(prob.p, dtype=np.float32)
        self.tau = np.ascontiguousarray(prob.tau, dtype=np.float32)
        self.size = np.ascontiguousarray(prob.size, dtype=np.float32)
        self.backend = np.ascontiguousarray(prob.backend, dtype=np.int32)
        self.w = np.ascontiguousarray(prob.w, dtype=np.float32)
        self.rho = np.ascontiguousarray(prob.rho, dtype=np.float32)
        self.c = DyProblem(int(prob.n_nodes), int(self.edges.shape[0]),
                           self.edges.ctypes.data if self.edges.size else None, self.radix.ctypes.data,
                           int(self.p.shape[1]), self.p.ctypes.data, self.tau.ctypes.data, self.size.ctypes.data,
                           self.backend.ctypes.data, self.w.ctypes.data, int(self.rho.shape[0]),
                           int(self.rho.shape[1]), self.rho.ctypes.data, ctypes.c_float(float(prob.slo)))
        self.obj = None
        if obj is not None:
            self.cost = np.ascontiguousarray(obj.cost, dtype=np.float32)
            self.levels = np.ascontiguousarray(obj.levels, dtype=np.float32)
            self.is_tool = None if obj.is_tool is None else np.ascontiguousarray(obj.is_tool, dtype=np.int32)
            self.obj = DyObjective(self.cost.ctypes.data, None if self.is_tool is None else self.is_tool.ctypes.data,
                                   obj.lambda_f, obj.lambda_c, obj.lambda_l, obj.lambda_ld, obj.beta, obj.effort,
                                   int(self.levels.shape[0]), self.levels.ctypes.data)
            self.c.objective = ctypes.pointer(self.obj)
        self.n_levels = int(self.levels.shape[0]) if obj is not None else int(self.rho.shape[0])


def create_raw(structs: Sequence[DyProblem], device: int = 0):
    """dy_plan_create on prepared structs; returns (status, handle or None)."""
    arr = (DyProblem * len(structs))(*structs)
    h = ctypes.c_void_p()
    st = lib().dy_plan_create(arr, len(structs), device, ctypes.byref(h))
    return st, (h.value if st == DY_OK else None)


def kernel_source(problem) -> str:
    """HIP source the library generates for one problem (a workload.Problem or
    a (Problem, Objective) pair); host-only, no device needed."""
    keep = _Arrays(*problem) if isinstance(problem, tuple) else _Arrays(problem)
    n = ctypes.c_uint64(0)
    st = lib().dy_kernel_source(ctypes.byref(keep.c), None, 0, ctypes.byref(n))
    if st != DY_OK:
        raise DyplanError(st, last_error(None))
    buf = ctypes.create_string_buffer(n.value + 1)
    st = lib().dy_kernel_source(ctypes.byref(keep.c), buf, n.value + 1, ctypes.byref(n))
    if st != DY_OK:
        raise DyplanError(st, last_error(None))
    return buf.value.decode()


def last_error(handle=None) -> str:
    msg = lib().dy_plan_last_error(handle)
    return msg.decode() if msg else ""


class Plan:
    """A handle over one or more planning problems staged on one device.  Each
    problem is a workload.Problem (corr / SLO selection) or a pair (Problem,
    Objective) for the paper's additive objective."""

    def __init__(self, problems, device: int = 0, _raw=None):
        if _raw is not None:  # prepared DyProblem structs and their level counts
            structs, self.n_levels = _raw
        else:
            if isinstance(problems, tuple) and len(problems) == 2 and hasattr(problems[1], "levels"):
                problems = [problems]
            probs = list(problems) if isinstance(problems, (list, tuple)) else [problems]
            keep = [_Arrays(*p) if isinstance(p, tuple) else _Arrays(p) for p in probs]
            structs, self.n_levels = [k.c for k in keep], [k.n_levels for k in keep]
        st, h = create_raw(structs, device)
        if st != DY_OK:
            raise DyplanError(st, last_error(None))
        self._h = h
        self.kmax = int(lib().dy_plan_max_levels(h))

    def close(self):
        if getattr(self, "_h", None):
            lib().dy_plan_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *a):
        self.close()

    def _check(self, st):
        if st != DY_OK:
            raise DyplanError(st, last_error(self._h))

    def set_option(self, option: int, value: int):
        self._check(lib().dy_plan_set_option(self._h, option, int(value)))

    def select(self, sources: Sequence[DySource], stream=None, static: bool = False) -> List[List[tuple]]:
        """Per source, the K choices (index, feasible, corr, cp, demand).
        static: through dy_plan_select_static (no allocation by the call)."""
        srcs = (DySource * len(sources))(*sources)
        out = (DyChoice * (len(sources) * self.kmax))()
        fn = lib().dy_plan_select_static if static else lib().dy_plan_select
        self._check(fn(self._h, srcs, len(sources), out, _stream(stream)))
        res = []
        for j, s in enumerate(sources):
            K = self.n_levels[s.problem]
            res.append([out[j * self.kmax + k].as_tuple() for k in range(K)])
        return res

    def select_raw(self, srcs, n: int, out, stream=None) -> int:
        """Unchecked call for timing loops: prepared ctypes arrays in and out."""
        return lib().dy_plan_select(self._h, srcs, n, out, _stream(stream))

    def score(self, source: DySource, corr=None, cp=None, demand=None, feas=None, stream=None):
        self._check(lib().dy_plan_score(self._h, ctypes.byref(source), _ptr(corr), _ptr(cp), _ptr(demand),
                                        _ptr(feas), _stream(stream)))

    def stats(self) -> DyStats:
        s = DyStats()
        self._check(lib().dy_plan_get_stats(self._h, ctypes.byref(s)))
        return s


class Suffix:
    """Residual problem of suffix recompilation (dy_suffix_*): `committed[n]`
    nonzero for completed or in-flight nodes.  plan() stages the residual
    problem; merge() joins a residual plan index with the committed bindings."""

    def __init__(self, prob, committed, obj=None):
        self._a = _Arrays(prob, obj)
        c = np.ascontiguousarray(committed, dtype=np.uint8)
        h = ctypes.c_void_p()
        st = lib().dy_suffix_create(ctypes.byref(self._a.c), c.ctypes.data, ctypes.byref(h))
        if st != DY_OK:
            raise DyplanError(st, last_error(None))
        self._h = h.value
        self.n_full = int(prob.n_nodes)
        self.n_nodes = int(lib().dy_suffix_nodes(self._h, None))
        self.node_map = np.zeros(self.n_nodes, np.int32)
        lib().dy_suffix_nodes(self._h, self.node_map.ctypes.data)
        self.n_levels = self._a.n_levels

    @property
    def problem(self) -> DyProblem:
        return lib().dy_suffix_problem(self._h).contents

    def plan(self, device: int = 0) -> "Plan":
        return Plan(None, device, _raw=([self.problem], [self.n_levels]))

    def merge(self, committed_impl, residual_index: int):
        """(implementation per full node, full plan index or -1)."""
        ci = np.ascontiguousarray(committed_impl, dtype=np.int32)
        out = np.zeros(self.n_full, np.int32)
        fi = ctypes.c_int64()
        st = lib().dy_suffix_merge(self._h, ci.ctypes.data, int(residual_index), out.ctypes.data, ctypes.byref(fi))
        if st != DY_OK:
            raise DyplanError(st, "suffix merge: bad committed id or residual index")
        return out, int(fi.value)

    def close(self):
        if getattr(self, "_h", None):
            lib().dy_suffix_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def annotate(prob, impl, model, n_models: int, obj=None):
    """dy_bundle_annotate: (per-model demand, dominant model, quality) of the
    plan impl[N]; model[N][R] gives each implementation's model class."""
    a = _Arrays(prob, obj)
    m = np.ascontiguousarray(model, dtype=np.int32)
    im = np.ascontiguousarray(impl, dtype=np.int32)
    dem = np.zeros(n_models, np.float64)
    dom = ctypes.c_int32()
    q = ctypes.c_double()
    st = lib().dy_bundle_annotate(ctypes.byref(a.c), m.ctypes.data, n_models, im.ctypes.data, dem.ctypes.data,
                                  ctypes.byref(dom), ctypes.byref(q))
    if st != DY_OK:
        raise DyplanError(st, "annotate: bad implementation or model id")
    return dem, int(dom.value), float(q.value)


def simulate(dominant, quality, times, loads, high: float, low: float, tolerance: float, margin: float = 0.0,
             dwell: float = 0.0):
    """dy_switch_simulate: (active variant after each load sample, switches)."""
    K = len(dominant)
    vs = (DyVariant * K)(*[DyVariant(int(d), float(q)) for d, q in zip(dominant, quality)])
    t = np.ascontiguousarray(times, dtype=np.float64)
    L = np.ascontiguousarray(loads, dtype=np.float64)
    n, nm = L.shape
    act = np.zeros(n, np.int32)
    sw = ctypes.c_int32()
    rules = DySwitchRules(high, low, tolerance, margin, dwell)
    st = lib().dy_switch_simulate(vs, K, nm, t.ctypes.data, L.ctypes.data, n, ctypes.byref(rules), act.ctypes.data,
                                  ctypes.byref(sw))
    if st != DY_OK:
        raise DyplanError(st, "simulate: bad arguments")
    return act, int(sw.value)
