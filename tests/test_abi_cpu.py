"""C-ABI checks that need no GPU: the library loads, exports every function the
header declares, its host self-checks pass, and dy_plan_create rejects bad
input with the documented status before touching the device."""
import ctypes
import math
import os
import re

import numpy as np
import pytest

from paper_2607_02942_amd import dyplan as D
from paper_2607_02942_amd import workload as wl

HEADER = os.path.join(os.path.dirname(os.path.dirname(__file__)), "include", "dyplan.h")


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(dy_[a-z_0-9]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    lib = D.lib()
    names = header_functions()
    assert "dy_plan_create" in names and "dy_plan_select" in names and "dy_plan_score" in names
    assert "dy_plan_destroy" in names
    for name in names:
        assert hasattr(lib, name), name
    assert set(names) <= set(D.EXPORTED)


def test_exports_equal_header_declarations():
    # every dy_* function the library exports is declared in the header, and
    # every declared one is exported (symbol table of the library built here)
    import subprocess
    out = subprocess.run(["nm", "-D", "--defined-only", D.LIB_PATH], check=True, capture_output=True,
                         text=True).stdout
    exported = sorted({f[2] for f in (l.split() for l in out.splitlines())
                       if len(f) == 3 and f[1] == "T" and f[2].startswith("dy_")})
    assert exported == header_functions()
    assert sorted(D.EXPORTED) == exported


def test_abi_version_status_strings_and_selftest():
    lib = D.lib()
    assert lib.dy_abi_version() == 4
    assert lib.dy_selftest() == 0
    for st in (D.DY_OK, D.DY_EINVAL, D.DY_ENOTDAG, D.DY_ELIMIT, D.DY_ENOMEM, D.DY_EDEVICE):
        assert lib.dy_status_str(st).decode() not in ("", "unknown status")
    assert lib.dy_status_str(-99).decode() == "unknown status"


def test_struct_layouts_match_header():
    assert ctypes.sizeof(D.DyChoice) == 24
    assert ctypes.sizeof(D.DySource) == 48
    assert ctypes.sizeof(D.DyProblem) == 104
    assert ctypes.sizeof(D.DyObjective) == 56
    assert ctypes.sizeof(D.DyStats) == 40


def _struct(prob):
    a = D._Arrays(prob)
    return a, a.c


def _create_status(prob):
    a, c = _struct(prob)
    st, h = D.create_raw([c])
    if h:
        D.lib().dy_plan_destroy(h)
    return st, D.last_error(None)


def _gpu_present():
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:
        return False


def test_validation_errors_before_device():
    base = wl.chain4()
    cases = []
    p = base.copy(); p.edges = np.array([[1, 0]], np.int32); cases.append(("edge order", p, D.DY_ENOTDAG))
    p = base.copy(); p.edges = np.array([[2, 2]], np.int32); cases.append(("self loop", p, D.DY_ENOTDAG))
    p = base.copy(); p.edges = np.array([[0, 9]], np.int32); cases.append(("edge range", p, D.DY_EINVAL))
    p = base.copy(); p.radix = p.radix.copy(); p.radix[1] = 0; cases.append(("radix 0", p, D.DY_EINVAL))
    p = base.copy(); p.p = p.p.copy(); p.p[0, 3] = 1.5; cases.append(("p > 1", p, D.DY_EINVAL))
    p = base.copy(); p.p = p.p.copy(); p.p[2, 0] = np.nan; cases.append(("p NaN", p, D.DY_EINVAL))
    p = base.copy(); p.tau = p.tau.copy(); p.tau[1, 1] = -1.0; cases.append(("tau < 0", p, D.DY_EINVAL))
    p = base.copy(); p.tau = p.tau.copy(); p.tau[1, 1] = np.inf; cases.append(("tau inf", p, D.DY_EINVAL))
    p = base.copy(); p.w = p.w.copy(); p.w[0] = 1.01; cases.append(("w > 1", p, D.DY_EINVAL))
    p = base.copy(); p.rho = p.rho.copy(); p.rho[1, 0] = 1.0; cases.append(("rho = 1", p, D.DY_EINVAL))
    p = base.copy(); p.backend = p.backend.copy(); p.backend[0, 0] = 2; cases.append(("backend", p, D.DY_EINVAL))
    p = base.copy(); p.slo = float("nan"); cases.append(("slo NaN", p, D.DY_EINVAL))
    p = base.copy(); p.slo = -1.0; cases.append(("slo < 0", p, D.DY_EINVAL))
    p = base.copy(); p.rho = np.zeros((33, 2), np.float32); cases.append(("levels", p, D.DY_ELIMIT))
    for name, prob, want in cases:
        st, msg = _create_status(prob)
        assert st == want, (name, st, msg)
        assert msg, name


def test_validation_limits_and_null_pointers():
    # 33 nodes
    n = 33
    prob = wl.Problem(n_nodes=n, edges=np.zeros((0, 2), np.int32), radix=np.ones(n, np.int32),
                      p=np.ones((n, 1), np.float32), tau=np.ones((n, 1), np.float32),
                      size=np.ones((n, 1), np.float32), backend=np.zeros((n, 1), np.int32),
                      w=np.zeros(n, np.float32), rho=np.zeros((1, 1), np.float32), slo=1.0)
    assert _create_status(prob)[0] == D.DY_ELIMIT
    # radix above 255
    prob = wl.Problem(n_nodes=1, edges=np.zeros((0, 2), np.int32), radix=np.array([256], np.int32),
                      p=np.ones((1, 256), np.float32), tau=np.ones((1, 256), np.float32),
                      size=np.ones((1, 256), np.float32), backend=np.zeros((1, 256), np.int32),
                      w=np.zeros(1, np.float32), rho=np.zeros((1, 1), np.float32), slo=1.0)
    assert _create_status(prob)[0] == D.DY_ELIMIT
    a, c = _struct(wl.chain4())
    c.tau = None
    assert D.create_raw([c])[0] == D.DY_EINVAL
    h = ctypes.c_void_p()
    assert D.lib().dy_plan_create(None, 1, 0, ctypes.byref(h)) == D.DY_EINVAL
    assert D.lib().dy_plan_create((D.DyProblem * 1)(), 1, 0, None) == D.DY_EINVAL
    # NULL handle everywhere
    assert D.lib().dy_plan_select(None, None, 1, None, None) == D.DY_EINVAL
    assert D.lib().dy_plan_score(None, None, None, None, None, None, None) == D.DY_EINVAL
    assert D.lib().dy_plan_set_option(None, 1, 1) == D.DY_EINVAL
    D.lib().dy_plan_destroy(None)


@pytest.mark.skipif(_gpu_present(), reason="checks the no-device path")
def test_valid_problem_without_device_reports_device_error():
    st, msg = _create_status(wl.chain4())
    assert st == D.DY_EDEVICE and msg


def _obj_status(prob, obj, mutate=None):
    a = D._Arrays(prob, obj)
    if mutate:
        mutate(a)
    st, h = D.create_raw([a.c])
    if h:
        D.lib().dy_plan_destroy(h)
    return st, D.last_error(None)


def test_objective_validation_errors_before_device():
    import dataclasses
    base = wl.chain4()
    obj = wl.paper_objective(base)

    def with_(**kw):
        return dataclasses.replace(obj, **kw)

    cost_nan = obj.cost.copy(); cost_nan[1, 2] = np.nan
    cost_big = obj.cost.copy(); cost_big[0, 0] = 3e38
    cases = [
        ("cost NaN", with_(cost=cost_nan), None, D.DY_EINVAL),
        ("utility too large", with_(cost=cost_big, lambda_c=1e9), None, D.DY_EINVAL),
        ("effort > 1", with_(effort=1.5), None, D.DY_EINVAL),
        ("lambda_l < 0", with_(lambda_l=-0.1), None, D.DY_EINVAL),
        ("lambda_ld NaN", with_(lambda_ld=float("nan")), None, D.DY_EINVAL),
        ("beta inf", with_(beta=float("inf")), None, D.DY_EINVAL),
        ("level < 0", with_(levels=np.array([0.0, -1.0], np.float32)), None, D.DY_EINVAL),
        ("33 levels", with_(levels=np.zeros(33, np.float32)), None, D.DY_ELIMIT),
        ("is_tool 2", with_(is_tool=np.array([0, 2, 0, 0], np.int32)), None, D.DY_EINVAL),
        ("cost NULL", obj, lambda a: setattr(a.obj, "cost", None), D.DY_EINVAL),
        ("levels NULL", obj, lambda a: setattr(a.obj, "levels", None), D.DY_EINVAL),
        ("n_levels 0", obj, lambda a: setattr(a.obj, "n_levels", 0), D.DY_EINVAL),
    ]
    for name, o, mut, want in cases:
        st, msg = _obj_status(base, o, mut)
        assert st == want, (name, st, msg)
        assert msg, name


@pytest.mark.skipif(_gpu_present(), reason="checks the no-device path")
def test_objective_ignores_corr_only_fields():
    # rho, size and backend are not read in objective mode (NULL is accepted), and
    # an SLO or rho that corr / SLO selection rejects does not matter
    base = wl.chain4()
    obj = wl.paper_objective(base)

    def strip(a):
        a.c.rho = None
        a.c.size = None
        a.c.backend = None
        a.c.slo = float("nan")
        a.c.n_levels = 0
        a.c.n_backends = 0

    st, msg = _obj_status(base, obj, strip)
    assert st == D.DY_EDEVICE and msg
