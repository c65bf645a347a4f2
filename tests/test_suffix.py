"""Suffix recompilation (Appendix "Suffix Recompilation and Its Timing Scope",
eq. suffix-repair) through the C-ABI: the residual problem on G[U_t], the
selection on it, and the merge with the committed bindings.

The reference side builds the induced subproblem independently here (plain
numpy: keep the undispatched nodes in order, the edges between them, their
rows) and selects on it with the fp64 oracle.  CPU tests check the library's
residual problem and merge; GPU tests the whole recompilation.
"""
import ctypes
import dataclasses

import numpy as np
import pytest

from oracle import oracle as orc
from paper_2607_02942_amd import dyplan as D
from paper_2607_02942_amd import workload as wl


def induced(prob, obj, committed):
    """(Problem, Objective or None, node list) of G[U_t]."""
    keep = [n for n in range(prob.n_nodes) if not committed[n]]
    rid = {n: r for r, n in enumerate(keep)}
    edges = [(rid[int(u)], rid[int(v)]) for u, v in prob.edges if int(u) in rid and int(v) in rid]
    sub = wl.Problem(n_nodes=len(keep), edges=np.array(edges, np.int32).reshape(-1, 2),
                     radix=prob.radix[keep].copy(), p=prob.p[keep].copy(), tau=prob.tau[keep].copy(),
                     size=prob.size[keep].copy(), backend=prob.backend[keep].copy(), w=prob.w[keep].copy(),
                     rho=prob.rho.copy(), slo=prob.slo)
    sobj = None
    if obj is not None:
        sobj = dataclasses.replace(obj, cost=obj.cost[keep].copy(),
                                   is_tool=None if obj.is_tool is None else obj.is_tool[keep].copy())
    return sub, sobj, keep


def read_back(sfx):
    """The library's residual problem as numpy arrays."""
    P = sfx.problem
    N, R = P.n_nodes, P.max_radix

    def arr(ptr, shape, ct):
        if not ptr:
            return None
        return np.ctypeslib.as_array(ctypes.cast(ptr, ctypes.POINTER(ct)), shape=shape).copy()

    out = {"n": N, "R": R, "edges": arr(P.edges, (P.n_edges, 2), ctypes.c_int32) if P.n_edges else
           np.zeros((0, 2), np.int32), "radix": arr(P.radix, (N,), ctypes.c_int32),
           "p": arr(P.p, (N, R), ctypes.c_float), "tau": arr(P.tau, (N, R), ctypes.c_float),
           "w": arr(P.w, (N,), ctypes.c_float)}
    if P.objective:
        o = P.objective.contents
        out["cost"] = arr(o.cost, (N, R), ctypes.c_float)
        out["is_tool"] = arr(o.is_tool, (N,), ctypes.c_int32)
        out["levels"] = arr(o.levels, (o.n_levels,), ctypes.c_float)
    else:
        out["size"] = arr(P.size, (N, R), ctypes.c_float)
        out["backend"] = arr(P.backend, (N, R), ctypes.c_int32)
        out["rho"] = arr(P.rho, (P.n_levels, P.n_backends), ctypes.c_float)
        out["slo"] = P.slo
    return out


def random_dag(rng, n, R):
    edges = [(i, j) for i in range(n) for j in range(i + 1, n) if rng.random() < 0.35]
    return wl.Problem(n_nodes=n, edges=np.array(edges, np.int32).reshape(-1, 2),
                      radix=rng.integers(1, R + 1, n).astype(np.int32),
                      p=rng.uniform(0.5, 1.0, (n, R)).astype(np.float32),
                      tau=rng.lognormal(0, 0.5, (n, R)).astype(np.float32),
                      size=rng.choice([1.0, 2.5, 6.0], (n, R)).astype(np.float32),
                      backend=rng.integers(0, 2, (n, R)).astype(np.int32), w=rng.uniform(0, 1, n).astype(np.float32),
                      rho=np.array([[0.0, 0.0], [0.5, 0.3], [0.8, 0.6]], np.float32), slo=np.float32(np.inf))


# ---------------------------------------------------------------------------
# CPU: the residual problem and the merge
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("objective", [False, True])
def test_residual_problem_is_the_induced_subgraph(objective):
    rng = np.random.default_rng(3)
    for trial in range(30):
        n = int(rng.integers(2, 9))
        prob = random_dag(rng, n, 5)
        obj = None
        if objective:
            obj = wl.paper_objective(prob, is_tool=(rng.random(n) < 0.3).astype(np.int32) if trial % 2 else None)
        committed = (rng.random(n) < 0.4).astype(np.uint8)
        if committed.all():
            committed[-1] = 0
        sub, sobj, keep = induced(prob, obj, committed)
        sfx = D.Suffix(prob, committed, obj)
        got = read_back(sfx)
        assert got["n"] == len(keep) and sfx.node_map.tolist() == keep
        assert np.array_equal(got["edges"], sub.edges)
        assert np.array_equal(got["radix"], sub.radix)
        R = got["R"]
        assert np.array_equal(got["p"], sub.p[:, :R]) and np.array_equal(got["tau"], sub.tau[:, :R])
        assert np.array_equal(got["w"], sub.w)
        if objective:
            assert np.array_equal(got["cost"], sobj.cost)
            assert np.array_equal(got["levels"], sobj.levels)
            if sobj.is_tool is None:
                assert got["is_tool"] is None
            else:
                assert np.array_equal(got["is_tool"], sobj.is_tool)
        else:
            assert np.array_equal(got["size"], sub.size) and np.array_equal(got["backend"], sub.backend)
            assert np.array_equal(got["rho"], sub.rho)


def test_merge_keeps_committed_bindings_and_decodes_the_suffix():
    prob = wl.forkjoin8()
    committed = np.array([1, 1, 0, 1, 0, 0, 0, 0], np.uint8)
    cimpl = np.array([3, 11, -7, 5, -1, -1, -1, -1], np.int32)  # free nodes' entries are ignored
    sfx = D.Suffix(prob, committed)
    assert sfx.node_map.tolist() == [2, 4, 5, 6, 7]
    rng = np.random.default_rng(1)
    for ridx in [0, 1, 12 ** 5 - 1] + rng.integers(0, 12 ** 5, 50).tolist():
        impl, full = sfx.merge(cimpl, ridx)
        digits = [(ridx // 12 ** (4 - r)) % 12 for r in range(5)]
        want = cimpl.copy()
        want[[2, 4, 5, 6, 7]] = digits
        assert impl.tolist() == want.tolist()
        assert full == sum(int(want[n]) * 12 ** (7 - n) for n in range(8))
    with pytest.raises(D.DyplanError):
        sfx.merge(cimpl, 12 ** 5)  # outside the residual plan space
    bad = cimpl.copy()
    bad[3] = 12
    with pytest.raises(D.DyplanError):
        sfx.merge(bad, 0)  # committed id out of range


def test_suffix_errors():
    prob = wl.chain4()
    with pytest.raises(D.DyplanError):
        D.Suffix(prob, np.ones(4, np.uint8))  # nothing to recompile
    bad = prob.copy()
    bad.tau = bad.tau.copy()
    bad.tau[0, 0] = -1.0
    with pytest.raises(D.DyplanError):
        D.Suffix(bad, np.zeros(4, np.uint8))
    a = D._Arrays(prob)
    h = ctypes.c_void_p()
    assert D.lib().dy_suffix_create(ctypes.byref(a.c), None, ctypes.byref(h)) == D.DY_EINVAL
    assert D.lib().dy_suffix_merge(None, None, 0, None, None) == D.DY_EINVAL
    assert D.lib().dy_suffix_nodes(None, None) == 0
    D.lib().dy_suffix_destroy(None)


def test_nothing_committed_gives_the_full_problem():
    prob = wl.forkjoin8()
    obj = wl.paper_objective(prob)
    sfx = D.Suffix(prob, np.zeros(8, np.uint8), obj)
    got = read_back(sfx)
    assert got["n"] == 8 and np.array_equal(got["edges"], prob.edges)
    impl, full = sfx.merge(np.zeros(8, np.int32), 123456789)
    assert full == 123456789


# ---------------------------------------------------------------------------
# GPU: recompilation end to end
# ---------------------------------------------------------------------------

def _gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)
    return torch


def check_suffix(prob, obj, committed, cimpl, ctx):
    torch = _gpu()
    sub, sobj, keep = induced(prob, obj, committed)
    total = sub.n_plans()
    want = orc.obj_select_range(sub, sobj, 0, total) if obj is not None else orc.select_range(sub, 0, total)
    sfx = D.Suffix(prob, committed, obj)
    with sfx.plan() as plan:
        got = plan.select([D.range_source(0, 0, total)], stream=torch.cuda.current_stream())[0]
    for k, (g, w) in enumerate(zip(got, want)):
        assert (g[0], g[1]) == (int(w[0]), int(w[1])), f"{ctx} level {k}: {g} vs {w}"
        if int(w[1]):
            assert g[2] == np.float32(w[2]) and g[3] == np.float32(w[3]) and g[4] == np.float32(w[4]), ctx
            impl, _ = sfx.merge(cimpl, g[0])
            assert all(impl[n] == cimpl[n] for n in range(prob.n_nodes) if committed[n]), ctx
            rad = sub.radix
            digits = []
            x = g[0]
            for r in range(sub.n_nodes - 1, -1, -1):
                digits.append(x % int(rad[r]))
                x //= int(rad[r])
            assert [int(impl[n]) for n in keep] == digits[::-1], ctx


@pytest.mark.gpu
def test_forkjoin8_objective_suffix():
    prob = wl.forkjoin8()
    obj = wl.paper_objective(prob)
    # node 0 completed, branch nodes 1 and 2 in flight: 3..7 are recompiled
    committed = np.array([1, 1, 1, 0, 0, 0, 0, 0], np.uint8)
    check_suffix(prob, obj, committed, np.array([4, 7, 1, 0, 0, 0, 0, 0], np.int32), "forkjoin8 J_L")
    # a later point: the first branch stage done
    committed = np.array([1, 1, 1, 1, 1, 0, 0, 0], np.uint8)
    check_suffix(prob, obj, committed, np.array([4, 7, 1, 2, 9, 0, 0, 0], np.int32), "forkjoin8 J_L late")


@pytest.mark.gpu
def test_layered10_suffix_corr_and_objective():
    prob = wl.layered10()
    committed = np.array([1, 1, 1, 1, 1, 1, 0, 0, 0, 0], np.uint8)  # 36^4 residual plans
    cimpl = np.array([5, 0, 35, 17, 2, 30, 0, 0, 0, 0], np.int32)
    check_suffix(prob, None, committed, cimpl, "layered10 corr")
    check_suffix(prob, wl.paper_objective(prob), committed, cimpl, "layered10 J_L")


@pytest.mark.gpu
def test_random_dags_random_masks():
    rng = np.random.default_rng(11)
    for trial in range(12):
        n = int(rng.integers(3, 9))
        prob = random_dag(rng, n, 6)
        cps = orc.cp0_values(prob, 0, prob.n_plans())
        prob.slo = float(np.float32(np.median(cps) * 1.2))
        committed = (rng.random(n) < 0.4).astype(np.uint8)
        if committed.all():
            committed[0] = 0
        cimpl = np.array([int(rng.integers(0, r)) for r in prob.radix], np.int32)
        obj = wl.paper_objective(prob, is_tool=(rng.random(n) < 0.25).astype(np.int32)) if trial % 2 else None
        check_suffix(prob, obj, committed, cimpl, f"trial {trial}")
