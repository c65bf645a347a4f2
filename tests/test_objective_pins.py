"""Pins of the oracle's additive objective (oracle/objective.c) to the paper.

The decisive pin solves the paper's ILP itself (Sec. 4.3: one implementation
per LLM node, precedence constraints a_v >= a_u + d(u), completion T >= a_n +
d(n), objective eq. admission-objective minus lambda_ld L D_tau of eq.
variant-objective) with an independent MILP solver on tiny DAGs; its optimum
must equal the oracle's brute-force maximum of J_k for every level.  The
critical path enters the ILP only through the precedence constraints and the
reach weights and utilities are recomputed here from the paper's formulas, so
a wrong sign, a dropped term, a wrong reach set or a tool node counted in D_tau
shows up as a different optimum.  Closed forms and identities follow.
"""
import numpy as np
import pytest

from oracle import oracle as orc
from paper_2607_02942_amd import workload as wl

scipy_opt = pytest.importorskip("scipy.optimize")


def f32(x):
    """The objective's weights are fp32 inputs."""
    return float(np.float32(x))


def reach_sizes(n, edges):
    succ = [[] for _ in range(n)]
    for u, v in edges:
        succ[int(u)].append(int(v))
    out = []
    for s in range(n):
        seen, stack = {s}, [s]
        while stack:
            x = stack.pop()
            for y in succ[x]:
                if y not in seen:
                    seen.add(y)
                    stack.append(y)
        out.append(len(seen))
    return out


def utilities(prob, obj):
    """u[n][i] from Sec. 4.3 (reach(n) q - lambda_f v (1 - q) - lambda_c c), in fp64."""
    n = prob.n_nodes
    sizes = reach_sizes(n, prob.edges)
    reach = [1.0 if n == 1 else 1.0 + f32(obj.beta) * f32(obj.effort) * (sizes[m] - 1) / (n - 1)
             for m in range(n)]
    q = prob.p.astype(np.float64)
    u = np.array(reach)[:, None] * q - f32(obj.lambda_f) * prob.w.astype(np.float64)[:, None] * (1 - q) \
        - f32(obj.lambda_c) * obj.cost.astype(np.float64)
    return reach, u


def random_problem(rng, n, rmax, tools=False):
    edges = [(i, j) for i in range(n) for j in range(i + 1, n) if rng.random() < 0.45]
    radix = rng.integers(1, rmax + 1, size=n).astype(np.int32)
    R = int(radix.max())
    prob = wl.Problem(
        n_nodes=n, edges=np.array(edges, np.int32).reshape(-1, 2), radix=radix,
        p=rng.uniform(0.5, 1.0, size=(n, R)).astype(np.float32),
        tau=rng.choice([0.5, 1.0, 1.5, 2.0, 3.0, 4.5], size=(n, R)).astype(np.float32),
        size=rng.choice([1.0, 2.5, 6.0], size=(n, R)).astype(np.float32),
        backend=np.zeros((n, R), np.int32), w=rng.uniform(0, 1, size=n).astype(np.float32),
        rho=np.zeros((1, 1), np.float32))
    obj = wl.paper_objective(prob, levels=(0.0, 1.5, 3.0), lambda_f=float(rng.uniform(0.2, 2.0)),
                             lambda_c=float(rng.uniform(0.0, 0.05)), lambda_l=float(rng.choice([0.05, 0.1, 0.4])),
                             lambda_ld=float(rng.uniform(0.0, 0.2)), beta=float(rng.uniform(0.5, 2.0)),
                             effort=float(rng.uniform(0.0, 1.0)))
    if tools:
        is_tool = np.zeros(n, np.int32)
        for m in range(n):
            if radix[m] == 1 and rng.random() < 0.7:
                is_tool[m] = 1
        obj.is_tool = is_tool
    return prob, obj


def ilp_optimum(prob, obj, level):
    """max J_level by the paper's ILP (scipy milp, HiGHS); returns (value, plan)."""
    n = prob.n_nodes
    _, u = utilities(prob, obj)
    tool = np.zeros(n, bool) if obj.is_tool is None else obj.is_tool.astype(bool)
    tau = prob.tau.astype(np.float64)
    cols = [(m, i) for m in range(n) for i in range(int(prob.radix[m]))]
    ny = len(cols)
    nv = ny + n + 1                       # y..., a_0..a_{n-1}, T
    mu = f32(obj.lambda_ld) * float(obj.levels[level])
    c = np.zeros(nv)
    for j, (m, i) in enumerate(cols):
        if not tool[m]:
            c[j] = -(u[m, i] - mu * tau[m, i])
    c[-1] = f32(obj.lambda_l)
    A, lo, hi = [], [], []
    for m in range(n):                    # one implementation per node
        row = np.zeros(nv)
        for j, (mm, i) in enumerate(cols):
            if mm == m:
                row[j] = 1.0
        A.append(row), lo.append(1.0), hi.append(1.0)
    for (a, b) in {(int(x), int(y)) for x, y in prob.edges}:   # a_b >= a_a + d(a)
        row = np.zeros(nv)
        row[ny + b], row[ny + a] = 1.0, -1.0
        for j, (mm, i) in enumerate(cols):
            if mm == a:
                row[j] = -tau[a, i]
        A.append(row), lo.append(0.0), hi.append(np.inf)
    for m in range(n):                    # T >= a_m + d(m)
        row = np.zeros(nv)
        row[-1], row[ny + m] = 1.0, -1.0
        for j, (mm, i) in enumerate(cols):
            if mm == m:
                row[j] = -tau[m, i]
        A.append(row), lo.append(0.0), hi.append(np.inf)
    integrality = np.zeros(nv)
    integrality[:ny] = 1
    bounds = scipy_opt.Bounds(np.zeros(nv), np.concatenate([np.ones(ny), np.full(n + 1, np.inf)]))
    res = scipy_opt.milp(c, constraints=scipy_opt.LinearConstraint(np.array(A), lo, hi),
                         integrality=integrality, bounds=bounds,
                         options={"mip_rel_gap": 0.0})
    assert res.success, res.message
    plan = [0] * n
    for j, (m, i) in enumerate(cols):
        if res.x[j] > 0.5:
            plan[m] = i
    return -res.fun, plan


@pytest.mark.parametrize("tools", [False, True])
def test_ilp_optimum_equals_oracle_maximum(tools):
    rng = np.random.default_rng(31 + tools)
    for trial in range(25):
        prob, obj = random_problem(rng, int(rng.integers(1, 6)), 4, tools)
        total = prob.n_plans()
        _, _, _, J = orc.obj_score(prob, obj, 0, total)
        got = orc.obj_select_range(prob, obj, 0, total)
        for k in range(obj.n_levels):
            opt, plan = ilp_optimum(prob, obj, k)
            # the solver's feasibility tolerance (~1e-7 on T) bounds the agreement; every term
            # of J is of order 1e-2 or more, so a modelling mistake is far outside 1e-5
            assert got[k][2] == pytest.approx(opt, rel=0, abs=1e-5), f"trial {trial} level {k}"
            assert J[got[k][0], k] == got[k][2]
            order = np.sort(J[:, k])[::-1]
            if total > 1 and order[0] - order[1] > 1e-5:       # unique optimum: same plan
                idx = 0
                for m in range(prob.n_nodes):
                    idx = idx * int(prob.radix[m]) + plan[m]
                assert idx == got[k][0], f"trial {trial} level {k}"


def test_reach_closed_forms():
    fj = wl.forkjoin8()
    r = orc.obj_reach(fj, wl.paper_objective(fj, beta=1.0, effort=0.5))
    # node 0 reaches all 8 nodes, a first-stage branch node 3, a second-stage one 2, the join 1
    want = [1 + 0.5 * 7 / 7] + [1 + 0.5 * 2 / 7] * 3 + [1 + 0.5 * 1 / 7] * 3 + [1.0]
    np.testing.assert_allclose(r, want, rtol=0, atol=1e-15)
    ch = wl.chain4()
    np.testing.assert_allclose(orc.obj_reach(ch, wl.paper_objective(ch, beta=2.0, effort=1.0)),
                               [3.0, 1 + 2 * 2 / 3, 1 + 2 / 3, 1.0], atol=1e-15)
    np.testing.assert_array_equal(orc.obj_reach(ch, wl.paper_objective(ch, effort=0.0)), [1.0] * 4)
    one = wl.Problem(n_nodes=1, edges=np.zeros((0, 2), np.int32), radix=np.array([2], np.int32),
                     p=np.ones((1, 2), np.float32), tau=np.ones((1, 2), np.float32),
                     size=np.ones((1, 2), np.float32), backend=np.zeros((1, 2), np.int32),
                     w=np.ones(1, np.float32), rho=np.zeros((1, 1), np.float32))
    assert orc.obj_reach(one, wl.paper_objective(one, beta=5.0, effort=1.0))[0] == 1.0


def test_separable_without_latency_and_demand_weights():
    # lambda_l = lambda_ld = 0: J is a sum of per-node utilities, so the best plan
    # takes every node's best implementation (lowest id among equals)
    rng = np.random.default_rng(8)
    for _ in range(10):
        prob, obj = random_problem(rng, int(rng.integers(2, 6)), 4)
        obj.lambda_l = 0.0
        obj.lambda_ld = 0.0
        _, u = utilities(prob, obj)
        idx = 0
        for m in range(prob.n_nodes):
            idx = idx * int(prob.radix[m]) + int(np.argmax(u[m, :prob.radix[m]]))
        for c in orc.obj_select_range(prob, obj, 0, prob.n_plans()):
            assert c[0] == idx


def test_quality_and_error_terms_weight_correctness_by_reach_plus_vulnerability():
    # Sec. 4.3: with r = 1 - q, rho q - lambda_f v r = (rho + lambda_f v) q - lambda_f v, so two
    # plans that differ at one node differ in U by (rho + lambda_f v)(q1 - q2) - lambda_c (c1 - c2)
    rng = np.random.default_rng(9)
    prob, obj = random_problem(rng, 5, 4)
    prob.radix[:] = 4
    prob.p = rng.uniform(0.5, 1, size=(5, 4)).astype(np.float32)
    prob.tau = np.ones((5, 4), np.float32)
    prob.size = np.ones((5, 4), np.float32)
    obj = wl.paper_objective(prob, lambda_f=0.7, lambda_c=0.03, beta=1.3, effort=0.9)
    reach = orc.obj_reach(prob, obj)
    base = np.zeros(5, np.int32)
    U0 = orc.obj_eval(prob, obj, base)[0]
    for m in range(5):
        for i in range(1, 4):
            plan = base.copy()
            plan[m] = i
            dq = float(prob.p[m, i]) - float(prob.p[m, 0])
            dc = float(obj.cost[m, i]) - float(obj.cost[m, 0])
            want = (reach[m] + f32(obj.lambda_f) * float(prob.w[m])) * dq - f32(obj.lambda_c) * dc
            assert orc.obj_eval(prob, obj, plan)[0] - U0 == pytest.approx(want, abs=1e-12)


def test_terms_by_hand_on_a_fork_join():
    # 0 -> {1, 2} -> 3 with one implementation each: T = tau0 + max(tau1, tau2) + tau3, D the sum
    tau = np.array([[2.0], [5.0], [3.0], [1.0]], np.float32)
    prob = wl.Problem(n_nodes=4, edges=np.array([[0, 1], [0, 2], [1, 3], [2, 3]], np.int32),
                      radix=np.ones(4, np.int32), p=np.full((4, 1), 0.5, np.float32), tau=tau,
                      size=np.ones((4, 1), np.float32), backend=np.zeros((4, 1), np.int32),
                      w=np.array([1.0, 0.0, 0.5, 0.25], np.float32), rho=np.zeros((1, 1), np.float32))
    obj = wl.Objective(cost=np.array([[1.0], [2.0], [0.0], [4.0]], np.float32),
                       levels=np.array([0.0, 2.0], np.float32), lambda_f=1.0, lambda_c=0.5, lambda_l=0.1,
                       lambda_ld=0.25, beta=1.0, effort=1.0)
    U, T, D, J = orc.obj_eval(prob, obj, [0, 0, 0, 0])
    reach = [1 + 3 / 3, 1 + 1 / 3, 1 + 1 / 3, 1.0]
    u = [reach[m] * 0.5 - 1.0 * [1.0, 0.0, 0.5, 0.25][m] * 0.5 - 0.5 * [1.0, 2.0, 0.0, 4.0][m] for m in range(4)]
    assert T == 8.0 and D == 11.0
    assert U == pytest.approx(sum(u), abs=1e-15)
    assert J[0] == pytest.approx(sum(u) - f32(0.1) * 8.0, abs=1e-15)
    assert J[1] == pytest.approx(sum(u) - f32(0.1) * 8.0 - 0.25 * 2.0 * 11.0, abs=1e-15)
    # node 1 as a tool node: its duration stays in T, leaves U and D
    obj.is_tool = np.array([0, 1, 0, 0], np.int32)
    U2, T2, D2, J2 = orc.obj_eval(prob, obj, [0, 0, 0, 0])
    assert T2 == 8.0 and D2 == 6.0
    assert U2 == pytest.approx(sum(u) - u[1], abs=1e-15)


def test_rows_equal_range_and_ties_go_to_lowest_index():
    rng = np.random.default_rng(12)
    prob, obj = random_problem(rng, 4, 3)
    prob.radix[:] = 3
    for arr in (prob.p, prob.tau, prob.size):      # implementation 2 duplicates implementation 1
        arr[:, 2] = arr[:, 1]
    obj = wl.paper_objective(prob)
    total = prob.n_plans()
    rows = np.stack([orc.decode(prob, i) for i in range(total)]).astype(np.uint8)
    assert orc.obj_select_rows(prob, obj, rows, 0) == orc.obj_select_range(prob, obj, 0, total)
    for c in orc.obj_select_range(prob, obj, 0, total):
        assert 2 not in orc.decode(prob, c[0])      # never the duplicate with the larger id
    # rows in another order, same plans: the same choices with the rows' own indices
    perm = rng.permutation(total)
    got = orc.obj_select_rows(prob, obj, rows[perm], 0)
    for g, w in zip(got, orc.obj_select_range(prob, obj, 0, total)):
        assert g[2] == w[2]
