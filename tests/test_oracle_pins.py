"""Pins of the fp64 CPU oracle against facts fixed by the paper and by mathematics.

Each test checks the oracle against something other than itself: the paper's
worked examples (fixtures under tests/golden/ with their citations), closed
forms, invariants, exact arithmetic on integer-valued inputs, and brute force
by independent algorithms on tiny inputs (all source->sink paths for the
critical path, all outcome patterns for correctness, a full sort for the
selection).
"""
import itertools
import json
import math
import os

import numpy as np
import pytest

from oracle import oracle as orc
from paper_2607_02942_amd.workload import Problem

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def make_problem(edges, tau, p=None, w=None, size=None, backend=None, rho=((0.0,),), slo=float("inf")):
    """tau: list of per-node lists of durations (ragged allowed)."""
    n = len(tau)
    R = max(len(t) for t in tau)
    T = np.zeros((n, R), np.float32)
    P = np.ones((n, R), np.float32)
    S = np.ones((n, R), np.float32)
    Bk = np.zeros((n, R), np.int32)
    for i, t in enumerate(tau):
        T[i, :len(t)] = t
        if p is not None:
            P[i, :len(p[i])] = p[i]
        if size is not None:
            S[i, :len(size[i])] = size[i]
        if backend is not None:
            Bk[i, :len(backend[i])] = backend[i]
    W = np.zeros(n, np.float32) if w is None else np.asarray(w, np.float32)
    return Problem(n_nodes=n, edges=np.asarray(edges, np.int32).reshape(-1, 2),
                   radix=np.array([len(t) for t in tau], np.int32), p=P, tau=T, size=S, backend=Bk,
                   w=W, rho=np.asarray(rho, np.float32), slo=float(np.float32(slo)))


def random_dag(rng, n, prob=0.4):
    e = [(i, j) for i in range(n) for j in range(i + 1, n) if rng.random() < prob]
    return np.array(e, np.int32).reshape(-1, 2)


def random_problem(rng, n, R, K=3, B=2, edge_p=0.4, integer_tau=False):
    edges = random_dag(rng, n, edge_p)
    radix = rng.integers(1, R + 1, size=n)
    if integer_tau:
        tau = [list(rng.integers(0, 9, size=r).astype(np.float32)) for r in radix]
    else:
        tau = [list(rng.lognormal(0, 0.5, size=r).astype(np.float32)) for r in radix]
    p = [list(rng.uniform(0.3, 1.0, size=r).astype(np.float32)) for r in radix]
    size = [list(rng.choice([0.5, 1.0, 2.5, 6.0], size=r).astype(np.float32)) for r in radix]
    backend = [list(rng.integers(0, B, size=r)) for r in radix]
    w = rng.uniform(0, 1, size=n)
    rho = np.sort(rng.uniform(0, 0.9, size=(K, B)).astype(np.float32), axis=0)
    return make_problem(edges, tau, p=p, w=w, size=size, backend=backend, rho=rho)


def all_paths(n, edges):
    """Every source->sink path of a DAG (sources: no predecessor; sinks: no successor)."""
    succ = {i: [] for i in range(n)}
    has_pred = [False] * n
    for u, v in edges:
        succ[int(u)].append(int(v))
        has_pred[int(v)] = True
    paths = []

    def walk(node, acc):
        acc = acc + [node]
        if not succ[node]:
            paths.append(acc)
        for v in succ[node]:
            walk(v, acc)

    for s in range(n):
        if not has_pred[s]:
            walk(s, [])
    return paths


def plan_index(radix, impl):
    idx = 0
    for r, i in zip(radix, impl):
        idx = idx * int(r) + int(i)
    return idx


# ---------------------------------------------------------------------------
# Paper worked examples
# ---------------------------------------------------------------------------

def test_forkjoin_verification_cost_example():
    g = json.load(open(os.path.join(GOLDEN, "forkjoin_example.json")))
    c_opts = g["impls"]["C"]
    d_opts = g["impls"]["D"]
    tau = [[0.0], [c_opts["27B"], c_opts["9B"]], [d_opts["9B"], d_opts["9B+verify"]], [0.0]]
    prob = make_problem(g["dag"]["edges"], tau)
    for case in g["verification_delta"]:
        ci = 0 if case["C"] == "27B" else 1
        with_v = orc.cp(prob, [0, ci, 1, 0], -1)
        without = orc.cp(prob, [0, ci, 0, 0], -1)
        assert with_v - without == case["delta"]


def test_walkthrough_latency_and_duration_sums():
    g = json.load(open(os.path.join(GOLDEN, "walkthrough.json")))
    tau = [[0.0], [t for _, t in g["impls"]["C"]], [t for _, t in g["impls"]["D"]], [0.0], [0.0]]
    prob = make_problem(g["dag"]["edges"], tau)
    for plan in g["plans"]:
        impl = [0, plan["C"], plan["D"], 0, 0]
        assert orc.cp(prob, impl, -1) == plan["fork_latency"], plan["name"]
        assert orc.demand(prob, impl) == plan["duration_sum"], plan["name"]
        # pressure on a single backend scales every duration: rho = 0.5 doubles them exactly
    prob2 = make_problem(g["dag"]["edges"], tau, rho=((0.0,), (0.5,), (0.75,)))
    for plan in g["plans"]:
        impl = [0, plan["C"], plan["D"], 0, 0]
        assert orc.cp(prob2, impl, 0) == plan["fork_latency"]
        assert orc.cp(prob2, impl, 1) == 2 * plan["fork_latency"]
        assert orc.cp(prob2, impl, 2) == 4 * plan["fork_latency"]


# ---------------------------------------------------------------------------
# Critical path
# ---------------------------------------------------------------------------

def test_chain_cp_is_sum_of_latencies_bit_exact():
    rng = np.random.default_rng(11)
    for n in (1, 2, 5, 9, 24):
        tau = [[float(x)] for x in rng.lognormal(0, 0.7, size=n).astype(np.float32)]
        rho = np.array([[0.0], [0.3], [0.85]], np.float32)
        prob = make_problem([(i, i + 1) for i in range(n - 1)], tau, rho=rho)
        for k in range(3):
            lat = [np.float64(t[0]) / (1.0 - np.float64(rho[k, 0])) for t in tau]
            s = 0.0
            for x in lat:
                s = s + x
            assert orc.cp(prob, [0] * n, k) == s
            assert abs(orc.cp(prob, [0] * n, k) - math.fsum(lat)) <= 1e-15 * s


def test_cp_equals_max_over_all_paths_integer_exact():
    rng = np.random.default_rng(12)
    for trial in range(60):
        n = int(rng.integers(1, 8))
        prob = random_problem(rng, n, 3, K=1, B=1, integer_tau=True)
        prob.rho[:] = 0.0
        paths = all_paths(n, prob.edges)
        for _ in range(5):
            impl = [int(rng.integers(0, r)) for r in prob.radix]
            d = [float(prob.tau[j, impl[j]]) for j in range(n)]
            expect = max(sum(d[j] for j in path) for path in paths)
            assert orc.cp(prob, impl, 0) == expect
            assert orc.cp(prob, impl, -1) == expect


def test_cp_brute_force_paths_float_with_backend_pressure():
    """Path enumeration with per-backend multipliers 2 and 4 (rho = .5, .75):
    checks that level k and the node's own backend pick the multiplier."""
    rng = np.random.default_rng(13)
    mult = {0.0: 1.0, 0.5: 2.0, 0.75: 4.0}
    for trial in range(40):
        n = int(rng.integers(2, 8))
        prob = random_problem(rng, n, 3, K=3, B=2)
        rho = np.array([[0.0, 0.5], [0.75, 0.0], [0.5, 0.75]], np.float32)
        prob.rho = rho
        paths = all_paths(n, prob.edges)
        for _ in range(4):
            impl = [int(rng.integers(0, r)) for r in prob.radix]
            for k in range(3):
                d = [float(prob.tau[j, impl[j]]) * mult[float(rho[k, prob.backend[j, impl[j]]])]
                     for j in range(n)]
                # multiplying by a power of two is exact; path sums are taken source-first
                best = 0.0
                for path in paths:
                    s = 0.0
                    for j in path:
                        s = d[j] + s
                    best = max(best, s)
                assert orc.cp(prob, impl, k) == best


def test_cp_monotone_in_pressure():
    rng = np.random.default_rng(14)
    prob = random_problem(rng, 6, 4, K=6, B=2)
    prob.rho = np.sort(rng.uniform(0, 0.95, size=(6, 2)).astype(np.float32), axis=0)
    for _ in range(50):
        impl = [int(rng.integers(0, r)) for r in prob.radix]
        cps = [orc.cp(prob, impl, k) for k in range(6)]
        assert all(a <= b for a, b in zip(cps, cps[1:]))
        assert cps[0] >= orc.cp(prob, impl, -1)


# ---------------------------------------------------------------------------
# Correctness
# ---------------------------------------------------------------------------

def test_corr_special_cases():
    rng = np.random.default_rng(21)
    n = 6
    p = [list(rng.uniform(0.5, 1.0, size=3).astype(np.float32)) for _ in range(n)]
    tau = [[1.0, 1.0, 1.0]] * n
    # no vulnerability: every factor is 1
    prob = make_problem([], tau, p=p, w=np.zeros(n))
    assert orc.corr(prob, [1] * n) == 1.0
    # perfect implementations: every factor is 1
    prob = make_problem([], tau, p=[[1.0] * 3] * n, w=rng.uniform(0, 1, n))
    assert orc.corr(prob, [2] * n) == 1.0
    # full vulnerability: product of success probabilities (exact for p in [0.5, 1])
    prob = make_problem([], tau, p=p, w=np.ones(n))
    impl = [int(rng.integers(0, 3)) for _ in range(n)]
    expect = 1.0
    for j in range(n):
        expect = expect * float(p[j][impl[j]])
    assert orc.corr(prob, impl) == expect


def test_corr_equals_outcome_pattern_brute_force():
    """Each node either succeeds (p), fails harmlessly ((1-p)(1-w)) or fails
    with impact ((1-p)w); the workflow is correct when no failure has impact."""
    rng = np.random.default_rng(22)
    for trial in range(30):
        n = int(rng.integers(1, 7))
        p = rng.uniform(0, 1, size=n).astype(np.float32)
        w = rng.uniform(0, 1, size=n).astype(np.float32)
        prob = make_problem([], [[1.0]] * n, p=[[x] for x in p], w=w)
        total = 0.0
        for pattern in itertools.product(range(3), repeat=n):
            pr = 1.0
            ok = True
            for j, o in enumerate(pattern):
                pj, wj = float(p[j]), float(w[j])
                if o == 0:
                    pr *= pj
                elif o == 1:
                    pr *= (1 - pj) * (1 - wj)
                else:
                    pr *= (1 - pj) * wj
                    ok = False
            if ok:
                total += pr
        c = orc.corr(prob, [0] * n)
        assert abs(c - total) <= 1e-12
        assert 0.0 <= c <= 1.0


def test_corr_monotone_in_each_success_probability():
    rng = np.random.default_rng(23)
    n = 5
    for _ in range(30):
        p = rng.uniform(0.1, 0.9, size=n).astype(np.float32)
        w = rng.uniform(0.05, 1, size=n).astype(np.float32)
        base = orc.corr(make_problem([], [[1.0]] * n, p=[[x] for x in p], w=w), [0] * n)
        for j in range(n):
            p2 = p.copy()
            p2[j] = np.float32(min(1.0, float(p[j]) + 0.05))
            c2 = orc.corr(make_problem([], [[1.0]] * n, p=[[x] for x in p2], w=w), [0] * n)
            assert c2 > base


# ---------------------------------------------------------------------------
# Demand and indexing
# ---------------------------------------------------------------------------

def test_demand_is_latency_times_size():
    prob = make_problem([(0, 1)], [[3.0, 4.0], [2.0]], size=[[2.5, 6.0], [1.0]])
    assert orc.demand(prob, [0, 0]) == 3.0 * 2.5 + 2.0
    assert orc.demand(prob, [1, 0]) == 4.0 * 6.0 + 2.0
    # demand ignores pressure and structure: a 2-branch fork sums both branches
    prob = make_problem([(0, 1), (0, 2)], [[1.0], [5.0], [7.0]], rho=((0.5,),))
    assert orc.demand(prob, [0, 0, 0]) == 13.0
    assert orc.cp(prob, [0, 0, 0], 0) == 16.0


def test_decode_is_mixed_radix_node0_most_significant():
    prob = make_problem([], [[0.0] * 3, [0.0] * 4, [0.0] * 5])
    assert list(orc.decode(prob, 0)) == [0, 0, 0]
    assert list(orc.decode(prob, 1)) == [0, 0, 1]
    assert list(orc.decode(prob, 5)) == [0, 1, 0]
    assert list(orc.decode(prob, 20)) == [1, 0, 0]
    assert list(orc.decode(prob, 59)) == [2, 3, 4]


# ---------------------------------------------------------------------------
# Selection
# ---------------------------------------------------------------------------

def sort_select(prob, slo):
    """Independent selection: score every plan, filter by CP_k <= SLO, sort by (-corr, index)."""
    radix = [int(r) for r in prob.radix]
    plans = list(itertools.product(*[range(r) for r in radix]))
    K = prob.rho.shape[0]
    out = []
    for k in range(K):
        feas = []
        for impl in plans:
            if orc.cp(prob, impl, k) <= slo:
                feas.append((-orc.corr(prob, impl), plan_index(radix, impl), impl))
        feas.sort()
        out.append(feas[0][1] if feas else -1)
    return out


def test_select_equals_full_sort_tiny():
    rng = np.random.default_rng(31)
    for trial in range(25):
        n = int(rng.integers(1, 5))
        prob = random_problem(rng, n, 4, K=3, B=2)
        cps = [orc.cp(prob, orc.decode(prob, j), -1) for j in range(prob.n_plans())]
        slo = float(np.float32(np.median(cps) * 1.5))
        got = orc.select_range(prob, 0, prob.n_plans(), slo=slo)
        assert [c[0] for c in got] == sort_select(prob, np.float64(np.float32(slo)))
        for c in got:
            if c[0] >= 0:
                impl = orc.decode(prob, c[0])
                assert c[1] == 1
                assert c[2] == orc.corr(prob, impl)
                assert c[4] == orc.demand(prob, impl)


def test_select_infinite_slo_is_per_node_argmax():
    rng = np.random.default_rng(32)
    n, R = 5, 4
    p = [list(rng.permutation(np.linspace(0.6, 0.95, R)).astype(np.float32)) for _ in range(n)]
    prob = make_problem(random_dag(rng, n), [[1.0] * R] * n, p=p, w=rng.uniform(0.2, 1, n),
                        rho=((0.0,), (0.5,)))
    got = orc.select_range(prob, 0, prob.n_plans(), slo=float("inf"))
    best = [int(np.argmax(p[j])) for j in range(n)]
    assert got[0][0] == plan_index([R] * n, best) == got[1][0]


def test_select_none_feasible_and_exact_boundary():
    tau = [[2.0, 3.0], [1.0, 4.0]]
    prob = make_problem([(0, 1)], tau, p=[[0.7, 0.9], [0.8, 0.6]], w=[1.0, 1.0], rho=((0.0,), (0.5,)))
    got = orc.select_range(prob, 0, 4, slo=2.9)   # min CP is 3
    assert all(c[0] == -1 and c[1] == 0 and math.isnan(c[2]) for c in got)
    # SLO exactly equal to a plan's CP is feasible (inclusive); level 1 doubles latencies
    got = orc.select_range(prob, 0, 4, slo=4.0)
    # plans: (0,0) cp 3 corr .56; (0,1) cp 6; (1,0) cp 4 corr .72; (1,1) cp 7
    assert got[0][0] == 2 and got[0][3] == 4.0
    assert got[1][0] == -1
    got = orc.select_range(prob, 0, 4, slo=6.0)
    assert got[1][0] == 0 and got[1][3] == 6.0


def test_select_ties_go_to_lowest_index():
    # duplicated implementation columns give exact twins
    p = [[0.8, 0.8, 0.7], [0.9, 0.6, 0.9]]
    prob = make_problem([(0, 1)], [[1.0, 1.0, 1.0], [1.0, 1.0, 1.0]], p=p, w=[0.5, 0.5])
    got = orc.select_range(prob, 0, 9, slo=10.0)
    assert got[0][0] == 0  # (0,0), (0,2), (1,0), (1,2) tie; lowest index 0
    got = orc.select_range(prob, 1, 8, slo=10.0)
    assert got[0][0] == 2


def test_select_monotone_in_level():
    rng = np.random.default_rng(33)
    for _ in range(10):
        prob = random_problem(rng, 4, 4, K=5, B=2)
        cps = [orc.cp(prob, orc.decode(prob, j), -1) for j in range(prob.n_plans())]
        slo = float(np.float32(np.median(cps) * 1.5))
        got = orc.select_range(prob, 0, prob.n_plans(), slo=slo)
        for a, b in zip(got, got[1:]):
            assert a[1] >= b[1]
            if b[1]:
                assert a[2] >= b[2]


def test_select_range_split_merges_exactly_and_rows_agree():
    rng = np.random.default_rng(34)
    prob = random_problem(rng, 4, 5, K=3, B=2)
    total = prob.n_plans()
    cps = [orc.cp(prob, orc.decode(prob, j), -1) for j in range(total)]
    slo = float(np.float32(np.median(cps) * 1.5))
    whole = orc.select_range(prob, 0, total, slo=slo)
    cut = total // 3
    parts = [orc.select_range(prob, 0, cut, slo=slo), orc.select_range(prob, cut, total - cut, slo=slo)]
    assert orc.merge_choices(parts) == whole
    rows = np.stack([orc.decode(prob, j) for j in range(total)]).astype(np.uint8)
    assert orc.select_rows(prob, rows, 0, slo=slo) == whole


def test_score_matches_scalar_entry_points():
    rng = np.random.default_rng(35)
    prob = random_problem(rng, 4, 4, K=3, B=2)
    prob.slo = 3.0
    corr, cp, dem, feas = orc.score_range(prob, 0, prob.n_plans())
    for j in range(prob.n_plans()):
        impl = orc.decode(prob, j)
        assert corr[j] == orc.corr(prob, impl)
        assert dem[j] == orc.demand(prob, impl)
        for k in range(3):
            assert cp[j, k] == orc.cp(prob, impl, k)
            assert bool(feas[j] >> k & 1) == (cp[j, k] <= 3.0)


# ---------------------------------------------------------------------------
# Score entry points over rows and over index lists
# ---------------------------------------------------------------------------

def _digits(radix, index):
    """Mixed-radix digits, node 0 most significant (independent of the oracle)."""
    out = []
    for r in reversed([int(x) for x in radix]):
        out.append(index % r)
        index //= r
    return out[::-1]


@pytest.mark.parametrize("seed", [36, 37, 38])
def test_score_rows_and_indices_equal_score_range(seed):
    rng = np.random.default_rng(seed)
    prob = random_problem(rng, 5, 5, K=3, B=2)
    prob.slo = 4.0
    total = prob.n_plans()
    corr, cp, dem, feas = orc.score_range(prob, 0, total)
    # rows with a stride wider than the node count; the padding bytes hold
    # values no id may take, so reading one would change the scores
    stride = prob.n_nodes + 3
    rows = np.full((total, stride), 250, np.uint8)
    for j in range(total):
        rows[j, :prob.n_nodes] = _digits(prob.radix, j)
    rc, rcp, rd, rf = orc.score_rows(prob, rows)
    assert np.array_equal(rc, corr) and np.array_equal(rcp, cp)
    assert np.array_equal(rd, dem) and np.array_equal(rf, feas)
    perm = rng.permutation(total).astype(np.uint64)
    ic, icp, idm, ifs = orc.score_indices(prob, perm)
    assert np.array_equal(ic, corr[perm]) and np.array_equal(icp, cp[perm])
    assert np.array_equal(idm, dem[perm]) and np.array_equal(ifs, feas[perm])


def test_score_rows_and_indices_on_workload_subsets():
    from paper_2607_02942_amd import workload as wl
    prob = wl.forkjoin8()
    begin, count = 123_456_789, 4096
    corr, cp, dem, feas = orc.score_range(prob, begin, count)
    rows = np.array([_digits(prob.radix, begin + j) for j in range(count)], np.uint8)
    rc, rcp, rd, rf = orc.score_rows(prob, rows)
    assert np.array_equal(rc, corr) and np.array_equal(rcp, cp)
    assert np.array_equal(rd, dem) and np.array_equal(rf, feas)
    rng = np.random.default_rng(39)
    sub = rng.permutation(count)[:1000]
    ic, icp, idm, ifs = orc.score_indices(prob, (begin + sub).astype(np.uint64))
    assert np.array_equal(ic, corr[sub]) and np.array_equal(icp, cp[sub])
    assert np.array_equal(idm, dem[sub]) and np.array_equal(ifs, feas[sub])


# ---------------------------------------------------------------------------
# The two-pass lower median that sets the stored SLOs (R-7: 1.5 x the lower
# median of the unpressured critical path over the scored plan set).  The
# stored SLOs use 24 histogram bits; the algorithm does not depend on the bit
# count, and the tests take 6 to 20 bits (a 2^24-entry histogram is slow to
# scan here)
# ---------------------------------------------------------------------------

def _sorted_lower_median(vals):
    return float(np.sort(vals)[(vals.size - 1) // 2])


def test_two_pass_median_chain4_full_space():
    from oracle import golden
    from paper_2607_02942_amd import workload as wl
    prob = wl.chain4(slo=0.0)
    total = prob.n_plans()
    got = golden.lower_median_cp0(prob, "range", total, golden.SerialPool(), 8000, bits=16)
    # a chain's unpressured CP is its durations summed in node order
    idx = np.arange(total)
    dig = np.stack(np.unravel_index(idx, tuple(int(r) for r in prob.radix)), axis=1)
    t = prob.tau.astype(np.float64)
    cp = t[0, dig[:, 0]]
    for n in range(1, prob.n_nodes):
        cp = cp + t[n, dig[:, n]]
    assert got == _sorted_lower_median(cp)
    assert total % 2 == 0
    # an odd count: the first total - 1 plans
    assert golden.lower_median_cp0(prob, "range", total - 1, golden.SerialPool(), total, bits=16) == \
        _sorted_lower_median(cp[: total - 1])


def test_two_pass_median_forkjoin8_prefix():
    from oracle import golden
    from paper_2607_02942_amd import workload as wl
    prob = wl.forkjoin8(slo=0.0)
    total = 1 << 22
    got = golden.lower_median_cp0(prob, "range", total, golden.SerialPool(), 1 << 20, bits=20)
    assert got == _sorted_lower_median(orc.cp0_values(prob, 0, total))


@pytest.mark.parametrize("count", [1 << 20, (1 << 20) + 1])
def test_two_pass_median_stream24_rows(count):
    from oracle import golden
    from paper_2607_02942_amd import workload as wl
    prob = wl.stream24(slo=0.0)
    got = golden.lower_median_cp0(prob, "rows", count, golden.SerialPool(), 1 << 19, bits=20)
    rows = wl.make_rows(count, prob.n_nodes, int(prob.radix[0]), threads=1)
    assert got == _sorted_lower_median(orc.cp0_values(prob, rows=rows))


@pytest.mark.parametrize("bits", [6, 16])
def test_two_pass_median_heavy_ties(bits):
    # integer durations: the CP takes few distinct values, so the median's
    # bucket holds many equal values (with 6 bits also many distinct ones)
    from oracle import golden
    rng = np.random.default_rng(40)
    prob = random_problem(rng, 6, 6, K=1, B=1, integer_tau=True)
    prob.rho = np.zeros((1, 1), np.float32)
    prob.backend = np.zeros_like(prob.backend)
    total = prob.n_plans()
    vals = np.array([orc.cp(prob, orc.decode(prob, j), 0) for j in range(total)])
    ref = _sorted_lower_median(vals)
    assert np.count_nonzero(vals == ref) > 10
    for count in (total, total - 1):
        got = golden.lower_median_cp0(prob, "range", count, golden.SerialPool(), max(1, count // 3), bits=bits)
        assert got == _sorted_lower_median(vals[:count])
