"""GPU parity of the objective mode (the paper's additive objective J_L,
Sec. 4.3 eq. admission-objective with Sec. 4.4 eq. variant-objective) against
the fp64 CPU oracle (oracle/objective.c), through the C-ABI.

Bar: selected indices bit-exact, every level admissible (feasible = 1); the
winner's J_k, T and D equal its fp64 values rounded to the nearest fp32 (the
library re-evaluates winners in fp64 in the definition's operation order).
Per-plan fp32 scores: |J_k(fp32) - J_k(fp64)| <= 1e-5 * A_k with A_k = the sum
over LLM nodes of the largest |u| + lambda_l T + lambda_ld L_k D (the derived
bound is (N + 6) 2^-24 A_k <= 2.2e-6 A_k at N <= 32); U and D likewise.
"""
import dataclasses
import json
import os

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import oracle as orc  # noqa: E402
from paper_2607_02942_amd import dyplan as D  # noqa: E402
from paper_2607_02942_amd import workload as wl  # noqa: E402

pytestmark = pytest.mark.gpu
RTOL = 1e-5


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    D.lib()
    torch.cuda.set_device(0)
    yield


def stream():
    return torch.cuda.current_stream()


def f32(x):
    return float(np.float32(x))


def assert_obj_choices(got, want, ctx=""):
    assert len(got) == len(want)
    for k, (g, w) in enumerate(zip(got, want)):
        assert g[0] == int(w[0]) and g[1] == 1 and int(w[1]) == 1, f"{ctx} level {k}: gpu {g} oracle {w}"
        assert g[2] == f32(w[2]) and g[3] == f32(w[3]) and g[4] == f32(w[4]), f"{ctx} level {k}: {g} vs {w}"


def select(prob, obj, sources, options=()):
    with D.Plan((prob, obj)) as plan:
        for o, v in options:
            plan.set_option(o, v)
        return plan.select(sources, stream=stream())


def util_bound(prob, obj):
    """Sum over LLM nodes of the largest |u| (a magnitude bound for U)."""
    reach = orc.obj_reach(prob, obj)
    q = prob.p.astype(np.float64)
    u = reach[:, None] * q - obj.lambda_f * prob.w[:, None].astype(np.float64) * (1 - q) \
        - obj.lambda_c * obj.cost.astype(np.float64)
    s = 0.0
    for n in range(prob.n_nodes):
        if obj.is_tool is not None and obj.is_tool[n]:
            continue
        s += np.abs(u[n, :prob.radix[n]]).max()
    return s


def with_tools(obj, n, tools):
    t = np.zeros(n, np.int32)
    t[list(tools)] = 1
    return dataclasses.replace(obj, is_tool=t)


def small_dag(n, radix, seed, edges=None):
    """A seeded random problem of n nodes (values in the paper workloads' ranges)."""
    rng = np.random.default_rng(seed)
    R = max(radix)
    if edges is None:
        edges = [(i, j) for i in range(n) for j in range(i + 1, n) if rng.random() < 0.4]
    e = np.array(edges, np.int32).reshape(-1, 2)
    return wl.Problem(n_nodes=n, edges=e, radix=np.array(radix, np.int32),
                      p=rng.uniform(0.6, 0.95, (n, R)).astype(np.float32),
                      tau=rng.lognormal(0.0, 0.5, (n, R)).astype(np.float32),
                      size=rng.choice([1.0, 2.5, 6.0], (n, R)).astype(np.float32),
                      backend=np.zeros((n, R), np.int32), w=rng.uniform(0.2, 1.0, n).astype(np.float32),
                      rho=np.zeros((1, 1), np.float32), slo=np.float32(np.inf))


# ---------------------------------------------------------------------------
# selection, enumerated sources (the prefix-shared sweep)
# ---------------------------------------------------------------------------

def test_chain4_full_space():
    prob = wl.chain4()
    obj = wl.paper_objective(prob)
    n = prob.n_plans()
    got = select(prob, obj, [D.range_source(0, 0, n)])[0]
    assert_obj_choices(got, orc.obj_select_range(prob, obj, 0, n), "chain4")


@pytest.mark.parametrize("begin,count", [(0, 1 << 20), (123457, 1000003), (429981696 - 777777, 777777),
                                         (5, 1), (144 * 1000 + 7, 143)])
def test_forkjoin8_ragged_ranges(begin, count):
    prob = wl.forkjoin8()
    obj = wl.paper_objective(prob)
    got = select(prob, obj, [D.range_source(0, begin, count)])[0]
    assert_obj_choices(got, orc.obj_select_range(prob, obj, begin, count), f"forkjoin8[{begin}+{count}]")


def test_forkjoin8_tools_weights_and_many_levels():
    prob = wl.forkjoin8()
    obj = with_tools(wl.paper_objective(prob, levels=np.linspace(0.0, 6.0, 12), lambda_l=0.4, lambda_c=0.1,
                                        effort=0.9), 8, (0, 7))
    for begin, count in ((0, 1 << 19), (3 * 12 ** 6 + 11, 600011)):
        got = select(prob, obj, [D.range_source(0, begin, count)])[0]
        assert_obj_choices(got, orc.obj_select_range(prob, obj, begin, count), f"tools[{begin}+{count}]")


@pytest.mark.parametrize("begin,count", [(0, 1 << 21), ((1 << 32) - 999999, 999999)])
def test_layered10_ranges(begin, count):
    prob = wl.layered10()
    obj = wl.paper_objective(prob)
    got = select(prob, obj, [D.range_source(0, begin, count)])[0]
    assert_obj_choices(got, orc.obj_select_range(prob, obj, begin, count), f"layered10[{begin}+{count}]")


@pytest.mark.parametrize("n,radix,seed", [(1, [7], 1), (2, [5, 9], 2), (3, [4, 1, 6], 3), (5, [3, 4, 2, 5, 3], 4),
                                          (6, [12] * 6, 5), (12, [3] * 12, 6)])
def test_small_dags_full_space(n, radix, seed):
    prob = small_dag(n, radix, seed)
    rng = np.random.default_rng(seed + 100)
    obj = wl.Objective(cost=(prob.tau * prob.size).astype(np.float32),
                       levels=rng.uniform(0, 4, 1 + seed % 5).astype(np.float32),
                       lambda_f=float(rng.uniform(-1, 2)), lambda_c=float(rng.uniform(-0.1, 0.2)),
                       lambda_l=float(rng.uniform(0, 0.5)), lambda_ld=float(rng.uniform(0, 0.3)),
                       beta=float(rng.uniform(-1, 2)), effort=float(rng.uniform(0, 1)),
                       is_tool=(rng.random(n) < 0.3).astype(np.int32))
    total = int(np.prod(radix))
    got = select(prob, obj, [D.range_source(0, 0, total)])[0]
    assert_obj_choices(got, orc.obj_select_range(prob, obj, 0, total), f"dag{n}")


@pytest.mark.parametrize("n,radix,seed", [(3, [4, 1, 6], 3), (5, [3, 4, 2, 5, 3], 4), (6, [12] * 6, 5),
                                          (12, [3] * 12, 6), (8, [5] * 8, 8)])
def test_generated_sweep_small_dags(n, radix, seed):
    # DY_OPT_JIT 2: the sweep generated for the DAG on every RANGE source
    prob = small_dag(n, radix, seed)
    rng = np.random.default_rng(seed + 100)
    obj = wl.Objective(cost=(prob.tau * prob.size).astype(np.float32),
                       levels=rng.uniform(0, 4, 1 + seed % 5).astype(np.float32),
                       lambda_f=float(rng.uniform(-1, 2)), lambda_c=float(rng.uniform(-0.1, 0.2)),
                       lambda_l=float(rng.uniform(0, 0.5)), lambda_ld=float(rng.uniform(0, 0.3)),
                       beta=float(rng.uniform(-1, 2)), effort=float(rng.uniform(0, 1)),
                       is_tool=(rng.random(n) < 0.3).astype(np.int32))
    total = int(np.prod(radix))
    begin, count = total // 9, total - total // 9 - total // 11
    with D.Plan((prob, obj)) as plan:
        plan.set_option(D.DY_OPT_JIT, 2)
        for call in range(2):
            got = plan.select([D.range_source(0, begin, count)], stream=stream())[0]
            assert_obj_choices(got, orc.obj_select_range(prob, obj, begin, count), f"dag{n} call {call}")


@pytest.mark.parametrize("begin,count", [(123457, 1000003), (429981696 - 777777, 777777)])
def test_forkjoin8_generated_sweep(begin, count):
    prob = wl.forkjoin8()
    obj = with_tools(wl.paper_objective(prob, levels=np.linspace(0.0, 6.0, 12), lambda_l=0.4), 8, (0, 7))
    with D.Plan((prob, obj)) as plan:
        plan.set_option(D.DY_OPT_JIT, 2)
        got = plan.select([D.range_source(0, begin, count)], stream=stream())[0]
    assert_obj_choices(got, orc.obj_select_range(prob, obj, begin, count), f"forkjoin8[{begin}+{count}] generated")


@pytest.mark.parametrize("jit", [0, 2])
@pytest.mark.parametrize("case", ["batch6", "lambda_l0", "negative", "two_sinks", "x_sink", "ragged", "subnormal"])
def test_shifted_thresholds_both_sweeps(case, jit):
    # DY_OPT_JIT 0: the library sweep of a 6-node problem with 12
    # implementations of node y tests each row's fma(-lambda_l, M, ux) against
    # bin thresholds lowered ahead by every implementation of y (ydiv_jobs
    # counts the source); DY_OPT_JIT 2: the sweep generated for the DAG, with
    # the same test and the offsets as literals.  batch6 DAGs have one sink; two_sinks adds a second
    # one (the path into it bounds T from below), x_sink leaves x without a
    # successor; negative makes most utilities negative (negative
    # thresholds); lambda_l0 drops the latency term; ragged cuts blocks;
    # subnormal makes every quality, hence every utility and G, subnormal
    # in fp32 (the bound's subnormal term), with a subnormal lambda_l.
    begin, count = 0, 12 ** 6
    if case in ("two_sinks", "x_sink"):
        edges = [(0, 1), (1, 2), (2, 3), (0, 4), (4, 5)] if case == "two_sinks" else \
                [(0, 1), (1, 2), (2, 3), (3, 5), (0, 4)]
        prob = small_dag(6, [12] * 6, 31 if case == "two_sinks" else 32, edges)
        obj = wl.paper_objective(prob, lambda_l=0.3)
    else:
        prob = wl.batch6_request(11)
        w = {"lambda_l0": dict(lambda_l=0.0), "negative": dict(lambda_c=2.0, lambda_l=0.3),
             "subnormal": dict(lambda_f=0.0, lambda_c=0.0, lambda_l=1e-44)}.get(case, {})
        if case == "subnormal":
            prob = dataclasses.replace(prob, p=(prob.p.astype(np.float64) * 1e-39).astype(np.float32))
        obj = wl.paper_objective(prob, **w)
        if case == "ragged":
            begin, count = 777, 3 * 12 ** 5 + 55
    with D.Plan((prob, obj)) as plan:
        plan.set_option(D.DY_OPT_JIT, jit)
        got = plan.select([D.range_source(0, begin, count)], stream=stream())[0]
        assert plan.stats().ydiv_jobs == 1
        assert plan.stats().generated_jobs == (1 if jit else 0)
    assert_obj_choices(got, orc.obj_select_range(prob, obj, begin, count), f"{case}[{begin}+{count}] jit {jit}")


def test_batch_mixed_with_corr_selection():
    # objective and corr / SLO problems in one call: both sweep groups run together
    probs = [wl.batch6_request(r) for r in range(4)]
    objs = [wl.paper_objective(p) for p in probs]
    items = [probs[0], (probs[1], objs[1]), probs[2], (probs[3], objs[3])]
    with D.Plan(items) as plan:
        got = plan.select([D.range_source(r, 0, 12 ** 6) for r in range(4)], stream=stream())
    for r in (1, 3):
        assert_obj_choices(got[r], orc.obj_select_range(probs[r], objs[r], 0, 12 ** 6), f"batch[{r}]")
    for r in (0, 2):
        want = orc.select_range(probs[r], 0, 12 ** 6)
        for g, w in zip(got[r], want):
            assert (g[0], g[1]) == (int(w[0]), int(w[1])), f"corr batch[{r}]"


# ---------------------------------------------------------------------------
# ties, overflow recovery and the exhaustive path
# ---------------------------------------------------------------------------

def test_exact_ties_go_to_the_lowest_index():
    # implementations 2k and 2k+1 identical in every table: each winner has
    # tie partners, and the lowest index must win
    prob = wl.chain4().copy()
    for a in ("p", "tau", "size", "backend"):
        t = getattr(prob, a).copy()
        t[:, 1::2] = t[:, 0::2]
        setattr(prob, a, t)
    obj = wl.paper_objective(prob)
    n = prob.n_plans()
    want = orc.obj_select_range(prob, obj, 0, n)
    got = select(prob, obj, [D.range_source(0, 0, n)])[0]
    assert_obj_choices(got, want, "ties")
    for c in got:
        impl = [(c[0] // 12 ** (3 - i)) % 12 for i in range(4)]
        assert all(x % 2 == 0 for x in impl), impl


def test_all_plans_tie_overflow_then_exhaustive():
    # every implementation identical: all plans tie at every level, the candidate
    # list overflows, reseeding cannot help, the exhaustive fp64 path decides
    prob = wl.chain4().copy()
    for a in ("p", "tau", "size"):
        t = getattr(prob, a).copy()
        t[:] = t[:, :1]
        setattr(prob, a, t)
    obj = wl.paper_objective(prob)
    begin, count = 777, 5000
    with D.Plan((prob, obj)) as plan:
        plan.set_option(D.DY_OPT_CAND_CAPACITY, 64)
        got = plan.select([D.range_source(0, begin, count)], stream=stream())[0]
        assert plan.stats().fallbacks == obj.n_levels
    assert_obj_choices(got, orc.obj_select_range(prob, obj, begin, count), "all tie")
    assert all(c[0] == begin for c in got)


def test_small_candidate_capacity_reseeds():
    prob = wl.forkjoin8()
    obj = wl.paper_objective(prob)
    begin, count = 1000, 1 << 20
    want = orc.obj_select_range(prob, obj, begin, count)
    with D.Plan((prob, obj)) as plan:
        plan.set_option(D.DY_OPT_CAND_CAPACITY, 16)
        plan.set_option(D.DY_OPT_SAMPLE_STRIDE, 1 << 20)  # a poor seed: many candidates on the first pass
        got = plan.select([D.range_source(0, begin, count)], stream=stream())[0]
    assert_obj_choices(got, want, "reseed")


def test_force_fp64_matches():
    prob = wl.forkjoin8()
    obj = with_tools(wl.paper_objective(prob), 8, (3,))
    begin, count = 4242, 300000
    want = orc.obj_select_range(prob, obj, begin, count)
    got = select(prob, obj, [D.range_source(0, begin, count)], options=((D.DY_OPT_FORCE_FP64, 1),))[0]
    assert_obj_choices(got, want, "fp64")


def test_graph_replay_matches():
    prob = wl.forkjoin8()
    obj = wl.paper_objective(prob)
    src = [D.range_source(0, 99, 1 << 20)]
    want = orc.obj_select_range(prob, obj, 99, 1 << 20)
    with D.Plan((prob, obj)) as plan:
        for rep in range(4):
            assert_obj_choices(plan.select(src, stream=stream())[0], want, f"replay {rep}")


# ---------------------------------------------------------------------------
# ROWS sources (the generic per-plan path)
# ---------------------------------------------------------------------------

def test_stream24_rows():
    prob = wl.stream24()
    obj = with_tools(wl.paper_objective(prob), 24, (0, 5, 23))
    n = 300007
    rows = wl.make_rows(n, 24, 36, row_begin=4321)
    want = orc.obj_select_rows(prob, obj, rows, index_base=4321)
    with D.Plan((prob, obj)) as plan:
        d = torch.from_numpy(rows).cuda()
        got = plan.select([D.rows_source(0, d, n, 24, 4321)], stream=stream())[0]
        assert_obj_choices(got, want, "stream24 rows")
        padded = np.zeros((n, 27), np.uint8)
        padded[:, :24] = rows
        dp = torch.from_numpy(padded).cuda()
        got = plan.select([D.rows_source(0, dp, n, 27, 4321)], stream=stream())[0]
        assert_obj_choices(got, want, "stream24 rows, odd stride")


def test_rows_bad_id_is_an_error():
    prob = wl.chain4()
    obj = wl.paper_objective(prob)
    rows = np.zeros((1000, 4), np.uint8)
    rows[517, 2] = 12
    with D.Plan((prob, obj)) as plan:
        d = torch.from_numpy(rows).cuda()
        with pytest.raises(D.DyplanError):
            plan.select([D.rows_source(0, d, 1000, 4)], stream=stream())


# ---------------------------------------------------------------------------
# per-plan scores
# ---------------------------------------------------------------------------

def check_scores(prob, obj, U, T, Dd, J, gu, gj, gd, gf):
    K = obj.n_levels
    su = util_bound(prob, obj)
    m = obj.lambda_ld * obj.levels.astype(np.float64)
    assert np.all(np.abs(gu - U) <= RTOL * su)
    assert np.all(np.abs(gd - Dd) <= RTOL * Dd.max())
    for k in range(K):
        A = su + obj.lambda_l * T + m[k] * Dd
        err = np.abs(gj[:, k].astype(np.float64) - J[:, k])
        assert np.all(err <= RTOL * A), (k, float((err / A).max()))
    assert np.all(gf == (1 << K) - 1)


@pytest.mark.parametrize("jit", [1, 0])
@pytest.mark.parametrize("n", [1, 2, 3, 5, 8, 11, 13, 16, 17])
def test_score_node_counts(n, jit):
    # a range of 32-bit plan indices: the row kernel with either JIT option
    rng = np.random.default_rng(70 + n)
    r = max(2, min(12, int(round(20000 ** (1.0 / n)))))
    prob = small_dag(n, [int(x) for x in rng.integers(1, r + 1, n)], 700 + n)
    obj = wl.paper_objective(prob, levels=(0.0, 0.5, 1.5, 3.0))
    if n > 2:
        obj = with_tools(obj, n, (n // 2,))
    K = obj.n_levels
    cnt = prob.n_plans()
    with D.Plan((prob, obj)) as plan:
        plan.set_option(D.DY_OPT_JIT, jit)
        u = torch.empty(cnt, dtype=torch.float32, device="cuda")
        j = torch.empty(cnt, K, dtype=torch.float32, device="cuda")
        d = torch.empty(cnt, dtype=torch.float32, device="cuda")
        f = torch.empty(cnt, dtype=torch.int32, device="cuda")
        plan.score(D.range_source(0, 0, cnt), u, j, d, f, stream=stream())
        torch.cuda.synchronize()
    U, T, Dd, J = orc.obj_score(prob, obj, 0, cnt)
    check_scores(prob, obj, U, T, Dd, J, u.cpu().numpy(), j.cpu().numpy(), d.cpu().numpy(),
                 f.cpu().numpy().astype(np.uint32))


def test_score_range_and_rows():
    prob = wl.forkjoin8()
    obj = with_tools(wl.paper_objective(prob, levels=(0.0, 0.5, 1.5, 3.0)), 8, (7,))
    K = obj.n_levels
    cnt = 200003
    with D.Plan((prob, obj)) as plan:
        u = torch.empty(cnt, dtype=torch.float32, device="cuda")
        j = torch.empty(cnt, K, dtype=torch.float32, device="cuda")
        d = torch.empty(cnt, dtype=torch.float32, device="cuda")
        f = torch.empty(cnt, dtype=torch.int32, device="cuda")
        plan.score(D.range_source(0, 31337, cnt), u, j, d, f, stream=stream())
        torch.cuda.synchronize()
        U, T, Dd, J = orc.obj_score(prob, obj, 31337, cnt)
        check_scores(prob, obj, U, T, Dd, J, u.cpu().numpy(), j.cpu().numpy(), d.cpu().numpy(),
                     f.cpu().numpy().astype(np.uint32))
        rows = wl.make_rows(cnt, 8, 12, row_begin=99)
        dr = torch.from_numpy(rows).cuda()
        plan.score(D.rows_source(0, dr, cnt, 8), u, j, d, f, stream=stream())
        torch.cuda.synchronize()
        U, T, Dd, J = orc.obj_score(prob, obj, rows=rows)
        check_scores(prob, obj, U, T, Dd, J, u.cpu().numpy(), j.cpu().numpy(), d.cpu().numpy(),
                     f.cpu().numpy().astype(np.uint32))


def test_rows_generated_kernel_matches_generic_path():
    # the DAG-specialised rows kernels and the generic per-plan path agree
    prob = wl.stream24()
    obj = with_tools(wl.paper_objective(prob, levels=(0.0, 0.7, 1.5, 3.0, 6.0)), 24, (2, 11))
    n = 1 << 20
    rows = wl.make_rows(n, 24, 36, row_begin=777)
    want = orc.obj_select_rows(prob, obj, rows, index_base=5)
    d = torch.from_numpy(rows).cuda()
    for jit in (1, 0):
        with D.Plan((prob, obj)) as plan:
            plan.set_option(D.DY_OPT_JIT, jit)
            got = plan.select([D.rows_source(0, d, n, 24, 5)], stream=stream())[0]
        assert_obj_choices(got, want, f"rows jit={jit}")


def test_score_odd_levels_unaligned_output():
    # three levels (rows of 12 bytes) into a CP output that is not 16-byte
    # aligned, a range that starts and ends inside rows of the last node
    prob = wl.forkjoin8()
    obj = with_tools(wl.paper_objective(prob, levels=(0.0, 0.7, 2.0)), 8, (3,))
    K = obj.n_levels
    begin, cnt = 1000005, 123457
    with D.Plan((prob, obj)) as plan:
        u = torch.empty(cnt, dtype=torch.float32, device="cuda")
        buf = torch.empty(cnt * K + 1, dtype=torch.float32, device="cuda")
        j = buf[1:].view(cnt, K)
        d = torch.empty(cnt, dtype=torch.float32, device="cuda")
        f = torch.empty(cnt, dtype=torch.int32, device="cuda")
        plan.score(D.range_source(0, begin, cnt), u, j, d, f, stream=stream())
        torch.cuda.synchronize()
    U, T, Dd, J = orc.obj_score(prob, obj, begin, cnt)
    check_scores(prob, obj, U, T, Dd, J, u.cpu().numpy(), j.cpu().numpy(), d.cpu().numpy(),
                 f.cpu().numpy().astype(np.uint32))


# ---------------------------------------------------------------------------
# local-search seeds under the objective
# ---------------------------------------------------------------------------

def _climb_select(prob, obj, total, climb):
    with D.Plan((prob, obj)) as plan:
        plan.set_option(D.DY_OPT_CLIMB, climb)
        got = plan.select([D.range_source(0, 0, total)], stream=stream())[0]
        return got, plan.stats().candidates


@pytest.mark.parametrize("seed", range(6))
def test_climb_small_dags_full_space(seed):
    # DY_OPT_CLIMB 2: every whole-space source of at most 8 nodes seeds each
    # level from a local search on the fp32 estimate of J_k; the choices equal
    # the oracle's with and without it and the candidate list never grows.
    # Seed 5 has lambda_l = 0 (the longest path does not count).
    rng = np.random.default_rng(700 + seed)
    n = int(rng.integers(2, 9))
    radix = [int(x) for x in rng.integers(1, 7, n)]
    prob = small_dag(n, radix, 900 + seed)
    obj = wl.Objective(cost=(prob.tau * prob.size).astype(np.float32),
                       levels=np.sort(rng.uniform(0, 4, 1 + seed % 4)).astype(np.float32),
                       lambda_f=float(rng.uniform(-1, 2)), lambda_c=float(rng.uniform(-0.1, 0.2)),
                       lambda_l=float(rng.uniform(0, 0.5)) if seed != 5 else 0.0,
                       lambda_ld=float(rng.uniform(0, 0.3)),
                       beta=float(rng.uniform(-1, 2)), effort=float(rng.uniform(0, 1)),
                       is_tool=(rng.random(n) < 0.3).astype(np.int32))
    total = int(np.prod(radix))
    want = orc.obj_select_range(prob, obj, 0, total)
    off, c_off = _climb_select(prob, obj, total, 0)
    on, c_on = _climb_select(prob, obj, total, 2)
    assert_obj_choices(off, want, f"dag{n} no climb")
    assert_obj_choices(on, want, f"dag{n} climb")
    assert c_on <= c_off, (c_on, c_off)


def test_batch6_objective_graph_replays():
    # 1,024 requests under J_L, repeated (graph replays): every call against
    # the stored oracle selections, the same candidate count each time
    path = os.path.join(os.path.dirname(__file__), "golden", "select_batch6_objective.json")
    want = [[(c[0], c[1], float(c[2]), float(c[3]), float(c[4])) for c in ch] for ch in json.load(open(path))["choices"]]
    nreq = 1024
    probs = wl.batch6(nreq)
    items = [(p, wl.paper_objective(p)) for p in probs]
    srcs = [D.range_source(r, 0, 12 ** 6) for r in range(nreq)]
    cands = []
    with D.Plan(items) as plan:
        for call in range(3):
            got = plan.select(srcs, stream=stream())
            cands.append(plan.stats().candidates)
            for r in range(nreq):
                assert_obj_choices(got[r], want[r], f"batch6 objective [{r}] call {call}")
    assert len(set(cands)) == 1, cands


def test_climb_batch6_objective_golden():
    # 256 of batch6's requests under J_L, with and without the local search,
    # against the stored oracle selections; a call mixing both objectives
    # launches both searches
    path = os.path.join(os.path.dirname(__file__), "golden", "select_batch6_objective.json")
    want = [[(c[0], c[1], float(c[2]), float(c[3]), float(c[4])) for c in ch] for ch in json.load(open(path))["choices"]]
    nreq = 256
    probs = wl.batch6(nreq)
    items = [(p, wl.paper_objective(p)) for p in probs]
    srcs = [D.range_source(r, 0, 12 ** 6) for r in range(nreq)]
    res = {}
    for climb in (0, 2):
        with D.Plan(items) as plan:
            plan.set_option(D.DY_OPT_CLIMB, climb)
            res[climb] = (plan.select(srcs, stream=stream()), plan.stats().candidates)
    for r in range(nreq):
        for climb in (0, 2):
            assert_obj_choices(res[climb][0][r], want[r], f"batch6 objective [{r}], climb {climb}")
    assert res[2][1] < res[0][1], (res[2][1], res[0][1])
    mixed = [probs[0], items[1], probs[2], items[3]]
    with D.Plan(mixed) as plan:
        plan.set_option(D.DY_OPT_CLIMB, 2)
        got = plan.select(srcs[:4], stream=stream())
    for r in (1, 3):
        assert_obj_choices(got[r], want[r], f"mixed [{r}]")
    for r in (0, 2):
        oc = orc.select_range(probs[r], 0, 12 ** 6)
        for g, w in zip(got[r], oc):
            assert (g[0], g[1]) == (int(w[0]), int(w[1])), f"mixed corr [{r}]"


@pytest.mark.parametrize("objective", [False, True])
@pytest.mark.parametrize("shape", ["npre9", "big"])
def test_library_sweep_odd_prefix_and_64bit_blocks(shape, objective):
    # The library sweep with R_y = 12 on 256 bins (thresholds divided ahead
    # by y's factor, or lowered by y's terms) for a prefix length without an
    # unrolled variant (nine prefix nodes: the recurrence in LDS columns) and
    # for block indices above 2^32 (64-bit digits), each on a ragged range
    # near the end of the space, in corr / SLO mode and under J_L.
    radix = [7] * 9 + [5, 12] if shape == "npre9" else [9] * 11 + [5, 12]
    n = len(radix)
    prob = small_dag(n, radix, 77 if shape == "npre9" else 78)
    total = int(np.prod(radix, dtype=np.float64))
    count = 4_000_037
    begin = total - count - 12345
    if objective:
        obj = wl.paper_objective(prob, lambda_l=0.2)
        item = (prob, obj)
        want = orc.obj_select_range(prob, obj, begin, count)
    else:
        t = prob.tau.astype(np.float64)
        prob = dataclasses.replace(prob, rho=np.array([[0.0], [0.3], [0.6]], np.float32),
                                   slo=np.float32(0.8 * n * t.mean()))
        item = prob
        want = orc.select_range(prob, begin, count)
    with D.Plan(item) as plan:
        plan.set_option(D.DY_OPT_JIT, 0)
        got = plan.select([D.range_source(0, begin, count)], stream=stream())[0]
        assert plan.stats().ydiv_jobs == 1
    ctx = f"{shape} objective={objective}"
    if objective:
        assert_obj_choices(got, want, ctx)
    else:
        for k, (g, w) in enumerate(zip(got, want)):
            assert (g[0], g[1]) == (int(w[0]), int(w[1])), f"{ctx} level {k}: gpu {g} oracle {w}"
            if int(w[1]):
                assert g[2] == f32(w[2]) and g[3] == f32(w[3]) and g[4] == f32(w[4]), f"{ctx} level {k}"
