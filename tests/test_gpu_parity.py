"""GPU parity: the HIP library (through its C-ABI) against the fp64 CPU oracle.

Bar: selected indices and feasibility flags bit-exact; a winner's corr / cp /
demand equal its fp64 values rounded to the nearest fp32 (the library
re-evaluates winners in fp64); per-plan fp32 scores within 1e-5 relative
(the derived bound is 2N * 2^-24 <= 3.9e-6 for N <= 32); feasibility bits exact.
Small and ragged ranges are checked against the oracle run live; full-size
workloads against the oracle's stored selections (oracle/golden.py).
"""
import json
import math
import os

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import oracle as orc  # noqa: E402
from paper_2607_02942_amd import dyplan as D  # noqa: E402
from paper_2607_02942_amd import workload as wl  # noqa: E402

pytestmark = pytest.mark.gpu
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
RTOL = 1e-5


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    D.lib()  # fails loudly if the HIP library is not built
    torch.cuda.set_device(0)
    yield


def stream():
    return torch.cuda.current_stream()


def f32(x):
    return float(np.float32(x))


def assert_choices(got, want, ctx=""):
    assert len(got) == len(want)
    for k, (g, w) in enumerate(zip(got, want)):
        assert (g[0], g[1]) == (int(w[0]), int(w[1])), f"{ctx} level {k}: gpu {g} oracle {w}"
        if int(w[1]):
            assert g[2] == f32(w[2]) and g[3] == f32(w[3]) and g[4] == f32(w[4]), f"{ctx} level {k}: {g} vs {w}"
        else:
            assert g[0] == -1 and math.isnan(g[2]) and math.isnan(g[3]) and math.isnan(g[4])


def golden(name):
    path = os.path.join(GOLDEN, f"select_{name}.json")
    if not os.path.exists(path):
        pytest.skip(f"{path} not generated")
    g = json.load(open(path))
    conv = lambda ch: [(c[0], c[1], float(c[2]), float(c[3]), float(c[4])) for c in ch]
    if name == "batch6":
        return g, [conv(ch) for ch in g["choices"]]
    return g, conv(g["choices"])


def select(prob_or_plan, sources):
    if isinstance(prob_or_plan, D.Plan):
        return prob_or_plan.select(sources, stream=stream())
    with D.Plan(prob_or_plan) as plan:
        return plan.select(sources, stream=stream())


# ---------------------------------------------------------------------------
# enumerated path, live oracle
# ---------------------------------------------------------------------------

def test_chain4_full_space():
    prob = wl.chain4()
    n = prob.n_plans()
    assert_choices(select(prob, [D.range_source(0, 0, n)])[0], orc.select_range(prob, 0, n), "chain4")


@pytest.mark.parametrize("begin,count", [(0, 1 << 20), (123457, 1000003), (429981696 - 777777, 777777),
                                         (5, 1), (144 * 1000 + 7, 143)])
def test_forkjoin8_ragged_ranges(begin, count):
    prob = wl.forkjoin8()
    got = select(prob, [D.range_source(0, begin, count)])[0]
    assert_choices(got, orc.select_range(prob, begin, count), f"forkjoin8[{begin}+{count}]")


@pytest.mark.parametrize("begin,count", [(0, 1 << 21), (2176782336 - 654321, 1300000), ((1 << 32) - 999999, 999999)])
def test_layered10_ranges(begin, count):
    prob = wl.layered10()
    got = select(prob, [D.range_source(0, begin, count)])[0]
    assert_choices(got, orc.select_range(prob, begin, count), f"layered10[{begin}+{count}]")


@pytest.mark.parametrize("n_src", [1, 64, 65])
def test_results_written_to_host_or_copied_back(n_src):
    # up to 64 sources the certification writes the choices straight to host
    # memory and the call waits on completion words; above, they are copied
    # back after the stream.  Repeated calls replay the captured graph.
    prob = wl.chain4()
    rng = np.random.default_rng(n_src)
    begins = rng.integers(0, 20000, n_src)
    counts = rng.integers(1, 737, n_src)
    srcs = [D.range_source(0, int(b), int(min(c, 20736 - b))) for b, c in zip(begins, counts)]
    want = [orc.select_range(prob, s.begin, s.count) for s in srcs]
    with D.Plan(prob) as plan:
        for call in range(3):
            got = plan.select(srcs, stream=stream())
            for q, (g, w) in enumerate(zip(got, want)):
                assert_choices(g, w, f"{n_src} sources, call {call}, source {q}")


def test_batch6_first_requests_live():
    probs = [wl.batch6_request(r) for r in range(6)]
    with D.Plan(probs) as plan:
        got = plan.select([D.range_source(r, 0, 12 ** 6) for r in range(6)], stream=stream())
    for r in range(6):
        assert_choices(got[r], orc.select_range(probs[r], 0, 12 ** 6), f"batch6[{r}]")


def test_stream24_rows_live_and_strides():
    prob = wl.stream24()
    n = 300007
    rows = wl.make_rows(n, 24, 36, row_begin=12345)
    want = orc.select_rows(prob, rows, index_base=12345)
    with D.Plan(prob) as plan:
        d = torch.from_numpy(rows).cuda()
        got = plan.select([D.rows_source(0, d, n, 24, 12345)], stream=stream())[0]
        assert_choices(got, want, "stream24 rows")
        # padded stride (word loads) and odd stride (byte loads) give the same answer
        for stride in (32, 27):
            padded = np.zeros((n, stride), np.uint8)
            padded[:, :24] = rows
            dp = torch.from_numpy(padded).cuda()
            got = plan.select([D.rows_source(0, dp, n, stride, 12345)], stream=stream())[0]
            assert_choices(got, want, f"stream24 stride {stride}")


# ---------------------------------------------------------------------------
# full sizes against stored oracle selections
# ---------------------------------------------------------------------------

def test_forkjoin8_full_golden():
    g, want = golden("forkjoin8")
    prob = wl.forkjoin8()
    assert prob.slo == g["slo"]
    with D.Plan(prob) as plan:
        got = plan.select([D.range_source(0, 0, 12 ** 8)], stream=stream())[0]
        # the generated sweep on 256 bins, thresholds divided ahead by y's factor
        assert plan.stats().ydiv_jobs == 1
    assert_choices(got, want, "forkjoin8 full")


def test_layered10_full_golden():
    g, want = golden("layered10")
    prob = wl.layered10()
    assert prob.slo == g["slo"]
    assert_choices(select(prob, [D.range_source(0, 0, 1 << 32)])[0], want, "layered10 full")


def test_batch6_full_golden():
    g, want = golden("batch6")
    probs = wl.batch6()
    with D.Plan(probs) as plan:
        got = plan.select([D.range_source(r, 0, 12 ** 6) for r in range(wl.N_BATCH)], stream=stream())
        # the library sweep on 256 bins, R_y = 12: thresholds divided ahead by y's factor
        assert plan.stats().ydiv_jobs == wl.N_BATCH
    for r in range(wl.N_BATCH):
        assert_choices(got[r], want[r], f"batch6[{r}]")


def test_batch6_graph_replays():
    # Repeated calls of the 4,096 sources replay the captured graph of the
    # call (local search, table, sweep, certification, copy-out): every call
    # gives the stored selections and the same candidate count.
    g, want = golden("batch6")
    probs = wl.batch6()
    srcs = [D.range_source(r, 0, 12 ** 6) for r in range(wl.N_BATCH)]
    cands = []
    with D.Plan(probs) as plan:
        for call in range(4):
            got = plan.select(srcs, stream=stream())
            cands.append(plan.stats().candidates)
            for r in range(wl.N_BATCH):
                assert_choices(got[r], want[r], f"batch6[{r}] call {call}")
    assert len(set(cands)) == 1, cands


def test_stream24_full_golden():
    g, want = golden("stream24")
    prob = wl.stream24()
    assert prob.slo == g["slo"]
    n = wl.STREAM_ROWS
    rows = wl.make_rows(n, 24, 36)
    d = torch.from_numpy(rows).cuda()
    del rows
    with D.Plan(prob) as plan:
        got = plan.select([D.rows_source(0, d, n, 24, 0)], stream=stream())[0]
    assert_choices(got, want, "stream24 full")


# ---------------------------------------------------------------------------
# per-plan scores
# ---------------------------------------------------------------------------

def run_score(plan, src, n, K):
    corr = torch.empty(n, dtype=torch.float32, device="cuda")
    cp = torch.empty(n, K, dtype=torch.float32, device="cuda")
    dem = torch.empty(n, dtype=torch.float32, device="cuda")
    feas = torch.empty(n, dtype=torch.int32, device="cuda")
    plan.score(src, corr, cp, dem, feas, stream=stream())
    torch.cuda.synchronize()
    return corr.cpu().numpy(), cp.cpu().numpy(), dem.cpu().numpy(), feas.cpu().numpy().view(np.uint32)


def assert_scores(got, want, ctx):
    gc, gcp, gd, gf = got
    oc, ocp, od, of = want
    off = np.flatnonzero(~np.isclose(gc, oc, rtol=RTOL, atol=0) | (np.isnan(gc) != np.isnan(oc)))
    assert off.size == 0, f"{ctx}: corr differs at {off[:10].tolist()} ({off.size}): gpu {gc[off[:5]]} oracle {oc[off[:5]]}"
    np.testing.assert_allclose(gc, oc, rtol=RTOL, atol=0, err_msg=ctx)
    np.testing.assert_allclose(gcp, ocp, rtol=RTOL, atol=0, err_msg=ctx)
    np.testing.assert_allclose(gd, od, rtol=RTOL, atol=0, err_msg=ctx)
    assert (gf == of).all(), ctx


@pytest.mark.parametrize("name,begin,count", [("chain4", 0, 20736), ("forkjoin8", 98765, 200003),
                                              ("layered10", (1 << 32) - 100003, 100003)])
def test_score_ranges(name, begin, count):
    prob = wl.by_name(name)
    with D.Plan(prob) as plan:
        got = run_score(plan, D.range_source(0, begin, count), count, prob.n_levels)
    assert_scores(got, orc.score_range(prob, begin, count), name)


def wide_last_problem(rng, n, K, ry):
    # nodes 0..n-2 of radix 1..4, the last node of radix ry; uniform pressure
    radix = np.concatenate([rng.integers(1, 5, size=n - 1), [ry]]).astype(np.int32)
    R = int(radix.max())
    edges = np.array([(i, j) for i in range(n) for j in range(i + 1, n) if rng.random() < 0.4],
                     np.int32).reshape(-1, 2)
    prob = wl.Problem(n_nodes=n, edges=edges, radix=radix, p=rng.uniform(0.4, 1.0, (n, R)).astype(np.float32),
                      tau=rng.lognormal(0, 0.6, (n, R)).astype(np.float32),
                      size=rng.choice([0.5, 1, 2.5, 6], (n, R)).astype(np.float32),
                      backend=rng.integers(0, 2, (n, R)).astype(np.int32), w=rng.uniform(0, 1, n).astype(np.float32),
                      rho=np.repeat(np.sort(rng.uniform(0, 0.9, K))[:, None], 2, axis=1).astype(np.float32), slo=0.0)
    prob.slo = f32(np.quantile(orc.cp0_values(prob, 0, prob.n_plans()), 0.5) * 1.3)
    return prob


@pytest.mark.parametrize("K", [1, 3, 4, 6, 8, 13, 32])
def test_score_row_shapes(K):
    # RANGE scores go by rows of the last node's implementations, the K
    # per-level values of a wave's plans stored lane-contiguously: level counts
    # with and without 16-byte rows, a CP output that is not 16-byte aligned,
    # ranges that start and end inside a row, last nodes with fewer and more
    # implementations than a wave's 64 plans
    rng = np.random.default_rng(4200 + K)
    for trial, ry in enumerate([1, 7, 64, 150]):
        prob = wide_last_problem(rng, int(rng.integers(2, 6)), K, ry)
        total = prob.n_plans()
        begin = int(rng.integers(0, max(1, total // 6)))
        count = max(1, int(total - begin - rng.integers(0, max(1, total // 6))))
        ctx = f"K {K}, last radix {ry}, plans [{begin}, {begin + count})"
        with D.Plan(prob) as plan:
            got = run_score(plan, D.range_source(0, begin, count), count, K)
            buf = torch.empty(count * K + 1, dtype=torch.float32, device="cuda")
            cp = buf[1:].view(count, K)  # 4-byte aligned only
            plan.score(D.range_source(0, begin, count), None, cp, None, None, stream=stream())
            torch.cuda.synchronize()
        want = orc.score_range(prob, begin, count)
        assert_scores(got, want, ctx)
        np.testing.assert_allclose(cp.cpu().numpy(), want[1], rtol=RTOL, atol=0, err_msg=ctx + ", unaligned cp")


@pytest.mark.parametrize("jit", [1, 0])
@pytest.mark.parametrize("n", list(range(1, 18)) + [20, 24, 32])
def test_score_every_node_count(n, jit):
    # ranges of 32-bit plan indices take the row kernel whatever the node
    # count and the JIT option (the generated kernels serve rows and the
    # selection); whole plan spaces of up to ~2^17 plans, else 2^17 plans at
    # a random offset
    rng = np.random.default_rng(900 + n)
    rmax = max(2, min(12, int(round(30000 ** (1.0 / n)))))
    if n <= 17:
        prob = tiny_problem(rng, n, rmax, 8, 2, True)
        total = prob.n_plans()
        begin = int(rng.integers(0, max(1, total // 7)))
        count = total - begin
    else:
        prob = tiny_problem_large(rng, n, 8)
        total = prob.n_plans()
        count = min(total, 1 << 17)
        begin = int(rng.integers(0, total - count + 1))
    with D.Plan(prob) as plan:
        plan.set_option(D.DY_OPT_JIT, jit)
        got = run_score(plan, D.range_source(0, begin, count), count, prob.n_levels)
    assert_scores(got, orc.score_range(prob, begin, count), f"{n} nodes, jit {jit}")


def tiny_problem_large(rng, n, K):
    # radix 1..2 per node (at most 2^32 plans), SLO near the middle of a sample's CPs
    edges = np.array([(i, j) for i in range(n) for j in range(i + 1, n) if rng.random() < 0.2],
                     np.int32).reshape(-1, 2)
    radix = rng.integers(1, 3, size=n).astype(np.int32)
    prob = wl.Problem(n_nodes=n, edges=edges, radix=radix, p=rng.uniform(0.4, 1.0, (n, 2)).astype(np.float32),
                      tau=rng.lognormal(0, 0.6, (n, 2)).astype(np.float32),
                      size=rng.choice([0.5, 1, 2.5, 6], (n, 2)).astype(np.float32),
                      backend=np.zeros((n, 2), np.int32), w=rng.uniform(0, 1, n).astype(np.float32),
                      rho=np.repeat(np.sort(rng.uniform(0, 0.9, K))[:, None], 1, axis=1).astype(np.float32),
                      slo=0.0)
    cps = orc.cp0_values(prob, 0, min(prob.n_plans(), 1 << 16))
    prob.slo = f32(np.median(cps) * 1.4)
    return prob


def test_generated_sweep_random_problems():
    # DY_OPT_JIT 2: every RANGE source runs the sweep generated for its DAG
    # (default: sources of 2^24 plans and more); ragged ranges, the SLO at
    # a CP quantile, one or two sinks besides y, an edge x -> y or not
    rng = np.random.default_rng(6060)
    for trial in range(7):
        n = int(rng.integers(3, 12))
        rmax = min(int(rng.choice([3, 6, 12])), int(3e6 ** (1.0 / n)))  # at most ~3e6 plans
        prob = tiny_problem(rng, n, rmax, int(rng.integers(1, 9)), 2, True, edge_p=float(rng.choice([0.2, 0.5])))
        total = prob.n_plans()
        begin = int(rng.integers(0, max(1, total // 5)))
        count = int(total - begin - rng.integers(0, max(1, total // 5)))
        want = orc.select_range(prob, begin, count)
        with D.Plan(prob) as plan:
            plan.set_option(D.DY_OPT_JIT, 2)
            for call in range(2):  # the second call replays the captured graph
                got = plan.select([D.range_source(0, begin, count)], stream=stream())[0]
                assert_choices(got, want, f"trial {trial} ({n} nodes, radix <= {rmax}), call {call}")


@pytest.mark.parametrize("begin,count", [(0, 1 << 20), (123457, 1000003), (429981696 - 777777, 777777)])
def test_forkjoin8_generated_sweep(begin, count):
    prob = wl.forkjoin8()
    with D.Plan(prob) as plan:
        plan.set_option(D.DY_OPT_JIT, 2)
        got = plan.select([D.range_source(0, begin, count)], stream=stream())[0]
    assert_choices(got, orc.select_range(prob, begin, count), f"forkjoin8 [{begin}+{count}] generated sweep")


@pytest.mark.parametrize("jit,stride", [(1, 24), (1, 27), (0, 24), (0, 27)])
def test_score_rows_and_bad_ids(jit, stride):
    # rows through the kernel generated for the DAG (jit 1) or the generic
    # kernel; stride 27 takes the byte-load path, its padding bytes are noise
    prob = wl.stream24()
    rows = wl.make_rows(50001, 24, 36)
    rows[77, 5] = 36  # an id out of range: NaN scores for that row only
    rows[901, 23] = 255
    buf = np.random.default_rng(stride).integers(0, 256, (50001, stride)).astype(np.uint8)
    buf[:, :24] = rows
    d = torch.from_numpy(buf).cuda()
    with D.Plan(prob) as plan:
        plan.set_option(D.DY_OPT_JIT, jit)
        got = run_score(plan, D.rows_source(0, d, 50001, stride), 50001, prob.n_levels)
        ok = np.ones(50001, bool)
        ok[[77, 901]] = False
        want = orc.score_rows(prob, np.where(ok[:, None], rows, 0))
        assert_scores(tuple(a[ok] for a in got), tuple(a[ok] for a in want), f"stream24 score, jit {jit}")
        for r in (77, 901):
            assert math.isnan(got[0][r]) and math.isnan(got[2][r]) and np.isnan(got[1][r]).all() and got[3][r] == 0
        with pytest.raises(D.DyplanError) as e:
            plan.select([D.rows_source(0, d, 50001, stride)], stream=stream())
        assert e.value.status == D.DY_EINVAL


def test_score_forkjoin8_full_size_sampled():
    prob = wl.forkjoin8()
    n = 12 ** 8
    with D.Plan(prob) as plan:
        corr = torch.empty(n, dtype=torch.float32, device="cuda")
        cp = torch.empty(n, prob.n_levels, dtype=torch.float32, device="cuda")
        feas = torch.empty(n, dtype=torch.int32, device="cuda")
        plan.score(D.range_source(0, 0, n), corr, cp, None, feas, stream=stream())
        torch.cuda.synchronize()
        idx = np.unique(np.concatenate([np.random.default_rng(5).integers(0, n, 20000), [0, n - 1]]))
        oc, ocp, od, of = orc.score_indices(prob, idx)
        ti = torch.from_numpy(idx.astype(np.int64)).cuda()
        np.testing.assert_allclose(corr[ti].cpu().numpy(), oc, rtol=RTOL, atol=0)
        np.testing.assert_allclose(cp[ti].cpu().numpy(), ocp, rtol=RTOL, atol=0)
        assert (feas[ti].cpu().numpy().view(np.uint32) == of).all()
        # feasibility bits are nested in the level for uniform pressure
        f = feas.cpu().numpy().view(np.uint32)
        assert ((f & (f >> 1)) == (f >> 1)).all()


# ---------------------------------------------------------------------------
# edge cases and small random problems
# ---------------------------------------------------------------------------

def tiny_problem(rng, n, rmax, K, B, uniform, edge_p=0.4, integer_tau=False):
    edges = np.array([(i, j) for i in range(n) for j in range(i + 1, n) if rng.random() < edge_p],
                     np.int32).reshape(-1, 2)
    radix = rng.integers(1, rmax + 1, size=n).astype(np.int32)
    R = int(radix.max())
    tau = (rng.integers(0, 6, size=(n, R)) if integer_tau else rng.lognormal(0, 0.6, size=(n, R))).astype(np.float32)
    p = rng.uniform(0.4, 1.0, size=(n, R)).astype(np.float32)
    size = rng.choice([0.5, 1, 2.5, 6], size=(n, R)).astype(np.float32)
    backend = rng.integers(0, B, size=(n, R)).astype(np.int32)
    w = rng.uniform(0, 1, size=n).astype(np.float32)
    if uniform:
        rho = np.repeat(np.sort(rng.uniform(0, 0.9, size=K))[:, None], B, axis=1).astype(np.float32)
    else:
        rho = rng.uniform(0, 0.9, size=(K, B)).astype(np.float32)
    prob = wl.Problem(n_nodes=n, edges=edges, radix=radix, p=p, tau=tau, size=size, backend=backend, w=w,
                      rho=rho, slo=0.0)
    cps = orc.cp0_values(prob, 0, prob.n_plans())
    prob.slo = f32(np.quantile(cps, rng.choice([0.05, 0.5, 0.9])) * 1.3)
    return prob


@pytest.mark.parametrize("uniform", [True, False])
def test_random_small_problems(uniform):
    rng = np.random.default_rng(101 if uniform else 202)
    for trial in range(40):
        n = int(rng.integers(1, 7))
        prob = tiny_problem(rng, n, 5, int(rng.integers(1, 6)), int(rng.integers(1, 4)), uniform,
                            integer_tau=bool(trial % 3 == 0))
        total = prob.n_plans()
        begin = int(rng.integers(0, total))
        count = int(rng.integers(1, total - begin + 1))
        got = select(prob, [D.range_source(0, 0, total), D.range_source(0, begin, count)])
        assert_choices(got[0], orc.select_range(prob, 0, total), f"trial {trial} full")
        assert_choices(got[1], orc.select_range(prob, begin, count), f"trial {trial} [{begin}+{count}]")
        with D.Plan(prob) as plan:
            sc = run_score(plan, D.range_source(0, 0, total), total, prob.n_levels)
        assert_scores(sc, orc.score_range(prob, 0, total), f"trial {trial} score")


def test_general_pressure_larger():
    rng = np.random.default_rng(7)
    prob = wl.forkjoin8()
    prob.rho = np.stack([prob.rho[:, 0], prob.rho[:, 0] * 0.5], axis=1).astype(np.float32)  # backend 1 lighter
    got = select(prob, [D.range_source(0, 1234567, 400000)])[0]
    assert_choices(got, orc.select_range(prob, 1234567, 400000), "general forkjoin8")


def test_slo_extremes_and_boundary():
    prob = wl.forkjoin8()
    begin, count = 5000000, 200000
    for slo in (0.0, 1e-3, float("inf"), f32(prob.slo * 0.35)):
        p = prob.copy()
        p.slo = slo
        assert_choices(select(p, [D.range_source(0, begin, count)])[0], orc.select_range(p, begin, count, slo=slo),
                       f"slo {slo}")
    # integer durations: some plan sits exactly on the SLO (inclusive)
    p = prob.copy()
    p.tau = np.round(p.tau * 2).astype(np.float32)
    cps = orc.cp0_values(p, begin, count)
    p.slo = float(np.median(cps))
    assert (cps == p.slo).any()
    p.rho[:] = 0.0
    assert_choices(select(p, [D.range_source(0, begin, count)])[0], orc.select_range(p, begin, count), "boundary")


def test_ties_go_to_lowest_index():
    prob = wl.chain4()
    p = prob.copy()
    # make implementations 0 and 1 (backends 0 and 1 of model 0, unverified) exact twins on every node
    p.p[:, 1] = p.p[:, 0]
    p.p[:, 3] = p.p[:, 2]
    p.tau[:, 1] = p.tau[:, 0]
    assert_choices(select(p, [D.range_source(0, 0, p.n_plans())])[0], orc.select_range(p, 0, p.n_plans()), "ties")
    # all plans identical: every feasible level picks index `begin`
    q = prob.copy()
    q.p[:] = 0.8
    q.tau[:] = 1.0
    q.slo = 10.0
    got = select(q, [D.range_source(0, 333, 5000)])[0]
    assert_choices(got, orc.select_range(q, 333, 5000), "all equal")
    assert all(c[0] == 333 for c in got if c[1])


def test_candidate_overflow_falls_back_exactly():
    q = wl.chain4()
    q.p[:] = 0.8  # every plan ties on corr: the candidate list overflows
    with D.Plan(q) as plan:
        plan.set_option(D.DY_OPT_CAND_CAPACITY, 16)
        got = plan.select([D.range_source(0, 100, 20000)], stream=stream())[0]
        assert plan.stats().fallbacks > 0
    assert_choices(got, orc.select_range(q, 100, 20000), "overflow")


def test_force_fp64_path_matches():
    prob = wl.forkjoin8()
    with D.Plan(prob) as plan:
        plan.set_option(D.DY_OPT_FORCE_FP64, 1)
        got = plan.select([D.range_source(0, 7777777, 300001)], stream=stream())[0]
    assert_choices(got, orc.select_range(prob, 7777777, 300001), "fp64 path")


def test_sample_stride_and_repeat_determinism():
    prob = wl.layered10()
    want = orc.select_range(prob, 10 ** 9, 1 << 20)
    with D.Plan(prob) as plan:
        for s in (1, 7, 32, 1000):
            plan.set_option(D.DY_OPT_SAMPLE_STRIDE, s)
            for _ in range(2):
                assert_choices(plan.select([D.range_source(0, 10 ** 9, 1 << 20)], stream=stream())[0], want,
                               f"stride {s}")


def test_multiple_sources_and_problems_in_one_call():
    probs = [wl.chain4(), wl.forkjoin8(), wl.layered10()]
    srcs = [D.range_source(0, 0, 20736), D.range_source(1, 1 << 20, 1 << 19), D.range_source(2, 5, 1 << 19),
            D.range_source(1, 0, 1000), D.range_source(0, 17, 3)]
    with D.Plan(probs) as plan:
        got = plan.select(srcs, stream=stream())
    for s, g in zip(srcs, got):
        assert_choices(g, orc.select_range(probs[s.problem], s.begin, s.count), f"source {s.problem}")


def test_select_argument_errors():
    with D.Plan(wl.chain4()) as plan:
        for src in (D.range_source(0, 0, 0), D.range_source(0, 20000, 737), D.range_source(1, 0, 1),
                    D.DySource(7, 0, 0, 1, None, 0, 0), D.rows_source(0, 0, 10, 4)):
            with pytest.raises(D.DyplanError):
                plan.select([src], stream=stream())


def test_overflow_recovered_by_reseeding():
    prob = wl.forkjoin8()
    begin, count = 3000000, 2000000
    with D.Plan(prob) as plan:
        plan.set_option(D.DY_OPT_SAMPLE_STRIDE, 1 << 30)  # one seed sample: weak thresholds
        plan.set_option(D.DY_OPT_CAND_CAPACITY, 1024)
        got = plan.select([D.range_source(0, begin, count)], stream=stream())[0]
        st = plan.stats()
    assert_choices(got, orc.select_range(prob, begin, count), "reseeded")
    assert st.fallbacks == 0


@pytest.mark.parametrize("jit", [1, 0])
def test_rows_generated_and_generic_kernels(jit):
    rng = np.random.default_rng(404)
    probs, rows_list = [], []
    for trial in range(6):
        n = int(rng.integers(1, 12))
        prob = tiny_problem(rng, n, 6, int(rng.integers(1, 5)), 2, True)
        cnt = int(rng.integers(1, 70000))
        rows = np.stack([rng.integers(0, r, size=cnt) for r in prob.radix], axis=1).astype(np.uint8)
        probs.append(prob)
        rows_list.append(rows)
    with D.Plan(probs) as plan:
        plan.set_option(D.DY_OPT_JIT, jit)
        for t, (prob, rows) in enumerate(zip(probs, rows_list)):
            d = torch.from_numpy(np.ascontiguousarray(rows)).cuda()
            got = plan.select([D.rows_source(t, d, rows.shape[0], rows.shape[1], 77)], stream=stream())[0]
            assert_choices(got, orc.select_rows(prob, rows, 77), f"rows trial {t} jit={jit}")


def test_rows_bad_ids_rejected_by_generated_kernel():
    prob = wl.stream24()
    rows = wl.make_rows(20000, 24, 36)
    with D.Plan(prob) as plan:
        for bad in (36, 63, 64, 200):
            r = rows.copy()
            r[12345, 7] = bad
            dr = torch.from_numpy(r).cuda()
            with pytest.raises(D.DyplanError) as e:
                plan.select([D.rows_source(0, dr, 20000, 24)], stream=stream())
            assert e.value.status == D.DY_EINVAL
        d = torch.from_numpy(rows).cuda()
        got = plan.select([D.rows_source(0, d, 20000, 24)], stream=stream())[0]
        assert_choices(got, orc.select_rows(prob, rows), "after bad rows")


def test_rows_radix_above_64_uses_generic_path():
    rng = np.random.default_rng(505)
    prob = tiny_problem(rng, 3, 2, 2, 2, True)
    R = 100
    prob.radix = np.array([R, 3, R], np.int32)
    for name in ("p", "tau", "size", "backend"):
        a = getattr(prob, name)
        b = np.zeros((3, R), a.dtype)
        b[:, :a.shape[1]] = a
        for c in range(a.shape[1], R):
            b[:, c] = a[:, c % a.shape[1]] * (1 if name in ("backend", "size") else 0.999)
        setattr(prob, name, b)
    prob.slo = 1e9
    rows = np.stack([rng.integers(0, r, size=30000) for r in prob.radix], axis=1).astype(np.uint8)
    with D.Plan(prob) as plan:
        d = torch.from_numpy(rows).cuda()
        got = plan.select([D.rows_source(0, d, 30000, 3)], stream=stream())[0]
    assert_choices(got, orc.select_rows(prob, rows), "radix 100 rows")


def row_problem(rng, n, rmax, K, edge_p):
    edges = np.array([(i, j) for i in range(n) for j in range(i + 1, n) if rng.random() < edge_p],
                     np.int32).reshape(-1, 2)
    radix = rng.integers(2, rmax + 1, size=n).astype(np.int32)
    R = int(radix.max())
    prob = wl.Problem(n_nodes=n, edges=edges, radix=radix,
                      p=rng.uniform(0.5, 1.0, size=(n, R)).astype(np.float32),
                      tau=rng.lognormal(0, 0.7, size=(n, R)).astype(np.float32),
                      size=rng.choice([0.5, 1, 2.5, 6], size=(n, R)).astype(np.float32),
                      backend=rng.integers(0, 2, size=(n, R)).astype(np.int32),
                      w=rng.uniform(0, 1, size=n).astype(np.float32),
                      rho=np.repeat(np.sort(rng.uniform(0, 0.9, size=K))[:, None], 2, axis=1).astype(np.float32),
                      slo=0.0)
    return prob


def skewed_rows(rng, prob, count, p_top=0.75):
    """Rows concentrated on each node's three highest-factor implementations, so
    that many rows sit near the per-level thresholds and the generated kernel
    abandons rows right at the edge of its bounds."""
    a = 1.0 - prob.w[:, None].astype(np.float64) * (1.0 - prob.p.astype(np.float64))
    cols = []
    for n in range(prob.n_nodes):
        R = int(prob.radix[n])
        top = np.argsort(-a[n, :R], kind="stable")[:min(3, R)]
        ids = np.where(rng.random(count) < p_top, rng.choice(top, size=count), rng.integers(0, R, size=count))
        cols.append(ids)
    return np.stack(cols, axis=1).astype(np.uint8)


@pytest.mark.parametrize("n_nodes", [8, 13, 21, 32])
def test_rows_early_exit_near_threshold(n_nodes):
    # DAG-specialised rows kernel with mid-row abandonment (N >= 8) on rows
    # crowded near the thresholds; tight and loose SLOs
    rng = np.random.default_rng(600 + n_nodes)
    for trial in range(3):
        prob = row_problem(rng, n_nodes, int(rng.integers(4, 41)), int(rng.integers(2, 9)),
                           float(rng.uniform(0.15, 0.5)))
        rows = skewed_rows(rng, prob, 150000)
        cps = orc.cp0_values(prob, rows=rows)
        prob.slo = f32(np.quantile(cps, (0.02, 0.3, 0.8)[trial]) * 1.05)
        want = orc.select_rows(prob, rows, index_base=5)
        with D.Plan(prob) as plan:
            d = torch.from_numpy(rows).cuda()
            got = plan.select([D.rows_source(0, d, rows.shape[0], n_nodes, 5)], stream=stream())[0]
        assert_choices(got, want, f"N={n_nodes} trial {trial}")


def test_graph_replay_matches_eager_calls():
    # repeated identical calls are replayed from a HIP graph; every replay, with
    # eager work and synchronisations in between and a different call in the
    # middle (which invalidates the graph), must give the oracle's answer
    prob = wl.forkjoin8()
    a, b = (D.range_source(0, 1000, 3000000),), (D.range_source(0, 5000000, 2000000),)
    want_a = orc.select_range(prob, 1000, 3000000)
    want_b = orc.select_range(prob, 5000000, 2000000)
    rows = wl.make_rows(200000, 24, 36, row_begin=777)
    want_r = orc.select_rows(wl.stream24(), rows, index_base=3)
    with D.Plan([prob, wl.stream24()]) as plan:
        d = torch.from_numpy(rows).cuda()
        r = (D.rows_source(1, d, 200000, 24, 3),)
        for i in range(6):
            assert_choices(plan.select(list(a), stream=stream())[0], want_a, f"replay {i}")
            x = torch.randn(4096, device="cuda")
            assert torch.isfinite((x * 2).sum()).item()
            torch.cuda.synchronize()
            if i == 3:
                assert_choices(plan.select(list(b), stream=stream())[0], want_b, "other range")
            if i % 2 == 1:
                assert_choices(plan.select(list(r), stream=stream())[0], want_r, f"rows replay {i}")
        plan.set_option(D.DY_OPT_TIMING, 1)  # timed calls launch directly
        for i in range(3):
            assert_choices(plan.select(list(a), stream=stream())[0], want_a, f"timed replay {i}")
            assert plan.stats().main_ms > 0
        plan.set_option(D.DY_OPT_GRAPH, 0)
        assert_choices(plan.select(list(a), stream=stream())[0], want_a, "eager")


@pytest.mark.parametrize("begin,count", [(0, 12 ** 8), (144 * 12, 144 * 1048584), (144 * 6, 144 * 1048580 + 77),
                                         (144 * 7 + 5, 144 * 1048576 + 1000)])
def test_library_sweep_block_runs(begin, count):
    # the library sweep (DY_OPT_JIT 0) gives each thread a run of up to 12
    # blocks that share the prefix but its last node, when the source's blocks
    # align (runs of 12, 6, ..., else single blocks; ragged ends): the choices
    # equal the generated sweep's, which the oracle pins on the same kind of
    # ranges, and on the whole space the stored oracle selection
    prob = wl.forkjoin8()
    src = [D.range_source(0, begin, count)]
    with D.Plan(prob) as plan:
        plan.set_option(D.DY_OPT_JIT, 0)
        lib = plan.select(src, stream=stream())[0]
        plan.set_option(D.DY_OPT_JIT, 2)
        gen = plan.select(src, stream=stream())[0]
    assert_choices(lib, [tuple(c) for c in gen], f"forkjoin8 [{begin}+{count}] library vs generated sweep")
    if (begin, count) == (0, 12 ** 8):
        assert_choices(lib, golden("forkjoin8")[1], "forkjoin8 whole space, library sweep")


@pytest.mark.parametrize("case", ["mixed", "tiny", "zero"])
def test_predivided_thresholds_small_and_zero_factors(case):
    # The sweeps compare x's product with bin thresholds divided ahead by each
    # implementation of y's factor a = 1 - w (1 - p).  Factors of 0 and below
    # 2^-20 take the threshold 0 (every plan of them passes the prefilter and
    # the exact test decides); factors near 1e-6 give thresholds near 1e-6.
    # Library sweep (jit 0) and generated sweep (jit 2), whole plan space of a
    # 6-node request with 12 implementations per node, against the oracle.
    import dataclasses
    base = wl.batch6_request(7)
    p = base.p.copy()
    w = base.w.copy()
    y = base.n_nodes - 1
    w[y] = 1.0  # a = p for node y
    if case == "mixed":
        p[y, :12] = np.array([0, 1e-7, 5e-7, 1e-6, 3e-6, 1e-3, 0.05, 0.2, 0.5, 0.7, 0.9, 1.0], np.float32)
    elif case == "tiny":
        p[y, :12] = np.linspace(2e-6, 9e-6, 12).astype(np.float32)
    else:
        p[y, :12] = 0.0
    prob = dataclasses.replace(base, p=p, w=w)
    n = prob.n_plans()
    want = orc.select_range(prob, 0, n)
    for jit in (0, 2):
        with D.Plan(prob) as plan:
            plan.set_option(D.DY_OPT_JIT, jit)
            got = plan.select([D.range_source(0, 0, n)], stream=stream())[0]
            assert plan.stats().ydiv_jobs in (0, 1)
        assert_choices(got, want, f"{case}, jit {jit}")
