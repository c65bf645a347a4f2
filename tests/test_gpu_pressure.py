"""GPU parity under per-backend pressure (rho_{k,b} differs between the
backends a level presses): the sweep, the generic rows path, the seeding
passes and the score API against the fp64 oracle, through the C-ABI.

Bar as in test_gpu_parity.py: indices and feasibility bit-exact, a winner's
values its fp64 values rounded to fp32, per-plan scores within 1e-5 relative.
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import oracle as orc  # noqa: E402
from paper_2607_02942_amd import dyplan as D  # noqa: E402
from paper_2607_02942_amd import workload as wl  # noqa: E402

from test_gpu_parity import assert_choices, assert_scores, run_score, select, stream, tiny_problem  # noqa: E402

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    D.lib()
    torch.cuda.set_device(0)
    yield


@pytest.mark.parametrize("factors", [(1.0, 0.5), (1.0, 0.0), (0.3, 1.0)])
@pytest.mark.parametrize("begin,count", [(0, 1 << 20), (123457, 1000003), (429981696 - 777777, 777777), (77, 1)])
def test_forkjoin8_per_class(factors, begin, count):
    prob = wl.per_class(wl.forkjoin8(), factors)
    got = select(prob, [D.range_source(0, begin, count)])[0]
    assert_choices(got, orc.select_range(prob, begin, count), f"forkjoin8 {factors} [{begin}+{count}]")


def test_random_pressure_per_level_and_backend():
    # every (level, backend) its own rho, levels not ordered
    rng = np.random.default_rng(77)
    prob = wl.forkjoin8()
    prob.rho = rng.uniform(0.0, 0.9, size=(8, 2)).astype(np.float32)
    for begin, count in ((0, 1 << 20), (5 * 12 ** 7 + 3, 999999)):
        got = select(prob, [D.range_source(0, begin, count)])[0]
        assert_choices(got, orc.select_range(prob, begin, count), f"random rho [{begin}+{count}]")


def test_layered10_per_class():
    prob = wl.per_class(wl.layered10(), (1.0, 0.6))
    for begin, count in ((0, 1 << 21), ((1 << 32) - 999999, 999999)):
        got = select(prob, [D.range_source(0, begin, count)])[0]
        assert_choices(got, orc.select_range(prob, begin, count), f"layered10 per class [{begin}+{count}]")


def test_wide_last_node_appends_per_level():
    # R_y > 64: the rare path may list a plan once per level; selection is unchanged
    rng = np.random.default_rng(5)
    n, R = 4, 100
    prob = wl.Problem(n_nodes=n, edges=np.array([[0, 1], [0, 2], [1, 3], [2, 3]], np.int32),
                      radix=np.array([3, 4, 5, R], np.int32),
                      p=rng.uniform(0.5, 1.0, (n, R)).astype(np.float32),
                      tau=rng.lognormal(0, 0.5, (n, R)).astype(np.float32),
                      size=np.ones((n, R), np.float32), backend=rng.integers(0, 3, (n, R)).astype(np.int32),
                      w=rng.uniform(0, 1, n).astype(np.float32),
                      rho=rng.uniform(0, 0.9, (6, 3)).astype(np.float32), slo=0.0)
    cps = orc.cp0_values(prob, 0, prob.n_plans())
    prob.slo = float(np.float32(np.median(cps) * 1.4))
    total = prob.n_plans()
    got = select(prob, [D.range_source(0, 0, total)])[0]
    assert_choices(got, orc.select_range(prob, 0, total), "wide y")


def test_batch_mixes_uniform_and_per_class():
    probs = [wl.batch6_request(r) for r in range(6)]
    probs = [wl.per_class(p, (1.0, 0.4)) if r % 2 else p for r, p in enumerate(probs)]
    with D.Plan(probs) as plan:
        got = plan.select([D.range_source(r, 0, 12 ** 6) for r in range(6)], stream=stream())
    for r in range(6):
        assert_choices(got[r], orc.select_range(probs[r], 0, 12 ** 6), f"batch[{r}]")


@pytest.mark.parametrize("jit", [1, 0])
@pytest.mark.parametrize("factors", [(1.0, 0.5), (0.3, 1.0)])
def test_rows_per_class(jit, factors):
    # the kernel generated for the DAG (jit 1: bands of the unpressured CP,
    # then each level's exact CP_k) or the generic kernel
    prob = wl.per_class(wl.stream24(), factors)
    n = 300007
    rows = wl.make_rows(n, 24, 36, row_begin=999)
    want = orc.select_rows(prob, rows, index_base=999)
    with D.Plan(prob) as plan:
        plan.set_option(D.DY_OPT_JIT, jit)
        d = torch.from_numpy(rows).cuda()
        got = plan.select([D.rows_source(0, d, n, 24, 999)], stream=stream())[0]
    assert_choices(got, want, f"stream24 per class {factors} rows, jit {jit}")


@pytest.mark.parametrize("jit", [1, 0])
def test_rows_random_pressure(jit):
    # random DAGs, every (level, backend) its own rho, SLO at a CP quantile;
    # rows drawn from the whole plan space, so boundary plans are present
    rng = np.random.default_rng(4242)
    for trial in range(8):
        n = int(rng.integers(3, 10))
        R = 6
        edges = np.array([(i, j) for i in range(n) for j in range(i + 1, n) if rng.random() < 0.4],
                         np.int32).reshape(-1, 2)
        K, B = int(rng.integers(1, 9)), 3
        prob = wl.Problem(n_nodes=n, edges=edges, radix=rng.integers(1, R + 1, n).astype(np.int32),
                          p=rng.uniform(0.4, 1.0, (n, R)).astype(np.float32),
                          tau=rng.integers(1, 6, (n, R)).astype(np.float32),
                          size=rng.choice([0.5, 1, 2.5], (n, R)).astype(np.float32),
                          backend=rng.integers(0, B, (n, R)).astype(np.int32),
                          w=rng.uniform(0, 1, n).astype(np.float32),
                          rho=rng.uniform(0, 0.9, (K, B)).astype(np.float32), slo=0.0)
        total = prob.n_plans()
        m = 40000
        idx = rng.integers(0, total, m)
        rows = np.stack([orc.decode(prob, int(i)) for i in idx]).astype(np.uint8)
        cps = orc.cp0_values(prob, rows=rows)
        prob.slo = float(np.float32(np.quantile(cps, rng.choice([0.1, 0.5])) * 1.5))
        want = orc.select_rows(prob, rows)
        with D.Plan(prob) as plan:
            plan.set_option(D.DY_OPT_JIT, jit)
            got = plan.select([D.rows_source(0, torch.from_numpy(rows).cuda(), m, n)], stream=stream())[0]
        assert_choices(got, want, f"trial {trial}, jit {jit}")


@pytest.mark.parametrize("factors", [(1.0, 0.5), (0.3, 1.0)])
@pytest.mark.parametrize("begin,count", [(0, 1 << 20), (123457, 1000003), (429981696 - 777777, 777777)])
def test_forkjoin8_per_class_generated_sweep(factors, begin, count):
    # DY_OPT_JIT 2: the sweep generated for the DAG, its rare path each
    # admitted level's exact CP_k; the library sweep (DY_OPT_JIT 0) beside it
    prob = wl.per_class(wl.forkjoin8(), factors)
    want = orc.select_range(prob, begin, count)
    for jit in (2, 0):
        with D.Plan(prob) as plan:
            plan.set_option(D.DY_OPT_JIT, jit)
            got = plan.select([D.range_source(0, begin, count)], stream=stream())[0]
            assert plan.stats().generated_jobs == (1 if jit else 0)
        assert_choices(got, want, f"forkjoin8 {factors} [{begin}+{count}], jit {jit}")


def test_generated_sweep_random_pressure():
    # random DAGs, every (level, backend) its own rho, ragged ranges, the SLO
    # at a CP quantile; every source through the generated sweep
    rng = np.random.default_rng(9191)
    for trial in range(8):
        n = int(rng.integers(3, 12))
        rmax = min(int(rng.choice([3, 6, 12])), int(3e6 ** (1.0 / n)))  # at most ~3e6 plans
        prob = tiny_problem(rng, n, rmax, int(rng.integers(1, 9)), 3, False, edge_p=float(rng.choice([0.2, 0.5])))
        total = prob.n_plans()
        begin = int(rng.integers(0, max(1, total // 5)))
        count = int(total - begin - rng.integers(0, max(1, total // 5)))
        want = orc.select_range(prob, begin, count)
        with D.Plan(prob) as plan:
            plan.set_option(D.DY_OPT_JIT, 2)
            for call in range(2):  # the second call replays the captured graph
                got = plan.select([D.range_source(0, begin, count)], stream=stream())[0]
                assert_choices(got, want, f"trial {trial} ({n} nodes, radix <= {rmax}), call {call}")


def test_small_capacity_reseeds_per_class():
    prob = wl.per_class(wl.forkjoin8(), (1.0, 0.0))
    begin, count = 4321, 1 << 20
    want = orc.select_range(prob, begin, count)
    with D.Plan(prob) as plan:
        plan.set_option(D.DY_OPT_CAND_CAPACITY, 16)
        plan.set_option(D.DY_OPT_SAMPLE_STRIDE, 1 << 20)
        got = plan.select([D.range_source(0, begin, count)], stream=stream())[0]
    assert_choices(got, want, "per class reseed")


def test_score_per_class():
    prob = wl.per_class(wl.forkjoin8(), (1.0, 0.5))
    begin, count = 98765, 200003
    with D.Plan(prob) as plan:
        got = run_score(plan, D.range_source(0, begin, count), count, prob.n_levels)
    assert_scores(got, orc.score_range(prob, begin, count), "per class scores")


def test_graph_replay_per_class():
    prob = wl.per_class(wl.forkjoin8(), (1.0, 0.5))
    src = [D.range_source(0, 31, 1 << 20)]
    want = orc.select_range(prob, 31, 1 << 20)
    with D.Plan(prob) as plan:
        for rep in range(3):
            assert_choices(plan.select(src, stream=stream())[0], want, f"replay {rep}")


@pytest.mark.parametrize("per_class", [False, True])
def test_score_feasibility_on_the_slo_boundary(per_class):
    # integer durations and the SLO on the median CP: many plans sit exactly on
    # the SLO at some level, inside the fp32 band, so the exact fp64 check decides
    prob = wl.forkjoin8()
    prob.tau = np.round(prob.tau * 2).astype(np.float32)
    if per_class:
        prob = wl.per_class(prob, (1.0, 0.5))
    begin, count = 777, 300007
    cps = orc.cp0_values(prob, begin, count)
    prob.slo = float(np.median(cps))
    assert (cps == prob.slo).sum() > 1000
    with D.Plan(prob) as plan:
        got = run_score(plan, D.range_source(0, begin, count), count, prob.n_levels)
    assert_scores(got, orc.score_range(prob, begin, count), f"boundary scores per_class={per_class}")
