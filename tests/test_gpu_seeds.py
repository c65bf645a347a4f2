"""GPU: seeds and the state a selection call leaves behind.

- Local-search seeds (DY_OPT_CLIMB 2: every eligible source) change only the work: on sources that
  cover a whole plan space the choices equal the oracle's with and without
  them, and the candidate lists never grow (a seed only raises thresholds).
- Consecutive calls on different streams, with rows rewritten in place at the
  same address (so the second call replays the first one's graph and skips the
  scratch initialisation), each equal the oracle on their own rows.
- Repeated calls on the same inputs (direct, graph-replayed, timed) choose the
  same plans and certify the same number of candidates.

Bar as in test_gpu_parity.py.
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import oracle as orc  # noqa: E402
from paper_2607_02942_amd import dyplan as D  # noqa: E402
from paper_2607_02942_amd import workload as wl  # noqa: E402

from test_gpu_parity import assert_choices, golden, stream, tiny_problem  # noqa: E402

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    D.lib()
    torch.cuda.set_device(0)
    yield


def select_with(plan, sources, climb):
    plan.set_option(D.DY_OPT_CLIMB, 2 if climb else 0)
    got = plan.select(sources, stream=stream())
    return got, plan.stats().candidates


@pytest.mark.parametrize("uniform", [True, False])
def test_climb_random_full_spaces(uniform):
    rng = np.random.default_rng(303 if uniform else 404)
    for trial in range(30):
        n = int(rng.integers(1, 8))
        prob = tiny_problem(rng, n, int(rng.choice([3, 5, 8])), int(rng.integers(1, 6)), int(rng.integers(1, 4)),
                            uniform, integer_tau=bool(trial % 4 == 0))
        total = prob.n_plans()
        want = orc.select_range(prob, 0, total)
        with D.Plan(prob) as plan:
            off, c_off = select_with(plan, [D.range_source(0, 0, total)], False)
            on, c_on = select_with(plan, [D.range_source(0, 0, total)], True)
            again, c_again = select_with(plan, [D.range_source(0, 0, total)], True)  # graph replay
        assert_choices(off[0], want, f"trial {trial} no climb")
        assert_choices(on[0], want, f"trial {trial} climb")
        assert_choices(again[0], want, f"trial {trial} climb, replay")
        assert c_on <= c_off and c_again == c_on, (trial, c_on, c_off, c_again)


def test_climb_batch6_requests_golden():
    _, want = golden("batch6")
    nreq = 256
    probs = wl.batch6(nreq)
    srcs = [D.range_source(r, 0, 12 ** 6) for r in range(nreq)]
    with D.Plan(probs) as plan:
        off, c_off = select_with(plan, srcs, False)
        on, c_on = select_with(plan, srcs, True)
    for r in range(nreq):
        assert_choices(off[r], want[r], f"batch6[{r}] no climb")
        assert_choices(on[r], want[r], f"batch6[{r}] climb")
    assert c_on < c_off, (c_on, c_off)


@pytest.mark.parametrize("factors", [(1.0, 0.5), (0.3, 1.0)])
def test_climb_per_class_full_spaces(factors):
    for prob in (wl.per_class(wl.chain4(), factors), wl.per_class(wl.batch6_request(5), factors)):
        total = prob.n_plans()
        want = orc.select_range(prob, 0, total)
        with D.Plan(prob) as plan:
            off, c_off = select_with(plan, [D.range_source(0, 0, total)], False)
            on, c_on = select_with(plan, [D.range_source(0, 0, total)], True)
        assert_choices(off[0], want, f"{prob.name} per class no climb")
        assert_choices(on[0], want, f"{prob.name} per class climb")
        assert c_on <= c_off


def test_forkjoin8_full_without_climb():
    g, want = golden("forkjoin8")
    prob = wl.forkjoin8()
    with D.Plan(prob) as plan:
        got, _ = select_with(plan, [D.range_source(0, 0, 12 ** 8)], False)
    assert_choices(got[0], want, "forkjoin8 full, sampled seeds only")


def test_partial_range_takes_no_climb():
    # a source that does not cover the whole plan space takes no local-search seed
    prob = wl.forkjoin8()
    src = [D.range_source(0, 1000, 12 ** 8 - 2000)]
    with D.Plan(prob) as plan:
        off, c_off = select_with(plan, src, False)
        on, c_on = select_with(plan, src, True)
    assert c_on == c_off
    assert_choices(on[0], [tuple(c) for c in off[0]], "forkjoin8 partial range")


def test_streams_alternate_with_rows_rewritten_in_place():
    prob = wl.stream24()
    n = 1 << 18
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    d = torch.empty((n, 24), dtype=torch.uint8, device="cuda")
    with D.Plan(prob) as plan:
        for call in range(6):
            rows = wl.make_rows(n, 24, 36, row_begin=call * 7919 * n)
            d.copy_(torch.from_numpy(rows))
            torch.cuda.synchronize()
            st = s1 if call % 2 == 0 else s2
            got = plan.select([D.rows_source(0, d, n, 24, 0)], stream=st)[0]
            assert_choices(got, orc.select_rows(prob, rows, 0), f"call {call} on stream {1 + call % 2}")


@pytest.mark.parametrize("per_class", [False, True])
def test_rows_calls_repeat_choices_and_candidates(per_class):
    prob = wl.stream24()
    if per_class:
        prob = wl.per_class(prob)
    n = 1 << 24
    d = torch.from_numpy(wl.make_rows(n, 24, 36)).cuda()
    src = [D.rows_source(0, d, n, 24, 0)]
    runs = []
    with D.Plan(prob) as plan:
        for call in range(3):  # direct, then graph replays
            runs.append((plan.select(src, stream=stream())[0], plan.stats().candidates))
        plan.set_option(D.DY_OPT_TIMING, 1)
        for call in range(2):  # timed calls launch directly
            runs.append((plan.select(src, stream=stream())[0], plan.stats().candidates))
    first, c0 = runs[0]
    for i, (got, c) in enumerate(runs[1:], 1):
        assert_choices(got, [tuple(x) for x in first], f"call {i}")
        assert c == c0, f"call {i}: {c} candidates, first call {c0}"


@pytest.mark.parametrize("per_class", [False, True])
@pytest.mark.parametrize("winners", ["first share", "second share"])
def test_rows_scored_in_two_shares(per_class, winners):
    # a rows source of 2^22 rows or more under per-backend pressure is scored
    # in two shares, the candidates of the first share (1/32 of the rows)
    # re-seeding the thresholds of the second (uniform pressure: one pass):
    # the choices equal the oracle's with every level's winner moved into the
    # first share, or into the second
    prob = wl.stream24()
    if per_class:
        prob = wl.per_class(prob)
    n = (1 << 22) + 777
    rows = wl.make_rows(n, 24, 36, row_begin=31 * n)
    win = sorted({int(c[0]) for c in orc.select_rows(prob, rows, 0) if int(c[0]) >= 0})
    for i, w in enumerate(win):
        to = 5 + 97 * i if winners == "first share" else n - 1 - 97 * i
        rows[[w, to]] = rows[[to, w]]
    want = orc.select_rows(prob, rows, 0)
    assert all(int(c[0]) < n // 32 for c in want if int(c[0]) >= 0) == (winners == "first share")
    d = torch.from_numpy(rows).cuda()
    with D.Plan(prob) as plan:
        for call in range(2):  # the second call replays the captured graph
            got = plan.select([D.rows_source(0, d, n, 24, 0)], stream=stream())[0]
            assert_choices(got, want, f"{prob.name}, winners in the {winners}, call {call}")


def test_repeated_calls_reuse_and_rebuild_the_call_plan():
    # a call whose sources, options and state repeat the previous call's reuses
    # the plan derived for it (groups, order, jobs); any change derives it
    # again: two source sets alternating, options changed between calls with
    # the same sources, a score call in between
    prob = wl.forkjoin8()
    a = [D.range_source(0, 0, 1 << 22)]
    b = [D.range_source(0, 5000, 1 << 21), D.range_source(0, 777777, 123457)]
    want = {"a": [orc.select_range(prob, 0, 1 << 22)],
            "b": [orc.select_range(prob, 5000, 1 << 21), orc.select_range(prob, 777777, 123457)]}
    srcs = {"a": a, "b": b}

    def check(plan, key, ctx):
        got = plan.select(srcs[key], stream=stream())
        for s, (g, w) in enumerate(zip(got, want[key])):
            assert_choices(g, w, f"{ctx}, source {s}")

    with D.Plan(prob) as plan:
        for i, key in enumerate("aabba"):
            check(plan, key, f"call {i} ({key})")
        plan.set_option(D.DY_OPT_SAMPLE_STRIDE, 7)
        check(plan, "a", "stride 7")
        check(plan, "a", "stride 7, again")
        plan.set_option(D.DY_OPT_CAND_CAPACITY, 1024)
        check(plan, "b", "1024 candidate slots")
        check(plan, "b", "1024 candidate slots, again")
        corr = torch.empty(1000, dtype=torch.float32, device="cuda")
        plan.score(D.range_source(0, 0, 1000), corr, None, None, None, stream=stream())
        check(plan, "b", "after a score call")
