"""Plan-bundle annotations and load-driven switching.

The oracle (oracle/bundle.py, plain Python written from Sec. 4.4 and Sec. 5.2)
is pinned to the paper's walkthrough (the dominant models of pi(0) and pi(1),
the switch to pi(1) under a 27B burst) and to each switching rule the paper
states; the library's host implementation (dy_bundle_annotate,
dy_switch_simulate) must agree with it exactly on random plans and load
traces; on the GPU, the bundle of a selected J_L problem is annotated and
replayed against the oracle's.
"""
import numpy as np
import pytest

from oracle import bundle as ob
from oracle import oracle as orc
from paper_2607_02942_amd import dyplan as D
from paper_2607_02942_amd import workload as wl

M9B, M27B = 0, 1


def walkthrough():
    """P -> {C, D} -> R -> A (Sec. 3.2 walkthrough): P, R, A take no time; C
    runs 27B (10), 27B + verification (14) or 9B (6); D runs 9B (4) or 9B +
    verification (7).  Illustrative accuracies as success probabilities."""
    edges = np.array([[0, 1], [0, 2], [1, 3], [2, 3], [3, 4]], np.int32)
    R = 3
    tau = np.zeros((5, R), np.float32)
    tau[1] = [10.0, 14.0, 6.0]
    tau[2, :2] = [4.0, 7.0]
    p = np.ones((5, R), np.float32)
    p[1] = [0.95, 0.97, 0.85]
    p[2, :2] = [0.9, 0.95]
    model = np.zeros((5, R), np.int32)
    model[1] = [M27B, M27B, M9B]
    prob = wl.Problem(n_nodes=5, edges=edges, radix=np.array([1, 3, 2, 1, 1], np.int32), p=p, tau=tau,
                      size=np.ones((5, R), np.float32), backend=np.zeros((5, R), np.int32),
                      w=np.array([0.0, 1.0, 1.0, 0.0, 0.0], np.float32), rho=np.zeros((1, 1), np.float32),
                      slo=np.float32(np.inf))
    return prob, model


PI0 = [0, 0, 1, 0, 0]  # C 27B, D 9B + verification: fork 10, duration sum 17
PI1 = [0, 2, 0, 0, 0]  # C 9B, D 9B: fork 6, duration sum 10


# ---------------------------------------------------------------------------
# oracle pins
# ---------------------------------------------------------------------------

def test_walkthrough_dominant_models():
    prob, model = walkthrough()
    d0, dom0, q0 = ob.annotate(prob, PI0, model, 2)
    d1, dom1, q1 = ob.annotate(prob, PI1, model, 2)
    assert d0 == [7.0, 10.0] and dom0 == M27B  # the paper: 27B dominates pi(0)
    assert d1 == [10.0, 0.0] and dom1 == M9B   # and 9B dominates pi(1)
    assert sum(d0) == 17.0 and sum(d1) == 10.0  # the walkthrough's duration sums
    assert q0 == pytest.approx(0.95 * 0.95) and q1 == pytest.approx(0.85 * 0.9)


def test_annotation_closed_forms():
    prob, model = walkthrough()
    p = prob.copy()
    p.w[:] = 0.0
    assert ob.annotate(p, PI0, model, 2)[2] == 1.0                  # no vulnerability: quality 1
    _, dom, _ = ob.annotate(prob, [0, 2, 1, 0, 0], np.zeros_like(model), 2)
    assert dom == 0
    tie = model.copy()
    tie[2, :] = M27B
    p = prob.copy()
    p.tau[2, 0] = 6.0
    d, dom, _ = ob.annotate(p, [0, 2, 0, 0, 0], tie, 2)             # 6 on each model: lowest id
    assert d == [6.0, 6.0] and dom == 0
    d, dom, q = ob.annotate(prob, PI0, model, 2, is_tool=np.ones(5, np.int32))
    assert dom == -1 and q == 1.0 and d == [0.0, 0.0]


RULES = dict(high=0.8, low=0.3, tolerance=0.15, margin=0.0, dwell=10.0)


def test_walkthrough_burst_switches_to_pi1_and_back():
    prob, model = walkthrough()
    dom = [ob.annotate(prob, pi, model, 2)[1] for pi in (PI0, PI1)]
    q = [ob.annotate(prob, pi, model, 2)[2] for pi in (PI0, PI1)]
    # loads (9B, 27B): calm, a 27B burst, calm again
    times = [0, 5, 20, 25, 40, 45, 60]
    loads = [(0.2, 0.2), (0.3, 0.95), (0.3, 0.95), (0.3, 0.5), (0.2, 0.2), (0.2, 0.2), (0.2, 0.2)]
    act, n = ob.simulate(dom, q, times, loads, **RULES)
    assert act == [0, 1, 1, 1, 0, 0, 0] and n == 2


def test_rule_dwell_blocks_switches_in_either_direction():
    dom, q = [1, 0], [0.9, 0.85]
    times = [0, 1, 2, 3, 12]
    loads = [(0.1, 0.9), (0.1, 0.1), (0.1, 0.1), (0.1, 0.1), (0.1, 0.1)]
    act, n = ob.simulate(dom, q, times, loads, **RULES)
    assert act == [1, 1, 1, 1, 0] and n == 2  # the return waits for the dwell time


def test_rule_same_dominant_model_is_skipped():
    # variant 1 only drops verification and keeps the congested 27B: insufficient
    dom, q = [1, 1, 0], [0.9, 0.88, 0.8]
    act, _ = ob.simulate(dom, q, [0], [(0.1, 0.9)], **RULES)
    assert act == [2]


def test_rule_overloaded_or_not_calmer_candidate_is_skipped():
    dom, q = [1, 0, 2], [0.9, 0.85, 0.85]
    act, _ = ob.simulate(dom, q, [0], [(0.85, 0.9, 0.1)], **RULES)      # 9B overloaded too
    assert act == [2]
    act, _ = ob.simulate(dom, q, [0], [(0.5, 0.9, 0.1)], **dict(RULES, margin=0.5))  # 9B not calm enough
    assert act == [2]


def test_rule_quality_tolerance_rejects_even_an_idle_backend():
    dom, q = [1, 0], [0.9, 0.7]
    act, n = ob.simulate(dom, q, [0], [(0.0, 0.95)], **RULES)
    assert act == [0] and n == 0


def test_rule_first_passing_later_variant_and_lowest_calm_return():
    dom, q = [1, 0, 2, 0], [0.9, 0.86, 0.89, 0.8]
    act, _ = ob.simulate(dom, q, [0], [(0.2, 0.9, 0.1)], **RULES)
    assert act == [1]  # the first that passes, not the best quality
    act, _ = ob.simulate(dom, q, [0, 20, 40], [(0.2, 0.9, 0.9), (0.9, 0.9, 0.2), (0.2, 0.2, 0.2)],
                         **dict(RULES, tolerance=1.0))
    assert act == [1, 2, 0]  # 9B overloads next: on to variant 2; calm: straight back to variant 0


def test_rule_no_eligible_transition_keeps_the_selection():
    dom, q = [1, 1], [0.9, 0.9]
    act, n = ob.simulate(dom, q, [0, 1, 2], [(0.9, 0.9)] * 3, **RULES)
    assert act == [0, 0, 0] and n == 0


# ---------------------------------------------------------------------------
# library against the oracle
# ---------------------------------------------------------------------------

def test_walkthrough_through_the_library():
    prob, model = walkthrough()
    for pi in (PI0, PI1):
        dem, dom, q = D.annotate(prob, pi, model, 2)
        want = ob.annotate(prob, pi, model, 2)
        assert dem.tolist() == want[0] and dom == want[1] and q == want[2]


def test_annotate_random_plans_match_oracle():
    rng = np.random.default_rng(21)
    for trial in range(200):
        n = int(rng.integers(1, 12))
        R = int(rng.integers(1, 8))
        nm = int(rng.integers(1, 5))
        prob = wl.Problem(n_nodes=n, edges=np.zeros((0, 2), np.int32), radix=rng.integers(1, R + 1, n).astype(np.int32),
                          p=rng.uniform(0, 1, (n, R)).astype(np.float32),
                          tau=rng.choice([0.0, 1.0, 2.5, rng.lognormal()], (n, R)).astype(np.float32),
                          size=np.ones((n, R), np.float32), backend=np.zeros((n, R), np.int32),
                          w=rng.uniform(0, 1, n).astype(np.float32), rho=np.zeros((1, 1), np.float32), slo=1.0)
        model = rng.integers(0, nm, (n, R)).astype(np.int32)
        impl = [int(rng.integers(0, r)) for r in prob.radix]
        obj = None
        tools = None
        if trial % 3 == 0:
            tools = (rng.random(n) < 0.4).astype(np.int32)
            obj = wl.paper_objective(prob, is_tool=tools)
        dem, dom, q = D.annotate(prob, impl, model, nm, obj)
        want = ob.annotate(prob, impl, model, nm, tools)
        assert dem.tolist() == want[0] and dom == want[1] and q == want[2], trial


def test_annotate_rejects_bad_ids():
    prob, model = walkthrough()
    with pytest.raises(D.DyplanError):
        D.annotate(prob, [0, 3, 0, 0, 0], model, 2)
    bad = model.copy()
    bad[1, 0] = 2
    with pytest.raises(D.DyplanError):
        D.annotate(prob, PI0, bad, 2)


def test_simulate_random_traces_match_oracle():
    rng = np.random.default_rng(5)
    for trial in range(60):
        K = int(rng.integers(1, 9))
        nm = int(rng.integers(1, 5))
        dom = rng.integers(-1, nm, K).tolist()
        q = rng.uniform(0.5, 1.0, K).round(2).tolist()
        T = int(rng.integers(1, 3000))
        times = np.cumsum(rng.exponential(1.0, T)).round(1)
        loads = rng.uniform(0, 1, (T, nm)).round(2)
        rules = dict(high=float(rng.uniform(0.5, 0.95)), low=float(rng.uniform(0.05, 0.5)),
                     tolerance=float(rng.choice([0.0, 0.05, 0.2, 1.0])), margin=float(rng.choice([0.0, 0.1])),
                     dwell=float(rng.choice([0.0, 2.0, 10.0])))
        act, n = D.simulate(dom, q, times, loads, **rules)
        want, wn = ob.simulate(dom, q, times.tolist(), loads.tolist(), **rules)
        assert act.tolist() == want and n == wn, trial


# ---------------------------------------------------------------------------
# GPU: a selected bundle, annotated and replayed
# ---------------------------------------------------------------------------

@pytest.mark.gpu
def test_bundle_of_selected_variants():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)
    prob = wl.forkjoin8()
    obj = wl.paper_objective(prob, levels=(0.0, 1.5, 3.0, 6.0, 12.0))
    model, nm = wl.model_table(prob)
    begin, count = 0, 1 << 22  # a slice of the space the oracle scans in seconds
    with D.Plan((prob, obj)) as plan:
        got = plan.select([D.range_source(0, begin, count)], stream=torch.cuda.current_stream())[0]
    want = orc.obj_select_range(prob, obj, begin, count)
    dom_g, q_g, dom_o, q_o = [], [], [], []
    for g, w in zip(got, want):
        assert g[0] == w[0]
        impl = [(g[0] // 12 ** (7 - i)) % 12 for i in range(8)]
        dem, dom, q = D.annotate(prob, impl, model, nm, obj)
        wd, wdom, wq = ob.annotate(prob, impl, model, nm, None)
        assert dem.tolist() == wd and dom == wdom and q == wq
        dom_g.append(dom)
        q_g.append(q)
    rng = np.random.default_rng(9)
    T = 5000
    times = np.arange(T, dtype=np.float64)
    loads = np.clip(0.3 + 0.6 * np.sin(times[:, None] / 300.0 + np.arange(nm)) + rng.normal(0, 0.05, (T, nm)), 0, 1)
    act, sw = D.simulate(dom_g, q_g, times, loads, high=0.8, low=0.3, tolerance=0.1, margin=0.05, dwell=30.0)
    want_act, want_sw = ob.simulate(dom_g, q_g, times.tolist(), loads.tolist(), high=0.8, low=0.3, tolerance=0.1,
                                    margin=0.05, dwell=30.0)
    assert act.tolist() == want_act and sw == want_sw
