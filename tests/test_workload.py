"""The seeded workload generator: determinism, DAG shape, distributions, the
native row generator against its numpy twin, and the stored SLOs against the
oracle's lower median (chain4 is small enough to recompute here)."""
import hashlib
import json
import os

import numpy as np

from oracle import oracle as orc
from paper_2607_02942_amd import workload as wl

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _digest(prob):
    h = hashlib.sha256()
    for a in (prob.edges, prob.radix, prob.p, prob.tau, prob.size, prob.backend, prob.w, prob.rho):
        h.update(np.ascontiguousarray(a).tobytes())
    return h.hexdigest()


def test_splitmix64_reference_values():
    # SplitMix64 seeded with 0: first outputs from the published generator
    x = wl.draw(0, np.arange(3, dtype=np.uint64))
    assert [hex(int(v)) for v in x] == ["0xe220a8397b1dcdaf", "0x6e789e6aa1b965f4", "0x6c45d188009454f"]


def test_generation_is_deterministic():
    for f in (wl.chain4, wl.forkjoin8, wl.layered10, wl.stream24):
        assert _digest(f()) == _digest(f())
    assert _digest(wl.batch6_request(17)) == _digest(wl.batch6_request(17))
    assert _digest(wl.batch6_request(17)) != _digest(wl.batch6_request(18))


def _single_source_sink(prob):
    n = prob.n_nodes
    has_pred = np.zeros(n, bool)
    has_succ = np.zeros(n, bool)
    for u, v in prob.edges:
        assert u < v
        has_pred[v] = True
        has_succ[u] = True
    return np.flatnonzero(~has_pred).tolist(), np.flatnonzero(~has_succ).tolist()


def test_dag_shapes():
    c = wl.chain4()
    assert c.edges.tolist() == [[0, 1], [1, 2], [2, 3]]
    f = wl.forkjoin8()
    assert sorted(map(tuple, f.edges.tolist())) == [(0, 1), (0, 2), (0, 3), (1, 4), (2, 5), (3, 6),
                                                     (4, 7), (5, 7), (6, 7)]
    l = wl.layered10()
    assert l.n_edges == 20 and _single_source_sink(l) == ([0], [9])
    s = wl.stream24()
    assert _single_source_sink(s) == ([0], [23])
    for r in range(64):
        b = wl.batch6_request(r)
        assert _single_source_sink(b) == ([0], [5])


def test_table_distributions():
    for f, R, sizes in ((wl.forkjoin8, 12, wl.SIZES_3), (wl.layered10, 36, wl.SIZES_6)):
        p = f()
        assert p.radix.tolist() == [R] * p.n_nodes
        V = 2 if R == 12 else 3
        B = 2
        for m in range(len(sizes)):
            for v in range(V):
                for b in range(B):
                    i = (m * V + v) * B + b
                    base = (m * V + 0) * B + b
                    assert np.all(p.size[:, i] == np.float32(sizes[m]))
                    assert np.all(p.backend[:, i] == b)
                    if v == 0:
                        assert np.all((p.p[:, i] >= 0.6) & (p.p[:, i] <= 0.95))
                    else:
                        gain = (p.p[:, i].astype(np.float64) - p.p[:, base]) / (1 - p.p[:, base].astype(np.float64))
                        assert np.all((gain > 0.3 - 1e-6) & (gain < 0.7 + 1e-6))
                        phi = p.tau[:, i].astype(np.float64) / p.tau[:, base]
                        lo, hi = ((1.3, 2.0), (1.8, 3.0))[v - 1]
                        assert np.all((phi > lo - 1e-5) & (phi < hi + 1e-5))
        assert np.all((p.w >= 0) & (p.w <= 1))
    assert np.allclose(wl.forkjoin8().rho[:, 0], np.linspace(0, 0.9, 8), atol=1e-7)
    assert np.allclose(wl.layered10().rho[:, 1], np.linspace(0, 0.95, 16), atol=1e-7)


def test_native_rows_match_numpy_twin():
    a = wl.make_rows(2048, 24, 36, row_begin=(1 << 28) - 2048)
    b = wl.make_rows_numpy(2048, 24, 36, row_begin=(1 << 28) - 2048)
    assert (a == b).all() and a.max() == 35
    c = wl.make_rows(100, 24, 36, stride=32)
    assert (c[:, :24] == wl.make_rows_numpy(100, 24, 36)).all() and (c[:, 24:] == 0).all()
    counts = np.bincount(wl.make_rows(1 << 15, 24, 36).ravel(), minlength=36)
    assert counts.min() > 0.8 * counts.mean()


def test_stored_slo_is_one_and_a_half_lower_median():
    slo = json.load(open(wl.SLO_FILE))
    prob = wl.chain4(slo=0.0)
    vals = orc.cp0_values(prob, 0, prob.n_plans())
    r = (vals.size - 1) // 2
    med = np.sort(vals)[r]
    assert slo["chain4"] == float(np.float32(1.5 * med))
    for key in ("forkjoin8", "layered10", "stream24"):
        if key in slo:
            assert slo[key] > 0
    if "batch6" in slo:
        assert len(slo["batch6"]) == wl.N_BATCH
        p3 = wl.batch6_request(3, slo=0.0)
        v3 = orc.cp0_values(p3, 0, p3.n_plans())
        assert slo["batch6"][3] == float(np.float32(1.5 * np.sort(v3)[(v3.size - 1) // 2]))
