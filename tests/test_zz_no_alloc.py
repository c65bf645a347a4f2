"""GPU: dy_plan_select_static, the selection entry point that allocates
nothing (its per-call device memory is the library's fixed array), against
dy_plan_select through the C-ABI: identical choices on two calls in a row,
the second with a smaller input, for range, batched and row sources, and the
documented limit on sources per call.

Bar as in test_gpu_parity.py: indices and feasibility bit-exact, and both
entry points report the winner's fp64 values rounded to fp32, so every field
is compared for equality.
"""
import ctypes

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import oracle as orc  # noqa: E402
from paper_2607_02942_amd import dyplan as D  # noqa: E402
from paper_2607_02942_amd import workload as wl  # noqa: E402

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    D.lib()
    torch.cuda.set_device(0)
    yield


def stream():
    return torch.cuda.current_stream()


def same(a, b, ctx):
    assert len(a) == len(b), ctx
    for j, (ra, rb) in enumerate(zip(a, b)):
        assert len(ra) == len(rb), ctx
        for k, (x, y) in enumerate(zip(ra, rb)):
            assert x[0] == y[0] and x[1] == y[1], f"{ctx} source {j} level {k}: static {x} select {y}"
            for u, v in zip(x[2:], y[2:]):
                assert u == v or (np.isnan(u) and np.isnan(v)), f"{ctx} source {j} level {k}: {x} vs {y}"


def both(plan, sources):
    st = plan.select(sources, stream=stream(), static=True)
    ref = plan.select(sources, stream=stream())
    return st, ref


def test_static_range_sources_two_calls():
    prob = wl.forkjoin8()
    with D.Plan(prob) as plan:
        st, ref = both(plan, [D.range_source(0, 0, 12 ** 8)])
        same(st, ref, "forkjoin8 full space")
        st, ref = both(plan, [D.range_source(0, 123457, 1000003)])  # second call, smaller
        same(st, ref, "forkjoin8 [123457 + 1000003]")
    chain = wl.chain4()
    with D.Plan(chain) as plan:
        st = plan.select([D.range_source(0, 0, chain.n_plans())], stream=stream(), static=True)
        want = orc.select_range(chain, 0, chain.n_plans())
        for g, w in zip(st[0], want):
            assert (g[0], g[1]) == (w[0], w[1])


def test_static_batch_two_calls():
    probs = wl.batch6(64)
    with D.Plan(probs) as plan:
        srcs = [D.range_source(r, 0, 12 ** 6) for r in range(64)]
        st, ref = both(plan, srcs)
        same(st, ref, "batch6 64 requests")
        srcs = [D.range_source(r, 1000, 500000) for r in range(10)]  # fewer, smaller sources
        st, ref = both(plan, srcs)
        same(st, ref, "batch6 10 partial requests")


def test_static_rows_two_calls():
    prob = wl.stream24()
    n1, n2 = 1 << 21, 300007
    rows = wl.make_rows(n1, 24, 36)
    d = torch.from_numpy(rows).cuda()
    with D.Plan(prob) as plan:
        st, ref = both(plan, [D.rows_source(0, d, n1, 24, 0)])
        same(st, ref, "stream24 rows")
        st, ref = both(plan, [D.rows_source(0, d[7:], n2, 24, 7)])
        same(st, ref, "stream24 rows, second call smaller")
        want = orc.select_rows(prob, rows[7:7 + n2], 7)
        for g, w in zip(st[0], want):
            assert (g[0], g[1]) == (w[0], w[1])


def test_static_rejects_more_sources_than_the_array_holds():
    probs = wl.batch6(65)
    with D.Plan(probs) as plan:
        srcs = (D.DySource * 65)(*[D.range_source(r, 0, 1000) for r in range(65)])
        out = (D.DyChoice * (65 * plan.kmax))()
        rc = D.lib().dy_plan_select_static(plan._h, srcs, 65, out, ctypes.c_void_p(None))
        assert rc == D.DY_ELIMIT
        assert "64" in D.last_error(plan._h)
        # the handle still works through both entry points
        st, ref = both(plan, [D.range_source(r, 0, 1000) for r in range(64)])
        same(st, ref, "64 sources after a rejected call")
