"""Graph replay (vfl_run over a bound resident dataset) against the per-call
path (vfl_step with host-built batches): bitwise equal parameters, losses,
traces and channel checks, across epoch wraps and short last groups."""
import numpy as np
import pytest

import vfl_synth as S

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("needs an MI355X")


def _pair(w, n_rows):
    from paper_2510_12494_amd.session import Session
    d = S.generate(w, n_rows)
    p = S.init_params(w)
    rows_of = lambda g: S.group_rows(w, g, n_rows)
    return p, Session(w, d, p, rows_of), Session(w, d, p, rows_of)


@pytest.mark.parametrize("name,extra_rows", [("dense_tabular", 1000), ("private", 3000),
                                              ("ctr", 777), ("tiny_sync", 0)])
def test_graph_run_equals_per_call_steps(name, extra_rows):
    from paper_2510_12494_amd import vfl as V
    w = S.get(name)
    R = w.rows_per_tick
    n_rows = 5 * R + extra_rows            # epochs of 5 or 6 groups, the last short
    epoch = (n_rows + R - 1) // R
    ticks = 3 * (w.staleness + 1) * 4 + 2 * (w.staleness + 1) + 3
    p, s1, s2 = _pair(w, n_rows)
    shapes = {k: v.shape for k, v in p.items()}
    try:
        for t in range(ticks):
            s1.step(t, epoch=epoch)
        warm = w.staleness + 1
        for t in range(warm):
            s2.step(t, epoch=epoch)
        s2.bind()
        s2.run(warm, ticks - warm)
        a, b = s1.params(shapes), s2.params(shapes)
        for k in a:
            assert np.array_equal(a[k], b[k]), k
        groups = range(ticks - w.staleness)
        assert np.array_equal(s1.losses(groups), s2.losses(groups))
        assert V.vfl_get_trace(s1.ctx) == V.vfl_get_trace(s2.ctx)
        assert V.vfl_check(s1.ctx) == 0 and V.vfl_check(s2.ctx) == 0
        # the per-call path continues seamlessly after a graph run
        for t in range(ticks, ticks + 2):
            s1.step(t, epoch=epoch)
            s2.step(t, epoch=epoch)
        a, b = s1.params(shapes), s2.params(shapes)
        for k in a:
            assert np.array_equal(a[k], b[k]), k
    finally:
        s1.close()
        s2.close()


def test_graph_run_requires_steady_state():
    from paper_2510_12494_amd import vfl as V
    w = S.get("dense_tabular")
    p, s1, s2 = _pair(w, 4 * w.rows_per_tick)
    try:
        s1.bind()
        with pytest.raises(V.VflError) as e:
            s1.run(0, 12)
        assert e.value.status == V.VFL_E_STATE
    finally:
        s1.close()
        s2.close()
