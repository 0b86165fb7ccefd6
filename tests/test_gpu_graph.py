"""Graph replay (vfl_run over a bound resident dataset) against the per-call
path (vfl_step with host-built batches): bitwise equal parameters, losses,
traces and channel checks, across epoch wraps and short last groups."""
import numpy as np
import pytest

import vfl_synth as S
from vfl_synth.workloads import Workload, PartySpec, TopSpec

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("needs an MI355X")


def _wide():
    """Party B's first layer at least 512 wide (its layer-1 input gradient is
    a layer product reading rows from the tick record), ragged widths."""
    return Workload(name="wide", n_rows=1401, dtype="bf16",
                    A=PartySpec(dense=24, widths=[32, 16]), B=PartySpec(dense=33, widths=[600, 264, 24]),
                    top=TopSpec(widths=[20, 1]), batch=300, staleness=2, replicas=2, lr=0.5,
                    clip=1.0, sigma=0.5, clip_emb=True, clip_grad=True, noise_emb=True,
                    noise_grad=True, labels="teacher", data_seed=71, init_seed=72, noise_seed=73)


def _get(name):
    return _wide() if name == "wide" else S.get(name)


def _pair(w, n_rows):
    from paper_2510_12494_amd.session import Session
    d = S.generate(w, n_rows)
    p = S.init_params(w)
    rows_of = lambda g: S.group_rows(w, g, n_rows)
    return p, Session(w, d, p, rows_of), Session(w, d, p, rows_of)


@pytest.mark.parametrize("name,extra_rows", [("dense_tabular", 1000), ("private", 3000),
                                              ("ctr", 777), ("tiny_sync", 0), ("hetero", 5000),
                                              ("wide", 77)])
def test_graph_run_equals_per_call_steps(name, extra_rows):
    from paper_2510_12494_amd import vfl as V
    w = _get(name)
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
        assert V.vfl_check(s1.ctx) == (0, 0) and V.vfl_check(s2.ctx) == (0, 0)
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


def test_graph_run_after_a_discard():
    """A discarded group leaves B's version one update behind the schedule's
    max(0, g - s): vfl_run refuses while groups published before the drop
    are in flight, and after s + 1 more ticks its replays write the headers
    and parameters of the per-call path (bitwise)."""
    from paper_2510_12494_amd import vfl as V
    w = S.get("dense_tabular").replace(fifo_discard=False)
    R = w.rows_per_tick
    n_rows = 7 * R + 300
    epoch = (n_rows + R - 1) // R
    s = w.staleness
    drop = 4
    p, s1, s2 = _pair(w, n_rows)
    shapes = {k: v.shape for k, v in p.items()}
    ticks = drop + s + 1 + (s + 1) + 2 * 4 * (s + 1)
    try:
        for sess in (s1, s2):
            sess.bind()
        t_run = None
        for t in range(ticks):
            for sess in (s1, s2):
                if t - s == drop:
                    V.vfl_discard(sess.ctx, drop)
            s1.step(t, epoch=epoch)
            if t_run is None:
                if t > drop + s:
                    # groups drop+1 .. t-1 ... in flight: the run is refused until
                    # every group in flight was published after the drop was applied
                    try:
                        s2.run(t, ticks - t)
                        t_run = t
                    except V.VflError as e:
                        assert e.status == V.VFL_E_STATE
                        s2.step(t, epoch=epoch)
                else:
                    s2.step(t, epoch=epoch)
        # group drop + s + 1 is the first published with the drop applied
        assert t_run == drop + 2 * s + 1
        a, b = s1.params(shapes), s2.params(shapes)
        for k in a:
            assert np.array_equal(a[k], b[k]), k
        assert V.vfl_get_trace(s1.ctx) == V.vfl_get_trace(s2.ctx)
        for g in range(ticks - s, ticks):
            assert s1.message(0, g)[1] == s2.message(0, g)[1]
        for g in range(ticks - 2 * s - 1, ticks - s):
            assert s1.message(1, g)[1] == s2.message(1, g)[1]
        assert V.vfl_check(s1.ctx) == (0, 0) and V.vfl_check(s2.ctx) == (0, 0)
    finally:
        s1.close()
        s2.close()
