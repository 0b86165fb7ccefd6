"""Checkpoint and resume through the C ABI (vfl_state_size, vfl_get_state,
vfl_set_state).  A run restored from a state image, into its own context or
into a fresh context on another workspace, continues bitwise as the
uninterrupted run: parameters, losses, channel messages and the schedule
trace, on the per-call path and under graph replay.  Images of another
configuration, truncated or foreign images, and images asked for while A is
inside a group's step are refused, and a refused image leaves the context
as it was."""
import numpy as np
import pytest

import vfl_synth as S

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("needs an MI355X")


def _session(w, d, p, n_rows):
    from paper_2510_12494_amd.session import Session
    return Session(w, d, p, lambda g: S.group_rows(w, g, n_rows))


def _same(sa, sb, shapes, groups, trace=True):
    from paper_2510_12494_amd import vfl as V
    a, b = sa.params(shapes), sb.params(shapes)
    for k in a:
        assert np.array_equal(a[k], b[k]), k
    assert np.array_equal(sa.losses(groups), sb.losses(groups))
    if trace:
        assert V.vfl_get_trace(sa.ctx) == V.vfl_get_trace(sb.ctx)
    assert V.vfl_check(sa.ctx) == (0, 0) and V.vfl_check(sb.ctx) == (0, 0)


@pytest.mark.parametrize("name", ["ctr", "private", "tiny_sync", "hetero"])
def test_restore_continues_bitwise(name):
    """Tables (ctr), clip + noise with two replicas (private), s = 0 float32
    (tiny_sync), s = 4 with four replicas and B's wide-layer product
    (hetero); the image is taken with s groups in flight and a short last
    group ahead."""
    from paper_2510_12494_amd import vfl as V
    w = S.get(name)
    R = w.rows_per_tick
    n_rows = 4 * R + (R // 3 if name != "tiny_sync" else 0)
    epoch = (n_rows + R - 1) // R
    s = w.staleness
    t1 = 2 * (s + 1) + 1
    t2 = t1 + 2 * (s + 1) + 3
    d, p = S.generate(w, n_rows), S.init_params(w)
    shapes = {k: v.shape for k, v in p.items()}
    # a fresh context starts from other parameters: the image must replace them
    p_other = {k: (v * 0.5).astype(v.dtype) for k, v in p.items()}
    ref, run, fresh = _session(w, d, p, n_rows), _session(w, d, p, n_rows), _session(w, d, p_other, n_rows)
    try:
        for t in range(t2):
            ref.step(t, epoch=epoch)
        for t in range(t1):
            run.step(t, epoch=epoch)
        img = V.vfl_get_state(run.ctx)
        assert img.nbytes == V.vfl_state_size(run.ctx)
        # run on past the image, then go back to it and run the same ticks
        for t in range(t1, t2):
            run.step(t, epoch=epoch)
        V.vfl_set_state(run.ctx, img)
        for t in range(t1, t2):
            run.step(t, epoch=epoch)
        V.vfl_set_state(fresh.ctx, img)
        for t in range(t1, t2):
            fresh.step(t, epoch=epoch)
        groups = range(t1 - s, t2 - s)
        _same(ref, run, shapes, groups)
        _same(ref, fresh, shapes, groups)
        # the messages still in the channel slots
        last = t2 - s - 1
        for which, g in ((0, t2 - 1), (1, last)):
            m0, h0 = ref.message(which, g)
            m1, h1 = fresh.message(which, g)
            assert np.array_equal(m0, m1) and h0 == h1, (which, g)
    finally:
        ref.close()
        run.close()
        fresh.close()


def test_restore_under_graph_replay():
    """dense_tabular: graph replay before the image, the image restored into
    a fresh context whose dataset is bound, replay after it."""
    from paper_2510_12494_amd import vfl as V
    w = S.get("dense_tabular")
    R, s = w.rows_per_tick, w.staleness
    n_rows = 5 * R + 500
    epoch = (n_rows + R - 1) // R
    cyc = 4 * (s + 1)
    warm, n1, n2 = s + 1, 2 * cyc, cyc + 2
    d, p = S.generate(w, n_rows), S.init_params(w)
    shapes = {k: v.shape for k, v in p.items()}
    ref, run, fresh = _session(w, d, p, n_rows), _session(w, d, p, n_rows), _session(w, d, p, n_rows)
    try:
        for sess in (ref, run):
            for t in range(warm):
                sess.step(t, epoch=epoch)
            sess.bind()
        ref.run(warm, n1 + n2)
        run.run(warm, n1)
        img = V.vfl_get_state(run.ctx)
        run.run(warm + n1, n2)
        V.vfl_set_state(run.ctx, img)
        run.run(warm + n1, n2)
        fresh.bind()
        V.vfl_set_state(fresh.ctx, img)
        fresh.run(warm + n1, n2)
        groups = range(warm + n1 - s, warm + n1 + n2 - s)
        _same(ref, run, shapes, groups)
        _same(ref, fresh, shapes, groups)
    finally:
        ref.close()
        run.close()
        fresh.close()


def test_image_between_forward_and_publish():
    """B has run the forward of group t but not yet published it: the image
    keeps the unpublished slot, and the restored context publishes it."""
    from paper_2510_12494_amd import vfl as V
    w = S.get("private")
    R, s = w.rows_per_tick, w.staleness
    n_rows = 4 * R
    d, p = S.generate(w, n_rows), S.init_params(w)
    shapes = {k: v.shape for k, v in p.items()}
    ref, run, fresh = _session(w, d, p, n_rows), _session(w, d, p, n_rows), _session(w, d, p, n_rows)
    try:
        t = 2 * (s + 1)
        for sess in (ref, run):
            for tt in range(t):
                sess.step(tt)
        for sess in (ref, run):
            V.vfl_bottom_forward(sess.ctx, V.VFL_PARTY_B, t, sess.batches("B", t))
        img = V.vfl_get_state(run.ctx)
        V.vfl_set_state(fresh.ctx, img)
        for sess in (ref, fresh):
            V.vfl_publish(sess.ctx, t)
            u = t - s
            V.vfl_bottom_forward(sess.ctx, V.VFL_PARTY_A, u, sess.batches("A", u))
            V.vfl_top_step(sess.ctx, u, sess.loss.data_ptr() + 4 * (u % sess.loss.numel()))
            V.vfl_bottom_backward(sess.ctx, V.VFL_PARTY_A, u)
            V.vfl_bottom_backward(sess.ctx, V.VFL_PARTY_B, u)
            sess.step(t + 1)
        _same(ref, fresh, shapes, [t - s, t + 1 - s])
        m0, h0 = ref.message(0, t)
        m1, h1 = fresh.message(0, t)
        assert np.array_equal(m0, m1) and h0 == h1
    finally:
        ref.close()
        run.close()
        fresh.close()


def test_refused_images_leave_the_context_unchanged():
    from paper_2510_12494_amd import vfl as V
    w = S.get("dense_tabular")
    R, s = w.rows_per_tick, w.staleness
    n_rows = 4 * R
    d, p = S.generate(w, n_rows), S.init_params(w)
    shapes = {k: v.shape for k, v in p.items()}
    wt = S.get("tiny_sync")
    dt, pt = S.generate(wt, 4 * wt.rows_per_tick), S.init_params(wt)
    ref, run = _session(w, d, p, n_rows), _session(w, d, p, n_rows)
    other = _session(wt, dt, pt, 4 * wt.rows_per_tick)
    try:
        T = 2 * (s + 1)
        for sess in (ref, run):
            for t in range(T):
                sess.step(t)
        img = V.vfl_get_state(run.ctx)
        foreign = img.copy()
        foreign[0] ^= 0xFF
        bad = [img[: img.nbytes // 2].copy(),     # truncated
               img[:64].copy(),                   # shorter than the header
               foreign,                           # not an image of this library
               V.vfl_get_state(other.ctx)]        # another configuration
        for b in bad:
            with pytest.raises(V.VflError) as e:
                V.vfl_set_state(run.ctx, b)
            assert e.value.status == V.VFL_E_INVALID
        # an image buffer smaller than vfl_state_size
        st = V.library().vfl_get_state(run.ctx, img.ctypes.data, 16)
        assert st == V.VFL_E_INVALID
        # A inside a group's step: no image
        u = T - s
        V.vfl_bottom_forward(run.ctx, V.VFL_PARTY_B, T, run.batches("B", T))
        V.vfl_publish(run.ctx, T)
        V.vfl_bottom_forward(run.ctx, V.VFL_PARTY_A, u, run.batches("A", u))
        with pytest.raises(V.VflError) as e:
            V.vfl_get_state(run.ctx)
        assert e.value.status == V.VFL_E_STATE
        V.vfl_top_step(run.ctx, u, run.loss.data_ptr() + 4 * (u % run.loss.numel()))
        V.vfl_bottom_backward(run.ctx, V.VFL_PARTY_A, u)
        V.vfl_bottom_backward(run.ctx, V.VFL_PARTY_B, u)
        ref.step(T)
        for sess in (ref, run):
            sess.step(T + 1)
        # tick T ran call by call on `run` (no trace row: only vfl_step and
        # vfl_run write them)
        _same(ref, run, shapes, [u, u + 1], trace=False)
    finally:
        ref.close()
        run.close()
        other.close()
