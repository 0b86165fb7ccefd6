"""GPU tests of the C ABI's channel state machine, error codes and
determinism (through the ctypes binding)."""
import numpy as np
import pytest

import vfl_synth as S
import gpu_harness as H

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("needs an MI355X")


def _session(name="dense_tabular", groups=6, **kw):
    from paper_2510_12494_amd.session import Session
    w = S.get(name).replace(**kw)
    n = groups * w.rows_per_tick
    d = S.generate(w, n)
    p = S.init_params(w)
    return w, Session(w, d, p, lambda g: S.group_rows(w, g, n)), p


def test_protocol_errors():
    from paper_2510_12494_amd import vfl as V
    w, s, _ = _session(staleness=1)
    try:
        # A cannot subscribe to a group B has not published
        V.vfl_bottom_forward(s.ctx, V.VFL_PARTY_A, 0, s.batches("A", 0))
        with pytest.raises(V.VflError) as e:
            V.vfl_top_step(s.ctx, 0, 0)
        assert e.value.status == V.VFL_E_NOT_READY
        # B publishes 0 and 1 (s + 1 = 2 in flight); a third is stale
        for g in (0, 1):
            V.vfl_bottom_forward(s.ctx, V.VFL_PARTY_B, g, s.batches("B", g))
            V.vfl_publish(s.ctx, g)
        with pytest.raises(V.VflError) as e:
            V.vfl_bottom_forward(s.ctx, V.VFL_PARTY_B, 2, s.batches("B", 2))
        assert e.value.status == V.VFL_E_STALE
        # out-of-order groups
        with pytest.raises(V.VflError) as e:
            V.vfl_publish(s.ctx, 5)
        assert e.value.status == V.VFL_E_STATE
        with pytest.raises(V.VflError) as e:
            V.vfl_bottom_backward(s.ctx, V.VFL_PARTY_B, 1)
        assert e.value.status == V.VFL_E_STATE
        # B's backward of 0 before its gradient exists
        with pytest.raises(V.VflError) as e:
            V.vfl_bottom_backward(s.ctx, V.VFL_PARTY_B, 0)
        assert e.value.status == V.VFL_E_NOT_READY
        # the legal continuation works and frees a slot
        V.vfl_top_step(s.ctx, 0, 0)
        V.vfl_bottom_backward(s.ctx, V.VFL_PARTY_A, 0)
        V.vfl_bottom_backward(s.ctx, V.VFL_PARTY_B, 0)
        V.vfl_bottom_forward(s.ctx, V.VFL_PARTY_B, 2, s.batches("B", 2))
        V.vfl_publish(s.ctx, 2)
        assert V.vfl_check(s.ctx) == (0, 0)
        # misaligned dense rows are rejected
        b = s.batches("B", 3)
        b[0].dense += 2
        with pytest.raises(V.VflError) as e:
            V.vfl_bottom_forward(s.ctx, V.VFL_PARTY_A, 1, b)
        assert e.value.status == V.VFL_E_INVALID
    finally:
        s.close()


@pytest.mark.parametrize("name", ["dense_tabular", "ctr", "private", "hetero"])
def test_individual_calls_equal_vfl_step(name):
    """Driving the phases one call at a time in the schedule's order gives
    bitwise the same parameters as vfl_step: tables (ctr), clip and noise
    (private), B's wide-layer product (hetero)."""
    from paper_2510_12494_amd import vfl as V
    w, s1, p = _session(name, groups=5)
    w, s2, _ = _session(name, groups=5)
    shapes = {k: v.shape for k, v in p.items()}
    try:
        for t in range(5 + w.staleness):
            s1.step(t, 5)
            if t < 5:
                V.vfl_bottom_forward(s2.ctx, V.VFL_PARTY_B, t, s2.batches("B", t))
                V.vfl_publish(s2.ctx, t)
            u = t - w.staleness
            if 0 <= u < 5:
                V.vfl_bottom_forward(s2.ctx, V.VFL_PARTY_A, u, s2.batches("A", u))
                V.vfl_top_step(s2.ctx, u, 0)
                V.vfl_bottom_backward(s2.ctx, V.VFL_PARTY_A, u)
                V.vfl_bottom_backward(s2.ctx, V.VFL_PARTY_B, u)
        a, b = s1.params(shapes), s2.params(shapes)
        for k in a:
            assert np.array_equal(a[k], b[k]), k
    finally:
        s1.close()
        s2.close()


@pytest.mark.parametrize("name", ["private", "ctr"])
def test_deterministic_and_overlap_independent(name):
    """Two runs give bitwise equal parameters, whether the party streams
    overlap freely or every tick is synchronised (which serialises them)."""
    import torch
    w = S.get(name)
    n = 5 * w.rows_per_tick
    d = S.generate(w, n)
    p = S.init_params(w)
    shapes = {k: v.shape for k, v in p.items()}
    from paper_2510_12494_amd.session import Session
    outs = []
    for serial in (False, True):
        s = Session(w, d, p, lambda g: S.group_rows(w, g, n))
        try:
            for t in range(5 + w.staleness):
                s.step(t, 5)
                if serial:
                    torch.cuda.synchronize()
            outs.append(s.params(shapes))
        finally:
            s.close()
    for k in outs[0]:
        assert np.array_equal(outs[0][k], outs[1][k]), k


def test_discard_protocol():
    """vfl_discard takes only A's next group, between A's steps; without
    VFL_FIFO_DISCARD a full channel stays VFL_E_STALE; graph replay and
    state images wait until B has released a discarded group."""
    from paper_2510_12494_amd import vfl as V
    w, sess, p = _session(groups=8)
    s = w.staleness
    try:
        for t in range(s + 1):
            sess.step(t, 8)
        u = 1                                   # A's next group
        for bad in (u + 1, u - 1):
            with pytest.raises(V.VflError) as e:
                V.vfl_discard(sess.ctx, bad)
            assert e.value.status == V.VFL_E_STATE
        V.vfl_bottom_forward(sess.ctx, V.VFL_PARTY_A, u, sess.batches("A", u))
        with pytest.raises(V.VflError) as e:
            V.vfl_discard(sess.ctx, u)              # A inside its step
        assert e.value.status == V.VFL_E_STATE
        V.vfl_top_step(sess.ctx, u, 0)
        V.vfl_bottom_backward(sess.ctx, V.VFL_PARTY_A, u)
        V.vfl_bottom_backward(sess.ctx, V.VFL_PARTY_B, u)
        V.vfl_discard(sess.ctx, u + 1)          # the deadline path
        sess.bind()
        with pytest.raises(V.VflError) as e:
            sess.run(s + 1, 12)
        assert e.value.status == V.VFL_E_STATE
        with pytest.raises(V.VflError) as e:
            V.vfl_get_state(sess.ctx)
        assert e.value.status == V.VFL_E_STATE
        # B: forward and publish s + 1 groups ahead, then one more: stale
        for g in range(s + 1, 2 * s + 3):
            if g <= u + 1 + s:
                V.vfl_bottom_forward(sess.ctx, V.VFL_PARTY_B, g, sess.batches("B", g))
                V.vfl_publish(sess.ctx, g)
        g = u + 2 + s
        with pytest.raises(V.VflError) as e:
            V.vfl_bottom_forward(sess.ctx, V.VFL_PARTY_B, g, sess.batches("B", g))
        assert e.value.status == V.VFL_E_STALE
        # B's backward releases the discarded group, then the forward goes on
        V.vfl_bottom_backward(sess.ctx, V.VFL_PARTY_B, u + 1)
        V.vfl_bottom_forward(sess.ctx, V.VFL_PARTY_B, g, sess.batches("B", g))
    finally:
        sess.close()
