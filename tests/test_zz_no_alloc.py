"""GPU test of vfl_create_static, the context creation that allocates no
device memory (its workspace is the library's static per-device array).

Two static contexts in a row, the second on a smaller batch, train bitwise
like vfl_create contexts on a caller-allocated workspace given the same
seeded inputs: parameters, per-group losses and the last embedding and
gradient messages with their headers.  The first also replays graphs
(vfl_run) on the static workspace.  Host-side refusals (a configuration
larger than the array, a second holder of the array) are checked while the
first static context is alive."""
import numpy as np
import pytest

import vfl_synth as S

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("needs an MI355X")


def _open(w, n_groups, static):
    from paper_2510_12494_amd.session import Session
    n = n_groups * w.rows_per_tick
    d = S.generate(w, n)
    p = S.init_params(w)
    sess = Session(w, d, p, lambda g: S.group_rows(w, g, n), static_ws=static)
    return sess, {k: v.shape for k, v in p.items()}


def _train(sess, shapes, w, run_ticks):
    """2(s+1) per-call ticks, then run_ticks replayed ticks; the results."""
    import torch
    s = w.staleness
    t0 = 2 * (s + 1)
    for t in range(t0):
        sess.step(t)
    if run_ticks:
        sess.bind()
        sess.run(t0, run_ticks)
    T = t0 + run_ticks
    torch.cuda.synchronize()
    out = {"params": sess.params(shapes), "loss": sess.losses(range(T - s))}
    out["emb"] = sess.message(0, T - 1)
    out["grad"] = sess.message(1, T - 1 - s)
    return out


def _same(a, b, tag):
    for k in a["params"]:
        assert np.array_equal(a["params"][k], b["params"][k]), (tag, k)
    assert np.array_equal(a["loss"], b["loss"]), (tag, "loss")
    for m in ("emb", "grad"):
        assert np.array_equal(a[m][0], b[m][0]), (tag, m)
        assert tuple(a[m][1]) == tuple(b[m][1]), (tag, m, "header")


def test_static_workspace_contexts_match_caller_workspace():
    from paper_2510_12494_amd import vfl as V
    from paper_2510_12494_amd.session import bottom_spec, top_spec, opts
    base = S.get("hetero")
    # first call: 4 replicas x 256 rows per tick, graph replay included
    w1 = base.replace(batch=256)
    ref, shapes = _open(w1, 12, static=False)
    try:
        r1 = _train(ref, shapes, w1, 2 * V.VFL_GRAPH_CYCLES * (w1.staleness + 1) + 3)
    finally:
        ref.close()
    st, _ = _open(w1, 12, static=True)
    try:
        assert st.ws is None
        # refusals on the host while the array is held
        big = base  # the full-size configuration needs far more than the array
        with pytest.raises(V.VflError) as e:
            V.vfl_create_static(bottom_spec(big.A), bottom_spec(big.B), top_spec(big.top), opts(big), 0, 0)
        assert e.value.status == V.VFL_E_NOMEM
        with pytest.raises(V.VflError) as e:
            V.vfl_create_static(bottom_spec(w1.A), bottom_spec(w1.B), top_spec(w1.top), opts(w1), 0, 0)
        assert e.value.status == V.VFL_E_STATE
        s1 = _train(st, shapes, w1, 2 * V.VFL_GRAPH_CYCLES * (w1.staleness + 1) + 3)
    finally:
        st.close()
    _same(r1, s1, "first")
    # second call: a smaller batch (100 rows per replica, ragged against the
    # kernels' tiles) on the same array, which still holds the first run's
    # contents
    w2 = base.replace(batch=100)
    st, shapes2 = _open(w2, 9, static=True)
    try:
        s2 = _train(st, shapes2, w2, 0)
    finally:
        st.close()
    ref, _ = _open(w2, 9, static=False)
    try:
        r2 = _train(ref, shapes2, w2, 0)
    finally:
        ref.close()
    _same(r2, s2, "second")
