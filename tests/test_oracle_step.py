"""Pins for the oracle's training loop (oracle/pubsub.py).

* closed form: linear bottoms and a logistic top reduce the step to logistic
  regression, whose gradient is known analytically;
* finite differences of the loss on a tiny model with embedding tables,
  ReLUs, and the clipped + noised exchanged embedding;
* an independently written PyTorch float64 formulation (tests/torch_reference.py)
  with a full history of B's parameter versions: s = 0 is synchronous
  centralized SGD, s > 0 the delayed update rule, k replicas the row-weighted
  parameter-server mean;
* the integer schedule trace against its closed form;
* precision-emulation modes store what the GPU stores.
"""
import numpy as np
import pytest

import vfl_synth as S
from vfl_synth.workloads import Workload, PartySpec, TopSpec
from oracle import PubSubOracle, schedule
from oracle.rounding import round_bf16
from torch_reference import run_history


def _mk(**kw):
    base = dict(name="t", n_rows=40, dtype="f32",
                A=PartySpec(dense=3, widths=[4, 3]), B=PartySpec(dense=4, widths=[5, 2]),
                top=TopSpec(widths=[3, 1]), batch=10, staleness=0, replicas=1, lr=0.1,
                labels="bernoulli", label_p=0.5, data_seed=11, init_seed=12, noise_seed=13)
    base.update(kw)
    return Workload(**base)


def _run(w, n_groups, precision="f64", **kw):
    d = S.generate(w)
    p = S.init_params(w)
    o = PubSubOracle(w, p, precision)
    recs = o.run(d, n_groups, lambda g: S.group_rows(w, g), **kw)
    return o, recs, d, p


def _relerr(a, b):
    return np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300)


# ------------------------------------------------------------ closed form
def test_closed_form_logistic_regression():
    """Linear one-layer bottoms, logit top: the step is logistic regression
    on x = [x_A | x_B] with r = sigmoid(l) - y:
    dL/du_X = Z_X^T r / R, dL/dW_X = u_X (r^T X_X) / R, dL/db_X = u_X sum(r)/R,
    dL/dc = sum(r)/R."""
    w = _mk(A=PartySpec(dense=3, widths=[2], relu=[False]),
            B=PartySpec(dense=4, widths=[3], relu=[False]),
            top=TopSpec(widths=[1]), batch=25, n_rows=25, lr=0.3)
    o, recs, d, p = _run(w, 1, keep_grads=True)
    R = 25
    XA, XB, y = d["xa"].astype(float), d["xb"].astype(float), d["y"].astype(float)
    ZA = XA @ p["A.W0"].T.astype(float) + p["A.b0"]
    ZB = XB @ p["B.W0"].T.astype(float) + p["B.b0"]
    u = p["top.W0"][0].astype(float)
    c = float(p["top.b0"][0])
    l = np.concatenate([ZA, ZB], 1) @ u + c
    r = 1.0 / (1.0 + np.exp(-l)) - y
    uA, uB = u[:2], u[2:]
    want = {"top.W0": np.concatenate([ZA, ZB], 1).T @ r / R,
            "top.b0": np.array([r.sum() / R]),
            "A.W0": np.outer(uA, r @ XA) / R, "A.b0": uA * r.sum() / R,
            "B.W0": np.outer(uB, r @ XB) / R, "B.b0": uB * r.sum() / R}
    g = recs[0]["grads"]
    for k, v in want.items():
        np.testing.assert_allclose(g[k].reshape(v.shape) / R, v, rtol=1e-12, atol=1e-15)
        np.testing.assert_allclose(o.p[k].reshape(v.shape),
                                   p[k].astype(float).reshape(v.shape) - w.lr * v, rtol=1e-12)
    loss = np.mean(np.maximum(l, 0) - y * l + np.log1p(np.exp(-np.abs(l))))
    assert abs(recs[0]["loss"] - loss) < 1e-13


def test_closed_form_linear_regression():
    """Linear one-layer bottoms and a linear output with the squared error:
    the prediction is l = u . [Z_A | Z_B] + c and, with r = 2 (l - y),
    dL/du = [Z_A | Z_B]^T r / R, dL/dW_X = u_X (r^T X_X) / R,
    dL/db_X = u_X sum(r) / R, dL/dc = sum(r) / R (the least-squares
    gradient); the loss is the mean of (l - y)^2."""
    w = _mk(A=PartySpec(dense=3, widths=[2], relu=[False]),
            B=PartySpec(dense=4, widths=[3], relu=[False]),
            top=TopSpec(widths=[1]), batch=25, n_rows=25, lr=0.3, labels="regression",
            loss="mse")
    o, recs, d, p = _run(w, 1, keep_grads=True)
    R = 25
    XA, XB, y = d["xa"].astype(float), d["xb"].astype(float), d["y"].astype(float)
    assert len(np.unique(y)) == R          # real-valued targets
    ZA = XA @ p["A.W0"].T.astype(float) + p["A.b0"]
    ZB = XB @ p["B.W0"].T.astype(float) + p["B.b0"]
    u = p["top.W0"][0].astype(float)
    c = float(p["top.b0"][0])
    l = np.concatenate([ZA, ZB], 1) @ u + c
    r = 2.0 * (l - y)
    uA, uB = u[:2], u[2:]
    want = {"top.W0": np.concatenate([ZA, ZB], 1).T @ r / R,
            "top.b0": np.array([r.sum() / R]),
            "A.W0": np.outer(uA, r @ XA) / R, "A.b0": uA * r.sum() / R,
            "B.W0": np.outer(uB, r @ XB) / R, "B.b0": uB * r.sum() / R}
    g = recs[0]["grads"]
    for k, v in want.items():
        np.testing.assert_allclose(g[k].reshape(v.shape) / R, v, rtol=1e-12, atol=1e-15)
        np.testing.assert_allclose(o.p[k].reshape(v.shape),
                                   p[k].astype(float).reshape(v.shape) - w.lr * v, rtol=1e-12)
    assert abs(recs[0]["loss"] - np.mean((l - y) ** 2)) < 1e-13


# ------------------------------------------------------ finite differences
def _fd_workload(loss="bce"):
    return _mk(A=PartySpec(dense=3, n_cat=2, vocab=7, emb_dim=2, widths=[4, 3]),
               B=PartySpec(dense=2, n_cat=2, vocab=7, emb_dim=2, widths=[4, 2]),
               top=TopSpec(widths=[3, 1]), n_rows=5, batch=5, clip=0.3,
               clip_emb=True, noise_emb=True, sigma=0.5, zipf_a=0.5,
               loss=loss, labels="regression" if loss == "mse" else "bernoulli")


@pytest.mark.parametrize("loss", ["bce", "mse"])
def test_finite_differences_whole_step(loss):
    w = _fd_workload(loss)
    d = S.generate(w)
    p0 = S.init_params(w)

    def loss_at(p):
        o = PubSubOracle(w, p, "f64")
        return o.run(d, 1, lambda g: S.group_rows(w, g), keep_messages=False)[0]["loss"]

    o = PubSubOracle(w, p0, "f64")
    rec = o.run(d, 1, lambda g: S.group_rows(w, g), keep_grads=True)[0]
    grads = rec["grads"]
    # the clip must bind on some rows and not on others
    n = o.S[0]["parts"][0]["n"]
    assert np.any(n > w.clip) and np.any(n < w.clip)
    h = 1e-6
    checked = 0
    for k, v in p0.items():
        g = grads[k] / 5.0
        flat = v.astype(np.float64).ravel()
        fd = np.zeros_like(flat)
        for i in range(flat.size):
            pp = {kk: vv.astype(np.float64).copy() for kk, vv in p0.items()}
            pm = {kk: vv.astype(np.float64).copy() for kk, vv in p0.items()}
            pp[k].ravel()[i] += h
            pm[k].ravel()[i] -= h
            fd[i] = (loss_at(pp) - loss_at(pm)) / (2 * h)
        scale = max(np.max(np.abs(fd)), 1e-3)
        assert np.max(np.abs(g.ravel() - fd)) < 1e-6 * scale + 1e-9, k
        checked += flat.size
    assert checked > 150


# ------------------------------------------- independent torch formulation
@pytest.mark.parametrize("s,k,loss", [(0, 1, "bce"), (1, 1, "bce"), (2, 2, "bce"), (3, 1, "bce"),
                                      (4, 4, "bce"), (2, 2, "mse")])
def test_equals_history_formulation(s, k, loss):
    """Ring + stash oracle == full-version-history torch autograd, with the
    private workload's clip and noise on both messages and embedding tables
    on both parties; k replicas == one batch of k * B rows; BCE and the
    squared error of a regression output."""
    w = _mk(A=PartySpec(dense=3, n_cat=2, vocab=7, emb_dim=2, widths=[6, 3]),
            B=PartySpec(dense=4, n_cat=1, vocab=5, emb_dim=3, widths=[5, 4]),
            top=TopSpec(widths=[5, 1]), staleness=s, replicas=k, batch=12 // k,
            n_rows=12 * 7 - 5, lr=0.5 if loss == "bce" else 0.05, clip=0.7, sigma=0.3,
            clip_emb=True, clip_grad=True, noise_emb=True, noise_grad=True, zipf_a=0.8,
            loss=loss, labels="regression" if loss == "mse" else "bernoulli")
    n_groups = 9          # wraps the 7-group epoch; its last group is short
    o, recs, d, p = _run(w, n_groups)
    losses, final = run_history(w, p, d, n_groups, lambda g: S.group_rows(w, g))
    got = [r["loss"] for r in recs if "loss" in r]
    np.testing.assert_allclose(got, losses, rtol=1e-13)
    for key, v in final.items():
        assert _relerr(o.p[key], v) < 1e-12, key
        d0 = p[key].astype(np.float64)
        assert _relerr(o.p[key] - d0, v - d0) < 1e-10, key


@pytest.mark.parametrize("s,discard", [(0, {1: "emb", 3: "grad"}),
                                       (2, {0: "grad", 2: "emb", 3: "emb", 6: "grad"})])
def test_discards_equal_history_formulation(s, discard):
    """Dropped embeddings and gradients (Section 4.1 "System Design"): the oracle's ring,
    stash and version counter against the history formulation, where B's
    forward of group u takes the version counted from the groups applied
    before it; with clip, noise and tables."""
    w = _mk(A=PartySpec(dense=3, n_cat=2, vocab=7, emb_dim=2, widths=[6, 3]),
            B=PartySpec(dense=4, n_cat=1, vocab=5, emb_dim=3, widths=[5, 4]),
            top=TopSpec(widths=[5, 1]), staleness=s, replicas=2, batch=6,
            n_rows=12 * 8, lr=0.5, clip=0.7, sigma=0.3, clip_emb=True,
            clip_grad=True, noise_emb=True, noise_grad=True, zipf_a=0.8)
    n_groups = 8
    o, recs, d, p = _run(w, n_groups, discard=discard)
    losses, final = run_history(w, p, d, n_groups, lambda g: S.group_rows(w, g), discard=discard)
    got = [r["loss"] for r in recs if "loss" in r]
    np.testing.assert_allclose(got, losses, rtol=1e-13)
    for key, v in final.items():
        assert _relerr(o.p[key], v) < 1e-12, key
    # B's version: one step per group it did not drop; A skipped the
    # dropped embeddings only
    assert o.vB == n_groups - len(discard)
    assert len(got) == n_groups - sum(1 for k in discard.values() if k == "emb")
    # a dropped group leaves B untouched over its tick, and a dropped
    # embedding leaves A untouched too
    vb = [r for r in o.trace if r[4] >= 0]
    for row in vb:
        u = row[4]
        applied = sum(1 for g in range(u + 1) if g not in discard)
        assert row[6] == applied, row


def test_synchronous_equals_centralized_sgd():
    """s = 0, k = 1, no clip or noise: one tick is one SGD step of the
    centralized network g([f_A(x_A) | f_B(x_B)]) on the batch mean BCE."""
    w = _mk(staleness=0, replicas=1, batch=8, n_rows=32)
    o, recs, d, p = _run(w, 4)
    losses, final = run_history(w, p, d, 4, lambda g: S.group_rows(w, g))
    np.testing.assert_allclose([r["loss"] for r in recs], losses, rtol=1e-13)
    for key, v in final.items():
        assert _relerr(o.p[key], v) < 1e-13


def test_replicas_equal_one_big_batch():
    base = dict(A=PartySpec(dense=3, widths=[4, 3]), B=PartySpec(dense=4, widths=[5, 2]),
                top=TopSpec(widths=[3, 1]), n_rows=96, staleness=2, clip=1.0, sigma=0.5,
                clip_emb=True, clip_grad=True, noise_emb=True, noise_grad=True)
    o1, r1, _, _ = _run(_mk(replicas=4, batch=6, **base), 4)
    o2, r2, _, _ = _run(_mk(replicas=1, batch=24, **base), 4)
    for k in o1.p:
        assert _relerr(o1.p[k], o2.p[k]) < 1e-13
    for a, b in zip(r1, r2):
        if "zhat" in a:
            np.testing.assert_allclose(a["zhat"], b["zhat"], rtol=1e-14, atol=1e-15)
        if "gtilde" in a:
            np.testing.assert_allclose(a["gtilde"], b["gtilde"], rtol=1e-13, atol=1e-14)


# ----------------------------------------------------------------- schedule
@pytest.mark.parametrize("s", [0, 1, 2, 3, 4])
def test_trace_closed_form(s):
    w = _mk(staleness=s, n_rows=60, batch=10)
    n_groups = 6 + s
    o, recs, _, _ = _run(w, n_groups)
    assert o.trace == schedule.trace(s, n_groups)
    for r in recs:
        if r["fwd_group"] >= 0:
            g = r["fwd_group"]
            assert r["emb_header"] == (g, r["tick"], max(0, g - s))
        if r["bwd_group"] >= 0:
            u = r["bwd_group"]
            assert r["grad_header"] == (u, r["tick"], max(0, u - s))
            assert r["tick"] - u == s               # delay of the message
            assert r["tick"] - u <= 4               # within the p = 5 buffer


# ---------------------------------------------------------------- precision
def test_bf16_mode_stores_bf16_and_stays_close():
    w = _mk(dtype="bf16", staleness=1, replicas=2, batch=8, n_rows=64,
            clip=1.0, sigma=0.5, clip_emb=True, clip_grad=True, noise_emb=True, noise_grad=True)
    d = S.generate(w)
    p = S.init_params(w)
    ob = PubSubOracle(w, p, "bf16")
    rb = ob.run(d, 4, lambda g: S.group_rows(w, g))
    of = PubSubOracle(w, p, "f64")
    rf = of.run(d, 4, lambda g: S.group_rows(w, g))
    for r in rb:
        for key in ("zhat", "gtilde"):
            if key in r:
                assert np.array_equal(round_bf16(r[key]), r[key])
    for k in ob.p:
        assert np.array_equal(ob.p[k].astype(np.float32).astype(np.float64), ob.p[k])
        d0 = p[k].astype(np.float64)
        assert _relerr(ob.p[k] - d0, of.p[k] - d0) < 5e-2


def test_ten_layer_bottoms_equal_history_formulation():
    """The paper's bottom model depth (a ten-layer MLP, Section 5 "Models")
    with linear layers between ReLU ones, the squared-error head, s = 3,
    k = 2: the oracle's chains against the autograd formulation."""
    relu = [True, False, True, True, True, False, True, True, True, True]
    w = _mk(A=PartySpec(dense=5, widths=[6, 5, 7, 4, 6, 5, 6, 4, 5, 8], relu=relu),
            B=PartySpec(dense=4, widths=[5, 6, 4, 7, 5, 6, 5, 4, 6, 3], relu=relu[::-1]),
            top=TopSpec(widths=[4, 3, 1]), staleness=3, replicas=2, batch=6, n_rows=12 * 6 - 1,
            lr=0.05, labels="regression", loss="mse")
    o, recs, d, p = _run(w, 8)
    losses, final = run_history(w, p, d, 8, lambda g: S.group_rows(w, g))
    np.testing.assert_allclose([r["loss"] for r in recs if "loss" in r], losses, rtol=1e-13)
    for key, v in final.items():
        assert _relerr(o.p[key], v) < 1e-12, key
        d0 = p[key].astype(np.float64)
        assert _relerr(o.p[key] - d0, v - d0) < 1e-9, key
