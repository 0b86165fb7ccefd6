"""Pins for the semi-asynchronous workers (oracle/semiasync.py; Section 4.1
"Intra-party Semi-asynchronous Mechanism", Eq. 5, and the aggregation step
of Algorithm 1).

* Eq. 5 against its logistic form: (1 + tanh x) / 2 = 1 / (1 + e^(-2x)), so
  Delta T_t = ceil(dt0 / (1 + exp(4 - 4t/dt0))); bounds, monotonicity, the
  value ceil(dt0/2) at t = dt0, and the Delta T_0 = 5 table and aggregation
  units written out by hand from the logistic form;
* Delta T = 1 with one local step per unit is the row-weighted gradient
  averaging of the k-replica oracle (which the history formulation pins in
  test_oracle_step.py), on ragged groups whose workers hold unequal rows,
  with staleness, clipping and noise;
* right after an average every worker holds the same parameters, and
  between averages the workers drift apart;
* the library's host function vfl_sync_interval equals the oracle.
"""
import math

import numpy as np
import pytest

import vfl_synth as S
from vfl_synth.workloads import Workload, PartySpec, TopSpec
from oracle import PubSubOracle
from oracle.semiasync import SemiAsyncOracle, sync_interval, average_due


def _mk(**kw):
    base = dict(name="sa", n_rows=115, dtype="f32",
                A=PartySpec(dense=3, widths=[5, 3]), B=PartySpec(dense=4, widths=[6, 2]),
                top=TopSpec(widths=[4, 1]), batch=10, staleness=0, replicas=3, lr=0.2,
                labels="bernoulli", label_p=0.5, data_seed=21, init_seed=22, noise_seed=23)
    base.update(kw)
    return Workload(**base)


def _worker_rows(w):
    n = w.n_rows
    return lambda r, g: S.group_rows(w, g, n)[r]


def _rel(a, b):
    return np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300)


# ------------------------------------------------------------- Eq. 5
def _logistic_form(dt0, t):
    return dt0 / (1.0 + math.exp(4.0 - 4.0 * t / dt0))


@pytest.mark.parametrize("dt0", [1, 2, 3, 5, 8, 13, 40])
def test_interval_equals_logistic_form(dt0):
    for t in range(0, 6 * dt0 + 20):
        v = _logistic_form(dt0, t)
        if abs(v - round(v)) < 1e-9:
            continue                      # a tie at an integer: both sides exact only in exact arithmetic
        assert sync_interval(dt0, t) == math.ceil(v), (dt0, t)


@pytest.mark.parametrize("dt0", [1, 2, 5, 7, 20])
def test_interval_bounds_and_shape(dt0):
    vals = [sync_interval(dt0, t) for t in range(0, 10 * dt0 + 10)]
    assert all(1 <= v <= dt0 for v in vals)
    assert all(a <= b for a, b in zip(vals, vals[1:]))        # non-decreasing in t
    assert sync_interval(dt0, dt0) == math.ceil(dt0 / 2)         # tanh(0) = 0
    assert sync_interval(dt0, 50 * dt0) == dt0                   # tanh -> 1


def test_interval_table_dt0_5():
    # 5 / (1 + e^(4 - 4t/5)) for t = 0..12: 0.090 0.196 0.416 0.840 1.550 2.500
    # 3.450 4.160 4.584 4.804 4.910 4.959 4.982
    assert [sync_interval(5, t) for t in range(13)] == [1, 1, 1, 1, 2, 3, 4, 5, 5, 5, 5, 5, 5]
    # Algorithm 1 averages after unit t when t mod Delta T_t == 0
    assert [t for t in range(1, 31) if average_due(5, t)] == [1, 2, 3, 4, 10, 15, 20, 25, 30]
    # Delta T_0 = 1: every unit
    assert all(average_due(1, t) for t in range(1, 50))


def test_library_interval_equals_oracle():
    from paper_2510_12494_amd import vfl as V
    for dt0 in (1, 2, 3, 5, 9, 16, 64):
        for t in range(0, 8 * dt0 + 5):
            assert V.vfl_sync_interval(dt0, t) == sync_interval(dt0, t), (dt0, t)
    with pytest.raises(V.VflError):
        V.vfl_sync_interval(0, 1)
    with pytest.raises(V.VflError):
        V.vfl_sync_interval(5, -1)


# ----------------------------------------- Delta T = 1 == gradient averaging
CASES = [
    dict(),                                                           # s = 0
    dict(staleness=2),                                                # delayed B
    dict(staleness=1, clip=0.7, clip_emb=True, clip_grad=True, sigma=0.3,
         noise_emb=True, noise_grad=True),                            # private channel
    dict(A=PartySpec(dense=2, widths=[4], n_cat=2, vocab=7, emb_dim=3),
         B=PartySpec(dense=0, widths=[5, 3], n_cat=3, vocab=5, emb_dim=2), staleness=1),
]


@pytest.mark.parametrize("case", range(len(CASES)))
def test_interval_one_is_gradient_averaging(case):
    """Averaging after every tick, one local step each: the workers' common
    parameters are those of the k-replica oracle after every tick.  The last
    group of each epoch is ragged (115 = 3 * 30 + 25 rows: workers take
    10, 10 and 5 rows), so a wrong weighting of the average shows."""
    w = _mk(**CASES[case])
    d = S.generate(w)
    p = S.init_params(w)
    n_groups = 9
    ref = PubSubOracle(w, p)
    rr = ref.run(d, n_groups, lambda g: S.group_rows(w, g), snapshot=lambda t: True)
    sa = SemiAsyncOracle(w, p, w.replicas)
    rs = sa.run(d, n_groups, _worker_rows(w), unit=1, dt0=1, snapshot=lambda t: True)
    worst = 0.0
    for a, b in zip(rr, rs):
        if "loss" in a:
            assert abs(a["loss"] - b["loss"]) <= 1e-12 * max(1.0, abs(a["loss"]))
        for wk in b["params"]:
            for k, v in a["params"].items():
                worst = max(worst, _rel(wk[k], v))
    assert worst < 1e-12, worst


def test_workers_equal_after_an_average_and_apart_between():
    w = _mk(staleness=1)
    d = S.generate(w)
    p = S.init_params(w)
    sa = SemiAsyncOracle(w, p, w.replicas)
    recs = sa.run(d, 14, _worker_rows(w), unit=1, dt0=5, snapshot=lambda t: True)
    # units 2-4 average (ticks 1-3; at tick 0 no group was consumed yet),
    # then units 10 and 15 (ticks 9 and 14)
    assert sa.averages == [1, 2, 3, 9, 14]
    for rec in recs:
        ps = rec["params"]
        spread = max(_rel(ps[r][k], ps[0][k]) for r in range(1, len(ps)) for k in ps[0])
        if rec["averaged"]:
            assert spread == 0.0, rec["tick"]
        elif rec["tick"] in (5, 6, 7, 8, 10, 11):
            assert spread > 1e-6, rec["tick"]


def test_no_average_workers_train_alone():
    """With the first average far away every worker is a one-replica run
    over its own rows only (local SGD with its own 1/n_r scaling)."""
    w = _mk(staleness=1)
    d = S.generate(w)
    p = S.init_params(w)
    sa = SemiAsyncOracle(w, p, w.replicas)
    sa.run(d, 6, _worker_rows(w), unit=100, dt0=5)
    assert sa.averages == []
    wr = w.replace(replicas=1)
    for r in range(w.replicas):
        o = PubSubOracle(wr, p)
        o.run(d, 6, lambda g, r=r: [_worker_rows(w)(r, g)])
        for k in o.p:
            assert np.array_equal(o.p[k], sa.workers[r].p[k]), (r, k)


# ----------------------------------------------------- planted mistakes
_AVERAGE = SemiAsyncOracle.average


def _equal_weights(self, party):
    for r in range(self.k):
        self.rows[r][party] = 1                     # every worker weighted alike
    _AVERAGE(self, party)


def _a_only(self, party):
    if party == "A":
        _AVERAGE(self, party)
    else:
        for r in range(self.k):
            self.rows[r][party] = 0


@pytest.mark.parametrize("mutant", [_equal_weights, _a_only])
def test_planted_mistakes_fail_the_gradient_averaging_pin(mutant, monkeypatch):
    """A mistake in the average (its weights, or a party left out) breaks
    the Delta T = 1 pin on ragged groups."""
    monkeypatch.setattr(SemiAsyncOracle, "average", mutant)
    with pytest.raises(AssertionError):
        test_interval_one_is_gradient_averaging(1)
