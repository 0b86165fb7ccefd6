"""Semi-asynchronous workers inside each party (Section 4.1 "Intra-party
Semi-asynchronous Mechanism", Eq. 5; the aggregation step of Algorithm 1).

Test infrastructure only (see ``oracle/__init__.py``).

Each party runs k workers.  Worker r keeps its own copy of its party's
parameters, runs the publisher/subscriber loop on its own rows of every
batch group and updates its copy with SGD on the mean gradient of those rows
alone (local SGD).  Worker r of B and worker r of A form a pair: B's worker
publishes the embedding of its rows, A's worker consumes it and returns the
gradient.  Ticks, slots, staleness and the delayed backward of each pair are
those of ``PubSubOracle`` (one replica).  After every unit t = 1, 2, ... the
parameter server of a party replaces all its workers' parameters by their
average (and so broadcasts it) when t is a multiple of the interval Delta T_t
of Eq. 5.

Readings of what the paper leaves open:
  * t counts epochs in Algorithm 1; here a unit is a fixed number of ticks
    (the ticks of an epoch for the paper's setting, 1 for a per-tick
    variant) and the test is Algorithm 1's "t mod Delta T_t == 0" on units
    counted from 1;
  * Eq. 5 grows from 1 towards Delta T_0 with t, while one sentence of the
    section says the interval shrinks as training proceeds; the equation is
    followed;
  * the average weights each worker by the rows it applied since the
    previous average (equal weights when the workers see as many rows), so
    that Delta T = 1 with one local step per unit is exactly the
    row-weighted gradient averaging of ``PubSubOracle`` with k replicas;
  * Algorithm 1 shows the aggregation for the active party's parameters,
    the section describes the mechanism for each party: both parties are
    averaged (A: its bottom model and the top model; B: its bottom model).
"""
from __future__ import annotations

import math

import numpy as np

from .pubsub import PubSubOracle


def sync_interval(dt0: int, t: int) -> int:
    """Delta T_t of Eq. 5 for unit t and initial interval dt0."""
    return math.ceil(dt0 / 2.0 * math.tanh(2.0 * t / dt0 - 2.0) + dt0 / 2.0)


def average_due(dt0: int, t: int) -> bool:
    """Algorithm 1's aggregation test after unit t (t >= 1)."""
    return t % sync_interval(dt0, t) == 0


PARTY_KEYS = {"A": ("A", "top"), "B": ("B",)}


class SemiAsyncOracle:
    """k workers per party, each a one-replica ``PubSubOracle`` over its own
    rows, averaged per party on the schedule of Eq. 5."""

    def __init__(self, w, params: dict, k: int, precision: str = "f64", points=None):
        self.w = w
        self.k = int(k)
        wr = w.replace(replicas=1)
        self.workers = [PubSubOracle(wr, params, precision, points) for _ in range(self.k)]
        self.rows = [{"A": 0, "B": 0} for _ in range(self.k)]
        self.averages = []                  # ticks after which the parties were averaged

    def average(self, party: str):
        """Row-weighted average of the party's parameters over the workers,
        written to every worker (stored as each worker stores its masters)."""
        n = np.array([self.rows[r][party] for r in range(self.k)], dtype=np.float64)
        assert n.sum() > 0, "no rows applied since the last average"
        wts = n / n.sum()
        w0 = self.workers[0]
        for key in w0.p:
            if key.split(".")[0] not in PARTY_KEYS[party]:
                continue
            m = sum(wts[r] * self.workers[r].p[key] for r in range(self.k))
            m = w0.rnd_master(m)
            for o in self.workers:
                o.p[key] = m.copy()
        for r in range(self.k):
            self.rows[r][party] = 0

    def run(self, data: dict, n_groups: int, worker_rows, unit: int, dt0: int,
            snapshot=None):
        """n_groups batch groups (n_groups + s ticks).  worker_rows(r, g) ->
        (start, count >= 1): worker r's rows of group g.  After tick tau,
        when (tau + 1) is a multiple of ``unit``, unit t = (tau + 1) / unit
        ends and both parties are averaged if t mod Delta T_t == 0.  Returns
        per-tick records: {"tick", "loss" (row-weighted mean over the
        workers, when a group was consumed), "averaged", "params" (per
        worker, when snapshot(tau))}."""
        s = self.workers[0].s
        recs = []
        for tau in range(n_groups + s):
            rec = {"tick": tau, "averaged": False}
            loss = rows = 0.0
            u = tau - s
            for r, o in enumerate(self.workers):
                part = o.tick(tau, data, n_groups, lambda g, r=r: [worker_rows(r, g)],
                              keep_messages=False)
                if 0 <= u < n_groups:
                    cnt = worker_rows(r, u)[1]
                    self.rows[r]["A"] += cnt
                    self.rows[r]["B"] += cnt
                    loss += part["loss"] * cnt
                    rows += cnt
            if rows:
                rec["loss"] = loss / rows
            if (tau + 1) % unit == 0 and average_due(dt0, (tau + 1) // unit):
                # a party that applied no rows since its last average (the
                # first s ticks) has nothing to average
                for party in ("A", "B"):
                    if any(self.rows[r][party] for r in range(self.k)):
                        self.average(party)
                        rec["averaged"] = True
                if rec["averaged"]:
                    self.averages.append(tau)
            if snapshot is not None and snapshot(tau):
                rec["params"] = [{key: v.copy() for key, v in o.p.items()} for o in self.workers]
            recs.append(rec)
        return recs
