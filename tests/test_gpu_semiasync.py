"""GPU parity of the semi-asynchronous workers (vfl_replica_average and
vfl_sync_interval; Section 4.1 "Intra-party Semi-asynchronous Mechanism",
Eq. 5, Algorithm 1's aggregation step) against oracle/semiasync.py.

Each worker is a one-replica context over its rows of every batch group
(worker r of group g: replica r of the k-replica split); after every unit
of ticks the test averages both parties when Algorithm 1's test holds for
the library's vfl_sync_interval.  Tolerances are the parity bounds of the
other GPU tests (tests/gpu_harness.py): float32 workloads 1e-4 relative per
parameter tensor; bf16 against the bf16 emulation (theta 1e-3, its change
1e-2 plus float32 ulps) and theta against float64 within 2e-2."""
import numpy as np
import pytest

import vfl_synth as S
from vfl_synth.workloads import PartySpec, TopSpec
import gpu_harness as H
from oracle.semiasync import SemiAsyncOracle

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("needs an MI355X")


def _f32_workload(**kw):
    """f32, k = 3 workers of 100 rows, s = 2, clipped and noised channels;
    1150 rows = 3 epochs' worth of groups plus a ragged 250-row group (the
    workers take 100, 100 and 50 rows of it)."""
    w = S.get("tiny_sync").replace(
        name="semiasync_f32", n_rows=1150, batch=100, replicas=3, staleness=2, lr=0.1,
        clip=1.5, clip_emb=True, clip_grad=True, sigma=0.2, noise_emb=True, noise_grad=True,
        A=PartySpec(dense=16, widths=[48, 24]), B=PartySpec(dense=24, widths=[40, 16]),
        top=TopSpec(widths=[24, 1]))
    return w.replace(**kw)


class Workers:
    """k one-replica sessions over the worker rows of a k-replica workload."""

    def __init__(self, w, data, params, rows=None):
        from paper_2510_12494_amd.session import Session
        self.w, self.k = w, w.replicas
        n = data["y"].shape[0]
        self.rows = rows or (lambda r, g: S.group_rows(w, g, n)[r])
        wr = w.replace(replicas=1)
        self.sess = [Session(wr, data, params, lambda g, r=r: [self.rows(r, g)]) for r in range(self.k)]
        self.shapes = {key: v.shape for key, v in params.items()}
        self.averaged = []

    def run(self, n_groups, unit, dt0, snap=()):
        from paper_2510_12494_amd import vfl as V
        s = self.w.staleness
        snaps = {}
        for t in range(n_groups + s):
            for ss in self.sess:
                ss.step(t, n_groups)
            if (t + 1) % unit == 0 and t >= s:
                tu = (t + 1) // unit
                if tu % V.vfl_sync_interval(dt0, tu) == 0:
                    V.vfl_replica_average([ss.ctx for ss in self.sess],
                                          (1 << V.VFL_PARTY_A) | (1 << V.VFL_PARTY_B))
                    self.averaged.append(t)
            if t in snap:
                snaps[t] = [ss.params(self.shapes) for ss in self.sess]
        self.final = [ss.params(self.shapes) for ss in self.sess]
        # row-weighted mean loss of each group over the workers
        L = np.array([ss.losses(range(n_groups)) for ss in self.sess])
        cnt = np.array([[self.rows(r, g)[1] for g in range(n_groups)] for r in range(self.k)], float)
        self.losses = (L * cnt).sum(0) / cnt.sum(0)
        return snaps

    def close(self):
        for ss in self.sess:
            ss.close()


def _check_f32(gpu_params, ora_params, where):
    worst = 0.0
    for r, (g, o) in enumerate(zip(gpu_params, ora_params)):
        for key, v in o.items():
            e = H.rel_inf(g[key], v)
            worst = max(worst, e)
            assert e <= H.F32_TOL, (where, r, key, e)
    H.record("theta rel", worst, H.F32_TOL, where)


@pytest.mark.parametrize("unit,dt0", [(1, 5), (2, 3)])
def test_f32_workers_match_oracle(unit, dt0):
    w = _f32_workload()
    d = S.generate(w)
    p = S.init_params(w)
    n_groups = 14
    snap = {5, 9, 12}
    gw = Workers(w, d, p)
    try:
        gsnaps = gw.run(n_groups, unit, dt0, snap)
    finally:
        gw.close()
    o = SemiAsyncOracle(w, p, w.replicas)
    recs = o.run(d, n_groups, gw.rows, unit, dt0, snapshot=lambda t: t in snap)
    assert gw.averaged == o.averages
    for t in sorted(snap):
        _check_f32(gsnaps[t], recs[t]["params"], f"tick {t}")
    _check_f32(gw.final, [wk.p for wk in o.workers], "final")
    ol = np.array([r["loss"] for r in recs if "loss" in r])
    e = np.max(np.abs(gw.losses - ol) / np.abs(ol))
    H.record("loss rel", e, H.F32_TOL)
    assert e <= H.F32_TOL


def test_interval_one_equals_replica_context():
    """Averaging after every tick equals one k-replica context (gradient
    averaging) up to float32 rounding."""
    w = _f32_workload()
    d = S.generate(w)
    p = S.init_params(w)
    n_groups = 10
    gw = Workers(w, d, p)
    try:
        gw.run(n_groups, 1, 1)
    finally:
        gw.close()
    run = H.Run(w, w.n_rows, n_groups, data=d, params=p, snap=lambda t: False, messages=False)
    worst = 0.0
    for g in gw.final:
        for key, v in run.final.items():
            worst = max(worst, H.rel_inf(g[key], v))
    H.record("theta rel vs k-replica context", worst, H.F32_TOL)
    assert worst <= H.F32_TOL


def test_bf16_hetero_workers_match_oracle():
    """hetero's shapes (B 500 -> 1024 -> 512 -> 128, k = 4, s = 4) at 128 rows
    per worker, Delta T_0 = 5 per tick, against the bf16 emulation and the
    float64 oracle."""
    w = S.get("hetero").replace(batch=128)
    n_groups = 12
    n = n_groups * w.rows_per_tick - 100          # a ragged last group
    d = S.generate(w, n)
    p = S.init_params(w)
    gw = Workers(w, d, p)
    try:
        gw.run(n_groups, 1, 5)
    finally:
        gw.close()
    emu = SemiAsyncOracle(w, p, w.replicas, precision="bf16")
    emu.run(d, n_groups, gw.rows, 1, 5)
    assert gw.averaged == emu.averages
    f64 = SemiAsyncOracle(w, p, w.replicas)
    f64.run(d, n_groups, gw.rows, 1, 5)
    # float32 roundings of a stored parameter: one per SGD update, and per
    # average k fused multiply-adds of float32-rounded weights (k + 1 ulps)
    n_upd = n_groups + (w.replicas + 1) * len(gw.averaged)
    worst = {"theta": 0.0, "dtheta": 0.0, "f64": 0.0}
    for r in range(w.replicas):
        for key, v in emu.workers[r].p.items():
            g = gw.final[r][key]
            worst["theta"] = max(worst["theta"], H.rel_inf(g, v))
            ok, e, bnd = H.delta_ok(g, v, p[key].astype(np.float64), H.BF16_DELTA_TOL, n_upd)
            worst["dtheta"] = max(worst["dtheta"], e / bnd if bnd > 0 else 0.0)
            assert ok, (r, key, e, bnd)
            worst["f64"] = max(worst["f64"], H.rel_inf(g, f64.workers[r].p[key]))
    H.record("theta rel", worst["theta"], H.BF16_THETA_EMU)
    H.record("dtheta err/bound", worst["dtheta"], 1.0)
    H.record("theta rel vs f64", worst["f64"], H.BF16_TOL)
    assert worst["theta"] <= H.BF16_THETA_EMU
    assert worst["f64"] <= H.BF16_TOL


def test_graph_replay_between_averages():
    """Workers bound to their own row shards run vfl_run for a unit of ticks
    between averages: bitwise the per-call run of the same shards."""
    from paper_2510_12494_amd import vfl as V
    w = _f32_workload(noise_emb=False, noise_grad=False)
    k, s = w.replicas, w.staleness
    n_groups, unit, dt0 = 3 * (s + 1) + 2 * 7, 7, 2
    n_full = n_groups * w.rows_per_tick
    full = S.generate(w, n_full)
    p = S.init_params(w)
    rows = lambda r, g: S.group_rows(w, g, n_full)[r]
    # worker r's shard: its rows of every group, in group order
    idx = [np.concatenate([np.arange(a, a + c) for a, c in (rows(r, g) for g in range(n_groups))])
           for r in range(k)]
    shard = lambda r: {key: (None if v is None else np.ascontiguousarray(v[idx[r]])) for key, v in full.items()}
    wr = w.replace(replicas=1)
    from paper_2510_12494_amd.session import Session
    shapes = {key: v.shape for key, v in p.items()}
    finals = []
    for graph in (False, True):
        sess = [Session(wr, shard(r), p, lambda g, r=r: S.group_rows(wr, g, len(idx[r])))
                for r in range(k)]
        try:
            t = 0
            t0 = s + 1
            for t in range(t0):
                for ss in sess:
                    ss.step(t)
            if graph:
                for ss in sess:
                    ss.bind()
            t = t0
            end = n_groups                 # ticks t0 .. end-1, averaging after every unit
            while t < end:
                stop = min(end, (t // unit + 1) * unit)
                for ss in sess:
                    if graph:
                        ss.run(t, stop - t)
                    else:
                        for tt in range(t, stop):
                            ss.step(tt)
                t = stop
                if t % unit == 0 and (t // unit) % V.vfl_sync_interval(dt0, t // unit) == 0:
                    V.vfl_replica_average([ss.ctx for ss in sess], 3)
            finals.append([ss.params(shapes) for ss in sess])
        finally:
            for ss in sess:
                ss.close()
    for r in range(k):
        for key in shapes:
            assert np.array_equal(finals[0][r][key], finals[1][r][key]), (r, key)


def test_average_refusals():
    from paper_2510_12494_amd import vfl as V
    w = _f32_workload()
    d = S.generate(w)
    p = S.init_params(w)
    gw = Workers(w, d, p)
    other = Workers(w.replace(batch=50, replicas=1), d, p)
    try:
        ctxs = [ss.ctx for ss in gw.sess]
        with pytest.raises(V.VflError) as e:          # nothing applied yet
            V.vfl_replica_average(ctxs, 3)
        assert e.value.status == V.VFL_E_STATE
        with pytest.raises(V.VflError) as e:
            V.vfl_replica_average([ctxs[0], ctxs[0]], 3)
        assert e.value.status == V.VFL_E_INVALID
        with pytest.raises(V.VflError) as e:
            V.vfl_replica_average([ctxs[0], other.sess[0].ctx], 3)
        assert e.value.status == V.VFL_E_INVALID
        with pytest.raises(V.VflError) as e:
            V.vfl_replica_average(ctxs, 4)
        assert e.value.status == V.VFL_E_INVALID
        for t in range(w.staleness + 1):
            for ss in gw.sess:
                ss.step(t)
        # A of one worker inside a group's step
        ss = gw.sess[0]
        V.vfl_bottom_forward(ss.ctx, V.VFL_PARTY_B, w.staleness + 1, ss.batches("B", w.staleness + 1))
        V.vfl_publish(ss.ctx, w.staleness + 1)
        V.vfl_bottom_forward(ss.ctx, V.VFL_PARTY_A, 1, ss.batches("A", 1))
        with pytest.raises(V.VflError) as e:
            V.vfl_replica_average(ctxs, 1 << V.VFL_PARTY_A)
        assert e.value.status == V.VFL_E_STATE
        V.vfl_replica_average(ctxs, 1 << V.VFL_PARTY_B)   # B alone is fine there
    finally:
        gw.close()
        other.close()
