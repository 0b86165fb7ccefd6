"""System profiling and planning on one GPU (Section 4.2 "System Profiling",
Eqs. 7-9; Section 4.3 "System Planning Phase", Eq. 14 and Algorithm 2).

The paper models each party's forward and backward delay as a power law of
the batch size B whose constants it fits from measured delays (the
Appendix's Table 7), and picks the configuration that minimises
max(T_A, T_P) + T_comm subject to a memory bound.  This module does that
for a workload on this GPU:

1. ``sweep`` runs the workload's tick at several replica batch sizes B (the
   workload's replica count k kept) and times each party's phases with HIP
   events on the party's stream, one stream for both parties so that no
   phase includes the other's work:
     T_f^(p)  party B's forward and publish      (vfl_bottom_forward + vfl_publish)
     T_f^(a) + T_top^(a)  party A's forward fused with the top model's
                          forward and backward  (vfl_top_step)
     T_b^(a)  party A's and the top model's weight gradients and SGD
     T_b^(p)  party B's delayed backward and SGD
   Each is turned into the delay of one pass over the workload's rows
   (per-tick time times ticks per epoch), the quantity whose fitted
   exponents are negative in Table 7.
2. ``fit`` fits every delay with vfl_fit_delay (least squares in log space)
   and the memory model M(B) = M0 + rho B (chi = 1) from vfl_workspace_size.
3. ``plan`` runs vfl_plan (Algorithm 2) over the candidate batch sizes with
   the fitted profiles; the chosen B (with the workload's k) is the run's
   configuration.  On one GPU the parties' messages are buffers in device
   memory read by the next kernel, so the exchange term is zero, and the
   fused top model's delay is part of A's forward term (lambda'_a = 0).

Run ``python -m paper_2510_12494_amd.planning --workload hetero`` on a GPU;
it prints one JSON object.  Host-side orchestration only: every step of the
training path runs in the library's kernels.
"""
from __future__ import annotations

import argparse
import json
import os
import sys

PHASES = ("b_fwd", "a_top", "a_bwd", "b_bwd")


def _sizes(w, batch):
    from .session import bottom_spec, top_spec, opts
    from . import vfl as V
    ww = w.replace(batch=int(batch))
    return V.vfl_workspace_size(bottom_spec(ww.A), bottom_spec(ww.B), top_spec(ww.top), opts(ww))


def sweep(w, batches, ticks: int = 12) -> dict:
    """Per-tick GPU time of each phase at each replica batch size (seconds,
    mean over ``ticks`` ticks after 2(s+1) warm-up ticks)."""
    import torch
    import vfl_synth as S
    from . import vfl as V
    from .session import Session
    out = {}
    s = w.staleness
    for B in batches:
        ww = w.replace(batch=int(B))
        R = ww.rows_per_tick
        n_rows = 2 * R
        data = S.generate(ww, n_rows)
        params = S.init_params(ww)
        rows_of = lambda g, ww=ww, n=n_rows: S.group_rows(ww, g, n)
        sess = Session(ww, data, params, rows_of, one_stream=True)
        try:
            st = sess.sa
            ev = {}
            acc = {k: 0.0 for k in PHASES}
            warm = 2 * (s + 1)
            for t in range(warm + ticks):
                timed = t >= warm
                g, u = t % 2, (t - s) % 2
                e = [torch.cuda.Event(enable_timing=True) for _ in range(5)]
                e[0].record(st)
                V.vfl_bottom_forward(sess.ctx, V.VFL_PARTY_B, t, sess.batches("B", g))
                V.vfl_publish(sess.ctx, t)
                e[1].record(st)
                if t >= s:
                    V.vfl_bottom_forward(sess.ctx, V.VFL_PARTY_A, t - s, sess.batches("A", u))
                    V.vfl_top_step(sess.ctx, t - s, sess.loss.data_ptr())
                    e[2].record(st)
                    V.vfl_bottom_backward(sess.ctx, V.VFL_PARTY_A, t - s)
                    e[3].record(st)
                    V.vfl_bottom_backward(sess.ctx, V.VFL_PARTY_B, t - s)
                    e[4].record(st)
                if timed:
                    ev[t] = e
            torch.cuda.synchronize()
            for e in ev.values():
                acc["b_fwd"] += e[0].elapsed_time(e[1])
                acc["a_top"] += e[1].elapsed_time(e[2])
                acc["a_bwd"] += e[2].elapsed_time(e[3])
                acc["b_bwd"] += e[3].elapsed_time(e[4])
            out[int(B)] = {k: v / 1e3 / ticks for k, v in acc.items()}
        finally:
            sess.close()
    return out


def fit(w, per_tick: dict) -> dict:
    """Per-pass delays (per-tick time x ticks per epoch of the workload's
    rows) fitted to coef * B**exp per phase, and the memory model."""
    from . import vfl as V
    Bs = sorted(per_tick)
    consts = {}
    for ph in PHASES:
        T = [per_tick[B][ph] * -(-w.n_rows // (w.replicas * B)) for B in Bs]
        consts[ph] = V.vfl_fit_delay([float(b) for b in Bs], T)
    m_lo, m_hi = _sizes(w, Bs[0]), _sizes(w, Bs[-1])
    rho = (m_hi - m_lo) / float(Bs[-1] - Bs[0])
    return {"delay": consts, "mem_base": m_lo - rho * Bs[0], "mem_coef": rho}


def plan(w, fitted: dict, batches, mem_cap: float):
    """Algorithm 2 over the candidate batch sizes with the fitted profiles;
    both parties share the GPU's one workspace (counted on party A)."""
    from . import vfl as V
    d = fitted["delay"]
    a = V.vfl_plan_party()
    a.lambda_, a.gamma = d["a_top"]
    a.phi, a.beta = d["a_bwd"]
    a.cores, a.w_min, a.w_max = 1.0, 1, 1
    a.mem_base, a.mem_coef, a.mem_cap = fitted["mem_base"], fitted["mem_coef"], mem_cap
    p = V.vfl_plan_party()
    p.lambda_, p.gamma = d["b_fwd"]
    p.phi, p.beta = d["b_bwd"]
    p.cores, p.w_min, p.w_max = 1.0, 1, 1
    link = V.vfl_plan_link()
    link.emb_bytes_per_row = link.grad_bytes_per_row = 0.0
    link.bandwidth, link.chi = 1.0, 1.0
    return V.vfl_plan(a, p, link, [int(b) for b in batches])


def main():
    ap = argparse.ArgumentParser(description="fit the delay model on this GPU and plan the batch size")
    ap.add_argument("--workload", default="hetero")
    ap.add_argument("--batches", default="1024,2048,4096,8192,16384")
    ap.add_argument("--ticks", type=int, default=12)
    ap.add_argument("--mem-cap-gb", type=float, default=200.0,
                    help="device memory the workspace may take (the rest holds the dataset)")
    args = ap.parse_args()
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    if root not in sys.path:
        sys.path.insert(0, root)
    import vfl_synth as S
    w = S.get(args.workload)
    batches = [int(b) for b in args.batches.split(",")]
    per_tick = sweep(w, batches, args.ticks)
    fitted = fit(w, per_tick)
    (wa, wp, B), cost = plan(w, fitted, batches, args.mem_cap_gb * 1e9)
    pred = {ph: c * B ** e for ph, (c, e) in fitted["delay"].items()}
    meas = {ph: per_tick[B][ph] * -(-w.n_rows // (w.replicas * B)) for ph in PHASES}
    print(json.dumps({
        "workload": w.name, "replicas": w.replicas, "batches": batches,
        "per_tick_s": {str(b): v for b, v in per_tick.items()},
        "fitted": {ph: {"coef": c, "exp": e} for ph, (c, e) in fitted["delay"].items()},
        "memory": {"base": fitted["mem_base"], "per_row": fitted["mem_coef"], "cap": args.mem_cap_gb * 1e9},
        "plan": {"w_a": wa, "w_p": wp, "batch": B, "replicas": w.replicas, "cost_s_per_pass": cost},
        "at_plan_per_pass_s": {"predicted": pred, "measured": meas},
    }), flush=True)


if __name__ == "__main__":
    main()
