"""Throughput of the two-party publisher/subscriber split-learning step on one
MI355X.

One step = one tick of the deterministic schedule: party B's bottom forward
and publish of group t, party A's bottom forward, top model, BCE, backward
and SGD of group t - s, and B's delayed backward + SGD of that group (both
parties' forward, backward and update).  Inputs are seeded synthetic data of
the workload's shape, resident in HBM before timing starts.

Prints one JSON line: samples/s (rows per tick / tick time), the MFMA
utilisation of the algorithmic matrix-product FLOPs, the roofline of the
dominant kernel class (the class with the most kernel time per tick in a
short run with both parties on one stream; its algorithmic FLOPs or bytes
per launch over its average duration, timed with HIP events on its own
stream during the timed region) and the oracle's CPU throughput on a
bounded sample.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK = {"bf16": 2.5e15, "f32": 157.3e12}     # dense MFMA FLOP/s (MI355X spec)
HBM_PEAK = 8.0e12                            # bytes/s
METRIC = "training samples/sec (both parties fwd+bwd+update) on 1 MI355X; MFMA util %"
GEMM_CLASSES = ("fwd", "active", "bwd", "dw", "gemm", "dwt")


def gemm_flops_per_tick(w) -> float:
    """Algorithmic matrix-product FLOPs of one tick (no padding): every layer's
    forward and weight gradient, and the input gradient of every layer but
    the first layer of a bottom model without embedding tables; the logit
    layer counted as a product of width 1."""
    R = w.rows_per_tick
    f = 0.0
    for spec in (w.A, w.B):
        for l, (fi, fo) in enumerate(spec.layer_dims()):
            f += 2 * 2.0 * R * fi * fo
            if l > 0:
                f += 2.0 * R * fi * fo
            elif spec.n_cat:
                f += 2.0 * R * (spec.n_cat * spec.emb_dim) * fo
    fi = w.top_in
    for fo in w.top.widths:
        f += 3 * 2.0 * R * fi * fo
        fi = fo
    return f


CSRC = "paper_2510_12494_amd/csrc"
# kernel class -> (kernel symbols, the sources its code and launch layout come from)
KERNEL_SOURCES = {
    "fwd": (("k_fwd<",), ["chain.hip"]), "active": (("k_active<",), ["chain.hip"]),
    "bwd": (("k_bwd<",), ["chain.hip"]), "dw": (("k_dw<", "k_dw32<"), ["dw.hip"]),
    "dwt": (("k_dwt(",), ["dw.hip"]),
    "reduce": (("k_dw_reduce<",), ["dw.hip"]), "cast": (("k_cast<",), ["rowops.hip"]),
    "avg": (("k_avg(",), ["rowops.hip"]),
    "emb_sgd": (("k_embed_sgd",), ["embed.hip"]), "gemm": (("k_lin(",), ["lin.hip"]),
}


def source_sha(kernel: str) -> str:
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[kernel][1] + ["kernels.h", "device.h", "api.cpp"]:
        with open(os.path.join(ROOT, CSRC, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def traffic_for(kernel: str, workload: str):
    """HBM traffic per launch from the committed rocprofv3 counter summary
    of this kernel class on this workload, or None when there is none or the
    kernel's sources changed since."""
    p = os.path.join(ROOT, "profiles", f"traffic_{kernel}.json")
    if not os.path.exists(p):
        return None
    with open(p) as fh:
        t = json.load(fh)
    if t.get("source_sha") != source_sha(kernel) or t.get("workload") != workload:
        return None
    return t.get("bytes_per_launch")


def _counter_rows(d: str, counter: str):
    import csv
    import glob
    files = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise SystemExit(f"no counter_collection.csv under {d}")
    out = []
    for f in files:
        with open(f) as fh:
            for r in csv.DictReader(fh):
                if r["Counter_Name"] == counter:
                    out.append((r["Kernel_Name"], float(r["Counter_Value"])))
    return out


def traffic_summary(fetch_dir: str, write_dir: str, kernel: str, copy_bytes: int, workload: str) -> dict:
    """HBM bytes per launch of one kernel class from two rocprofv3 --pmc
    runs of this script with --copy-bytes (FETCH_SIZE, then WRITE_SIZE, KiB
    per dispatch), each counter scaled so that the plain copy of known size
    in the same run reads exactly its bytes."""
    syms = KERNEL_SOURCES[kernel][0]
    res = {"kernel": kernel, "workload": workload, "copy_bytes": copy_bytes}
    for name, d in (("FETCH_SIZE", fetch_dir), ("WRITE_SIZE", write_dir)):
        rows = _counter_rows(d, name)
        copy = [v for k, v in rows if "copy" in k.lower()]
        if not copy:
            raise SystemExit(f"{name}: no copy dispatch in {d}")
        cal = copy_bytes / (max(copy) * 1024.0)
        ks = [v for k, v in rows if any(sym in k for sym in syms)]
        if not ks:
            raise SystemExit(f"{name}: no {'/'.join(syms)} dispatch in {d}")
        res[name] = {"dispatches": len(ks), "kib_per_dispatch": sum(ks) / len(ks),
                     "copy_kib": max(copy), "scale": cal,
                     "bytes_per_launch": cal * 1024.0 * sum(ks) / len(ks)}
    res["bytes_per_launch"] = res["FETCH_SIZE"]["bytes_per_launch"] + res["WRITE_SIZE"]["bytes_per_launch"]
    res["source_sha"] = source_sha(kernel)
    return res


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(w, data, params, seconds: float) -> dict:
    """The oracle (float64 numpy) on this host over the same resident dataset,
    for about ``seconds`` of CPU work: a probe run sizes the sample, and a
    sample that ends well short of ``seconds`` is run again, longer."""
    import vfl_synth as S
    from oracle import PubSubOracle
    affinity = len(os.sched_getaffinity(0))
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = affinity
    R = w.rows_per_tick
    rows_of = lambda g: S.group_rows(w, g)
    # size the sample from a 1-group run after a 1-group warm-up; a run
    # under half of the target is repeated with the groups scaled to it
    PubSubOracle(w, params, "f64").run(data, 1, rows_of, keep_messages=False)
    groups, dt = 1, 0.0
    for _ in range(4):
        o = PubSubOracle(w, params, "f64")
        t0 = time.perf_counter()
        o.run(data, groups, rows_of, keep_messages=False)
        dt = time.perf_counter() - t0
        if dt >= 0.5 * seconds or groups >= 8192:
            break
        groups = int(max(groups + 1, min(8192, groups * seconds / max(dt, 1e-6))))
    return {"value": groups * R / dt, "unit": "samples/s", "cores": int(threads), "kind": "oracle",
            "sample": f"first {groups} batch groups of {R} rows of the same dataset "
                      f"({groups + w.staleness} ticks incl. the s={w.staleness} lead-in), "
                      f"float64 numpy, {dt:.1f} s",
            "affinity_cores": affinity, "blas_threads": int(threads), "cpu_model": cpu_model()}


def serial_probe(w, data, params, epoch, ticks: int = 24) -> dict:
    """Kernel time per tick of every class with both parties on one stream
    (no overlap, so each class's time is its own): picks the dominant class."""
    import torch
    import vfl_synth as S
    from paper_2510_12494_amd import vfl as V
    from paper_2510_12494_amd.session import Session
    sess = Session(w, data, params, lambda g: S.group_rows(w, g), one_stream=True)
    try:
        t = 0
        for _ in range(2 * (w.staleness + 1)):
            sess.step(t, epoch=epoch)
            t += 1
        torch.cuda.synchronize()
        V.vfl_timing_enable(sess.ctx, (1 << len(V.KERNEL_CLASSES)) - 1)
        for _ in range(ticks):
            sess.step(t, epoch=epoch)
            t += 1
        out = {}
        for i, name in enumerate(V.KERNEL_CLASSES):
            ms, n, wk = V.vfl_timing_read(sess.ctx, i)
            out[name] = (ms / ticks, n / ticks, wk / ticks)
        V.vfl_timing_enable(sess.ctx, 0)
    finally:
        sess.close()
    return out


def semi_async(args, w, data, params) -> dict:
    """The workload as k semi-asynchronous workers (one context each, over a
    contiguous 1/k of the rows; Section 4.1, Eq. 5): every worker runs `unit`
    ticks by graph replay, then both parties are averaged when Algorithm 1's
    test holds for unit t.  Returns the JSON line's fields."""
    import torch
    import vfl_synth as S
    from paper_2510_12494_amd import vfl as V
    from paper_2510_12494_amd.session import Session
    k, s, U = w.replicas, w.staleness, args.unit
    wr = w.replace(replicas=1)
    n = data["y"].shape[0] // k
    shards = [{key: (None if v is None else v[r * n:(r + 1) * n]) for key, v in data.items()}
              for r in range(k)]
    sess = [Session(wr, shards[r], params, lambda g: S.group_rows(wr, g, n)) for r in range(k)]
    both = (1 << V.VFL_PARTY_A) | (1 << V.VFL_PARTY_B)
    n_avg = [0]

    def advance(t, stop, graph):
        # ticks t .. stop-1, averaging after every unit that Eq. 5 selects
        while t < stop:
            end = min(stop, (t // U + 1) * U)
            for ss in sess:
                if graph:
                    ss.run(t, end - t)
                else:
                    for tt in range(t, end):
                        ss.step(tt)
            t = end
            if t % U == 0 and t > s and (t // U) % V.vfl_sync_interval(args.dt0, t // U) == 0:
                V.vfl_replica_average([ss.ctx for ss in sess], both)
                n_avg[0] += 1
        return t

    try:
        warm = max(args.warmup, 2 * (s + 1))
        t = advance(0, warm, False)
        for ss in sess:
            ss.bind()
        avg_i = V.KERNEL_CLASSES.index("avg")
        V.vfl_timing_enable(sess[0].ctx, 1 << avg_i)
        t = advance(t, t + args.steps, True)          # captures the replayed graphs
        V.vfl_timing_read(sess[0].ctx, avg_i)
        torch.cuda.synchronize()
        n_avg[0] = 0
        t0 = time.perf_counter()
        t = advance(t, t + args.steps, True)
        torch.cuda.synchronize()
        dt = time.perf_counter() - t0
        ms, launches, work = V.vfl_timing_read(sess[0].ctx, avg_i)
        V.vfl_timing_enable(sess[0].ctx, 0)
    finally:
        for ss in sess:
            ss.close()
    avg_s = ms / 1e3 / max(launches, 1)
    per_launch = work / max(launches, 1)
    achieved = per_launch / avg_s if avg_s > 0 else 0.0
    return {
        "value": args.steps * w.rows_per_tick / dt, "ms_per_step": dt / args.steps * 1e3,
        "warmup": warm,
        "semi_async": {"workers": k, "rows_per_worker_tick": w.batch, "dt0": args.dt0,
                       "unit_ticks": U, "averages_in_timed_region": n_avg[0]},
        "roofline": {"bound": "hbm", "achieved": achieved / 1e9, "peak": HBM_PEAK / 1e9,
                     "unit": "GB/s", "frac": achieved / HBM_PEAK, "traffic": None,
                     "kernel": "avg", "launches": launches, "avg_us": avg_s * 1e6,
                     "work_per_launch": per_launch},
    }


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=2400)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--workload", default="hetero")
    ap.add_argument("--id-stride", type=int, default=1,
                    help="categorical ids k * stride mod vocab (a stride coprime with the vocabulary "
                         "scatters the frequent ids, as hashed ids would)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-bytes", type=int, default=0,
                    help="first run one plain device copy of this many bytes "
                         "(the calibration dispatch of a counter run)")
    ap.add_argument("--traffic-summary", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="no GPU: summarise two rocprofv3 --pmc runs (FETCH_SIZE, "
                         "WRITE_SIZE) into profiles/traffic_<kernel>.json")
    ap.add_argument("--kernel", default="active", choices=sorted(KERNEL_SOURCES))
    ap.add_argument("--semi-async", action="store_true",
                    help="run the workload as k semi-asynchronous workers averaged on the "
                         "schedule of Eq. 5 (roofline: the averaging kernel)")
    ap.add_argument("--dt0", type=int, default=5, help="initial interval of Eq. 5")
    ap.add_argument("--unit", type=int, default=1, help="ticks per unit t of Eq. 5")
    args = ap.parse_args()
    if args.traffic_summary:
        res = traffic_summary(*args.traffic_summary, args.kernel, args.copy_bytes, args.workload)
        with open(os.path.join(ROOT, "profiles", f"traffic_{args.kernel}.json"), "w") as fh:
            json.dump(res, fh, indent=1)
        print(json.dumps(res))
        return
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU: both parties share a single MI355X as two HIP "
              f"streams; --gpus {args.gpus} (WORLD_SIZE {world}) is not supported",
              file=sys.stderr)
        sys.exit(2)

    import torch
    import vfl_synth as S
    from paper_2510_12494_amd import vfl as V
    from paper_2510_12494_amd.session import Session

    if args.copy_bytes:
        n = args.copy_bytes // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda:0")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    w = S.get(args.workload)
    if args.id_stride != 1:
        w = w.replace(id_stride=args.id_stride)
    data = S.generate(w)
    params = S.init_params(w)
    if args.semi_async:
        res = semi_async(args, w, data, params)
        out = {
            "metric": METRIC, "value": res["value"], "unit": "samples/s", "n_gpus": 1,
            "steps": args.steps, "warmup": res["warmup"], "ms_per_step": res["ms_per_step"],
            "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
            "dtype": w.dtype, "data": "synthetic (seeded, resident in HBM)",
            "mfma_util_pct": 100.0 * gemm_flops_per_tick(w) / (res["ms_per_step"] / 1e3) / PEAK[w.dtype],
            "config": {"workload": w.name, "mode": "semi-asynchronous workers",
                       **res["semi_async"], "staleness": w.staleness},
            "roofline": res["roofline"],
        }
        if not args.no_cpu_baseline:
            out["cpu_baseline"] = cpu_baseline(w, data, params, args.cpu_seconds)
        print(json.dumps(out), flush=True)
        return
    epoch = w.ticks_per_epoch()
    probe = serial_probe(w, data, params, epoch)
    dom = max(probe, key=lambda k: probe[k][0])
    dom_i = V.KERNEL_CLASSES.index(dom)
    sess = Session(w, data, params, lambda g: S.group_rows(w, g))
    # warm-up through the per-call path (every stash slot gets current
    # operand copies), then bind the resident dataset for graph replay
    warm = max(args.warmup, 2 * (w.staleness + 1))
    t = 0
    for _ in range(warm):
        sess.step(t, epoch=epoch)
        t += 1
    sess.bind()
    cyc = V.VFL_GRAPH_CYCLES * (w.staleness + 1)
    V.vfl_timing_enable(sess.ctx, 1 << dom_i)
    sess.run(t, args.steps)                # captures the graphs the timed region replays
    t += args.steps
    V.vfl_timing_read(sess.ctx, dom_i)

    torch.cuda.synchronize()
    t0 = time.perf_counter()
    sess.run(t, args.steps)
    t += args.steps
    t_host = time.perf_counter() - t0
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    ms, launches, work = V.vfl_timing_read(sess.ctx, dom_i)
    V.vfl_timing_enable(sess.ctx, 0)
    losses = sess.losses([t - w.staleness - 1])
    sess.close()

    R = w.rows_per_tick
    value = args.steps * R / dt
    tick_s = dt / args.steps
    flops = gemm_flops_per_tick(w)
    mfma = flops / tick_s / PEAK[w.dtype]
    is_gemm = dom in GEMM_CLASSES
    avg_s = ms / 1e3 / max(launches, 1)
    per_launch = work / max(launches, 1)
    achieved = per_launch / avg_s if avg_s > 0 else 0.0
    if is_gemm:
        roof = {"bound": "mfma", "achieved": achieved / 1e12, "peak": PEAK[w.dtype] / 1e12,
                "unit": "TFLOP/s"}
    else:
        roof = {"bound": "hbm", "achieved": achieved / 1e9, "peak": HBM_PEAK / 1e9, "unit": "GB/s"}
    roof["frac"] = roof["achieved"] / roof["peak"]
    roof["traffic"] = traffic_for(dom, w.name)
    roof["kernel"] = dom
    roof["launches"] = launches
    roof["avg_us"] = avg_s * 1e6
    roof["work_per_launch"] = per_launch

    out = {
        "metric": METRIC, "value": value, "unit": "samples/s", "n_gpus": 1,
        "steps": args.steps, "warmup": warm, "ms_per_step": tick_s * 1e3,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": w.dtype, "data": "synthetic (seeded, resident in HBM)",
        "mfma_util_pct": 100.0 * mfma, "gemm_gflop_per_step": flops / 1e9,
        "host_enqueue_us_per_step": t_host / args.steps * 1e6,
        "config": {"workload": w.name, "rows": w.n_rows, "rows_per_tick": R, "batch": w.batch,
                   "replicas": w.replicas, "staleness": w.staleness,
                   "bottom_A": "-".join(map(str, [w.A.d_in] + w.A.widths)),
                   "bottom_B": "-".join(map(str, [w.B.d_in] + w.B.widths)),
                   "top": "-".join(map(str, [w.top_in] + w.top.widths)), "lr": w.lr,
                   **({"id_stride": w.id_stride} if w.id_stride != 1 else {})},
        "roofline": roof,
        "kernel_classes_us_per_step_serial": {k: 1e3 * v[0] for k, v in probe.items() if v[1]},
        "graph_ticks": cyc,
        "last_loss": float(losses[0]),
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, data, params, args.cpu_seconds)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
