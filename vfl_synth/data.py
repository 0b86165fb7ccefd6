"""Seeded synthetic inputs for the split-learning workloads.

Everything here is input generation: feature matrices, categorical ids,
labels, initial parameters and the rows a batch group covers.  None of the
training step's arithmetic lives in this module; both the oracle and the GPU
harness consume what it produces.

Stand-ins: the dense workloads stand in for the paper's 1M x 500 synthetic
tabular set (Section 5, "Datasets"); the categorical workload mimics the
13 numeric + 26 categorical fields of Criteo 1TB (Appendix, "System
Performance on Large Dataset").  No dataset items are reproduced.

Rows are generated in fixed chunks of 2**20 rows, each from its own seeded
stream, so that any prefix of a dataset is reproducible on its own.
"""
from __future__ import annotations

import numpy as np
import torch

from .workloads import Workload

CHUNK = 1 << 20


def _rng(*keys) -> np.random.Generator:
    return np.random.default_rng([int(k) & 0xFFFFFFFF for k in keys])


def to_bf16_values(a: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even) and return
    them as float32 (torch's conversion is the rounding routine)."""
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return t.to(torch.bfloat16).to(torch.float32).numpy()


def _zipf_cdf(vocab: int, a: float) -> np.ndarray:
    k = np.arange(1, vocab + 1, dtype=np.float64)
    p = k ** (-a)
    c = np.cumsum(p)
    return c / c[-1]


def _chunks(n_rows: int):
    c = 0
    while c * CHUNK < n_rows:
        lo = c * CHUNK
        yield c, lo, min(n_rows, lo + CHUNK)
        c += 1


def generate(w: Workload, n_rows: int | None = None) -> dict:
    """Return the dataset of ``n_rows`` rows (default ``w.n_rows``).

    Keys: ``xa``, ``xb`` float32 [n, dense] (bf16-exact values when
    ``w.dtype == 'bf16'``, None when a party has no dense features), ``ida``,
    ``idb`` int32 [n, n_cat] (None without categorical fields), ``y`` float32
    [n] in {0, 1} (real-valued targets for ``labels == 'regression'``).
    """
    n = w.n_rows if n_rows is None else int(n_rows)
    out = {"xa": None, "xb": None, "ida": None, "idb": None}
    for key, spec, pid in (("xa", w.A, 0), ("xb", w.B, 1)):
        if spec.dense:
            a = np.empty((n, spec.dense), np.float32)
            for c, lo, hi in _chunks(n):
                a[lo:hi] = _rng(w.data_seed, c, pid, 0).standard_normal(
                    (hi - lo, spec.dense), dtype=np.float32)
            if w.dtype == "bf16":
                a = to_bf16_values(a)
            out[key] = a
    for key, spec, pid in (("ida", w.A, 0), ("idb", w.B, 1)):
        if spec.n_cat:
            cdf = _zipf_cdf(spec.vocab, w.zipf_a)
            ids = np.empty((n, spec.n_cat), np.int32)
            for c, lo, hi in _chunks(n):
                u = _rng(w.data_seed, c, pid, 1).random((hi - lo, spec.n_cat))
                k = np.minimum(np.searchsorted(cdf, u, side="right"), spec.vocab - 1)
                ids[lo:hi] = (k.astype(np.int64) * w.id_stride + w.id_shift) % spec.vocab
            out[key] = ids
    out["y"] = _labels(w, out, n)
    return out


def _labels(w: Workload, d: dict, n: int) -> np.ndarray:
    if w.labels == "bernoulli":
        y = np.empty(n, np.float32)
        for c, lo, hi in _chunks(n):
            y[lo:hi] = _rng(w.data_seed, c, 9, 2).random(hi - lo) < w.label_p
        return y
    xs = [x for x in (d["xa"], d["xb"]) if x is not None]
    dim = sum(x.shape[1] for x in xs)
    if w.labels == "logistic":
        # y ~ Bernoulli(sigmoid(v . x)), v ~ N(0, 1/dim)
        v = _rng(w.data_seed, 7, 0).standard_normal(dim) / np.sqrt(dim)
        y = np.empty(n, np.float32)
        for c, lo, hi in _chunks(n):
            x = np.concatenate([a[lo:hi].astype(np.float64) for a in xs], axis=1)
            p = 1.0 / (1.0 + np.exp(-(x @ v)))
            y[lo:hi] = _rng(w.data_seed, c, 9, 3).random(hi - lo) < p
        return y
    if w.labels in ("teacher", "regression"):
        # random 2-layer teacher dim -> 32 -> 1 (ReLU, zero biases,
        # weights ~ N(0, 1/fan_in)); label = teacher output above its
        # median, or (regression) the teacher output itself
        r = _rng(w.data_seed, 7, 1)
        w1 = r.standard_normal((32, dim)) / np.sqrt(dim)
        w2 = r.standard_normal(32) / np.sqrt(32)
        t = np.empty(n, np.float64)
        for c, lo, hi in _chunks(n):
            x = np.concatenate([a[lo:hi].astype(np.float64) for a in xs], axis=1)
            t[lo:hi] = np.maximum(x @ w1.T, 0.0) @ w2
        if w.labels == "regression":
            return t.astype(np.float32)
        return (t > np.median(t)).astype(np.float32)
    raise ValueError(w.labels)


def init_params(w: Workload) -> dict:
    """Initial parameters, float32 numpy arrays keyed ``"<party>.<kind><layer>"``.

    Dense layers: W [out, in] and b [out] ~ U(-1/sqrt(in), 1/sqrt(in));
    embedding tables ``<party>.T`` [n_cat * vocab, emb_dim] ~ N(0, 0.05^2),
    field f occupying rows [f * vocab, (f + 1) * vocab).
    """
    p = {}
    for pname, spec, pid in (("A", w.A, 0), ("B", w.B, 1)):
        for l, (fi, fo) in enumerate(spec.layer_dims()):
            r = _rng(w.init_seed, pid, l)
            lim = 1.0 / np.sqrt(fi)
            p[f"{pname}.W{l}"] = r.uniform(-lim, lim, (fo, fi)).astype(np.float32)
            p[f"{pname}.b{l}"] = r.uniform(-lim, lim, fo).astype(np.float32)
        if spec.n_cat:
            r = _rng(w.init_seed, pid, 99)
            p[f"{pname}.T"] = (0.05 * r.standard_normal(
                (spec.n_cat * spec.vocab, spec.emb_dim))).astype(np.float32)
    fi = w.top_in
    for l, fo in enumerate(w.top.widths):
        r = _rng(w.init_seed, 2, l)
        lim = 1.0 / np.sqrt(fi)
        p[f"top.W{l}"] = r.uniform(-lim, lim, (fo, fi)).astype(np.float32)
        p[f"top.b{l}"] = r.uniform(-lim, lim, fo).astype(np.float32)
        fi = fo
    return p


def group_rows(w: Workload, g: int, n_rows: int | None = None):
    """Rows of batch group ``g``: no shuffling, groups walk the dataset in
    order and wrap at the end of an epoch; the last group of an epoch may be
    short.  Returns [(start, count)] per replica, consecutive chunks of at
    most ``w.batch`` rows."""
    n = w.n_rows if n_rows is None else int(n_rows)
    R = w.rows_per_tick
    T = (n + R - 1) // R
    start = (g % T) * R
    count = min(R, n - start)
    out, o = [], 0
    while o < count:
        c = min(w.batch, count - o)
        out.append((start + o, c))
        o += c
    return out
