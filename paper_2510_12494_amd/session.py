"""Device-side harness around the C ABI: allocates the workspace and the
resident dataset with PyTorch, creates the two party streams, uploads
parameters and marshals batch descriptors.  No arithmetic of the training
step happens here.
"""
from __future__ import annotations

import ctypes as C

import numpy as np
import torch

from . import vfl as V


def _ld(n: int) -> int:
    return max(8, (n + 7) // 8 * 8)


def bottom_spec(p) -> V.vfl_bottom_spec:
    s = V.vfl_bottom_spec()
    s.dense_in, s.n_cat, s.vocab, s.emb_dim = p.dense, p.n_cat, p.vocab, p.emb_dim
    s.n_layers = len(p.widths)
    for i, wd in enumerate(p.widths):
        s.widths[i] = wd
    s.relu_mask = sum(1 << i for i, r in enumerate(p.relu) if r)
    return s


def top_spec(t) -> V.vfl_top_spec:
    s = V.vfl_top_spec()
    s.n_layers = len(t.widths)
    for i, wd in enumerate(t.widths):
        s.widths[i] = wd
    s.relu_mask = sum(1 << i for i, r in enumerate(t.relu) if r)
    return s


def opts(w) -> V.vfl_opts:
    o = V.vfl_opts()
    o.dtype = V.VFL_BF16 if w.dtype == "bf16" else V.VFL_F32
    o.batch, o.staleness, o.replicas = w.batch, w.staleness, w.replicas
    o.lr, o.clip_c, o.sigma = w.lr, (w.clip if w.clip > 0 else 0.0), w.sigma
    o.seed = w.noise_seed
    o.flags = ((V.VFL_NOISE_EMB if w.noise_emb else 0) | (V.VFL_NOISE_GRAD if w.noise_grad else 0)
               | (V.VFL_CLIP_EMB if w.clip_emb else 0) | (V.VFL_CLIP_GRAD if w.clip_grad else 0)
               | (V.VFL_FIFO_DISCARD if getattr(w, "fifo_discard", False) else 0)
               | (V.VFL_LOSS_MSE if getattr(w, "loss", "bce") == "mse" else 0))
    return o


class Session:
    """One training context of workload ``w`` on ``device`` over the resident
    dataset ``data`` (numpy arrays from the seeded generators); ``rows_of(g)``
    gives the [(start, count)] replica rows of batch group g."""

    def __init__(self, w, data: dict, params: dict, rows_of, device: str = "cuda:0",
                 one_stream: bool = False, static_ws: bool = False):
        self.w = w
        self.dev = torch.device(device)
        self.rows_of = rows_of
        self.tdt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
        self.esz = 2 if w.dtype == "bf16" else 4
        self.specA, self.specB = bottom_spec(w.A), bottom_spec(w.B)
        self.specT, self.o = top_spec(w.top), opts(w)
        self.nbytes = V.vfl_workspace_size(self.specA, self.specB, self.specT, self.o)
        with torch.cuda.device(self.dev):
            self.sa = torch.cuda.Stream(device=self.dev)
            # one_stream: both parties on one stream (no overlap between them)
            self.sb = self.sa if one_stream else torch.cuda.Stream(device=self.dev)
        if static_ws:
            # the library's own per-device workspace (vfl_create_static)
            self.ws = None
            with torch.cuda.device(self.dev):
                self.ctx = V.vfl_create_static(self.specA, self.specB, self.specT, self.o,
                                               self.sa.cuda_stream, self.sb.cuda_stream)
        else:
            self.ws = torch.empty(self.nbytes, dtype=torch.uint8, device=self.dev)
            self.ctx = V.vfl_create(self.specA, self.specB, self.specT, self.o, self.ws.data_ptr(),
                                    self.nbytes, self.sa.cuda_stream, self.sb.cuda_stream)
        self.data = {}
        for key in ("xa", "xb"):
            x = data.get(key)
            if x is None:
                self.data[key] = None
                continue
            n, d = x.shape
            ld = _ld(d)
            t = torch.zeros((n, ld), dtype=self.tdt, device=self.dev)
            t[:, :d] = torch.from_numpy(np.ascontiguousarray(x)).to(self.tdt).to(self.dev)
            self.data[key] = t
        for key in ("ida", "idb"):
            x = data.get(key)
            self.data[key] = None if x is None else torch.from_numpy(np.ascontiguousarray(x)).to(self.dev)
        self.data["y"] = torch.from_numpy(np.ascontiguousarray(data["y"])).to(self.dev)
        torch.cuda.synchronize(self.dev)
        self.set_params(params)
        self.loss = torch.zeros(1 << 16, dtype=torch.float32, device=self.dev)
        self._cache = {}

    # ------------------------------------------------------------ params
    @staticmethod
    def _key(k: str):
        party, name = k.split(".")
        pid = {"A": V.VFL_PARTY_A, "B": V.VFL_PARTY_B, "top": V.VFL_TOP}[party]
        if name == "T":
            return pid, 0, V.VFL_PARAM_TABLE
        kind = V.VFL_PARAM_W if name[0] == "W" else V.VFL_PARAM_B
        return pid, int(name[1:]), kind

    def set_params(self, params: dict):
        for k, v in params.items():
            pid, layer, kind = self._key(k)
            a = np.ascontiguousarray(v, dtype=np.float32)
            V.vfl_set_param(self.ctx, pid, layer, kind, a.ctypes.data, a.nbytes, False)

    def params(self, keys) -> dict:
        out = {}
        for k, shape in keys.items():
            pid, layer, kind = self._key(k)
            a = np.empty(shape, dtype=np.float32)
            V.vfl_get_param(self.ctx, pid, layer, kind, a.ctypes.data, a.nbytes, False)
            out[k] = a
        return out

    # ----------------------------------------------------------- batches
    def batches(self, party: str, g: int):
        reps = self.rows_of(g)
        x = self.data["xa" if party == "A" else "xb"]
        ids = self.data["ida" if party == "A" else "idb"]
        y = self.data["y"]
        out = []
        for start, cnt in reps:
            b = V.vfl_batch()
            if x is not None:
                b.dense = x.data_ptr() + start * x.shape[1] * self.esz
                b.ld = x.shape[1]
            if ids is not None:
                b.ids = ids.data_ptr() + start * ids.shape[1] * 4
            if party == "A":
                b.labels = y.data_ptr() + start * 4
            b.rows = cnt
            b.row0 = start
            out.append(b)
        return out

    def _cached(self, party: str, g: int):
        """ctypes array of group g's replica batches (cached per group)."""
        key = (party, g)
        hit = self._cache.get(key)
        if hit is None:
            bs = self.batches(party, g)
            hit = ((V.vfl_batch * len(bs))(*bs), len(bs))
            if len(self._cache) < 4096:
                self._cache[key] = hit
        return hit

    def step(self, t: int, n_groups: int | None = None, epoch: int | None = None):
        """Tick t of the deterministic schedule (n_groups None: unbounded).
        ``epoch``: groups per epoch, so that batch descriptors are reused."""
        s = self.w.staleness
        lib = V.library()
        nb = na = 0
        bb = aa = None
        if n_groups is None or t < n_groups:
            bb, nb = self._cached("B", t if epoch is None else t % epoch)
        u = t - s
        if u >= 0 and (n_groups is None or u < n_groups):
            aa, na = self._cached("A", u if epoch is None else u % epoch)
        lp = self.loss.data_ptr() + 4 * (u % self.loss.numel()) if na else None
        st = lib.vfl_step(self.ctx, t, aa, na, bb, nb, lp)
        if st != V.VFL_OK:
            V._chk(st, "vfl_step", self.ctx)

    def bind(self):
        """Bind the resident dataset (all rows) for run()."""
        ds = []
        for party in ("A", "B"):
            x = self.data["xa" if party == "A" else "xb"]
            ids = self.data["ida" if party == "A" else "idb"]
            d = V.vfl_dataset()
            if x is not None:
                d.dense, d.ld = x.data_ptr(), x.shape[1]
            if ids is not None:
                d.ids = ids.data_ptr()
            if party == "A":
                d.labels = self.data["y"].data_ptr()
            ds.append(d)
        V.vfl_bind_dataset(self.ctx, ds[0], ds[1], self.data["y"].shape[0])

    def run(self, t0: int, n: int):
        """Ticks t0 .. t0+n-1 over the bound dataset by graph replay; group
        u's loss lands in the loss ring at u mod its length."""
        V.vfl_run(self.ctx, t0, n, self.loss.data_ptr(), self.loss.numel())

    def message(self, which: int, g: int) -> tuple[np.ndarray, tuple]:
        rows = sum(c for _, c in self.rows_of(g))
        d = self.w.B.widths[-1]
        if self.esz == 2:
            raw = np.empty((rows, d), dtype=np.uint16)
            hdr = V.vfl_get_message(self.ctx, which, g, raw.ctypes.data, raw.nbytes)
            vals = (raw.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
        else:
            raw = np.empty((rows, d), dtype=np.float32)
            hdr = V.vfl_get_message(self.ctx, which, g, raw.ctypes.data, raw.nbytes)
            vals = raw.astype(np.float64)
        return vals, hdr

    def losses(self, groups) -> np.ndarray:
        torch.cuda.synchronize(self.dev)
        l = self.loss.cpu().numpy()
        return np.array([l[u % l.size] for u in groups], dtype=np.float64)

    def close(self):
        if self.ctx:
            V.vfl_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
