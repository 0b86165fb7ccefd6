"""The five synthetic workloads of the two-party split-learning training step.

Each workload is a plain description (shapes, schedule knobs, seeds); it holds
none of the method's arithmetic.  Party A is the active party (it holds the
labels and the top model), party B the passive party that publishes its
embeddings (paper, Section 3 "Problem Formulation").

Bottom widths list the output width of each layer; the input width of a
bottom model is ``n_cat * emb_dim + dense`` (gathered embeddings first, dense
features after).  Top widths list the hidden layers followed by the single
logit unit; the top input is ``widths_A[-1] + widths_B[-1]``.

Learning rate: the paper trains with SGD at 0.001 (Section 5, "Parameters");
the tiny synchronous workload uses 0.05 so that a single epoch moves the
parameters measurably.
"""
from __future__ import annotations

import copy
from dataclasses import dataclass, field, asdict
from typing import List


@dataclass
class PartySpec:
    dense: int
    widths: List[int]
    n_cat: int = 0
    vocab: int = 0
    emb_dim: int = 0
    relu: List[bool] | None = None  # per layer; default: ReLU after every layer

    def __post_init__(self):
        if self.relu is None:
            self.relu = [True] * len(self.widths)

    @property
    def d_in(self) -> int:
        return self.n_cat * self.emb_dim + self.dense

    @property
    def d_out(self) -> int:
        return self.widths[-1]

    def layer_dims(self):
        """[(in, out)] per layer."""
        dims, k = [], self.d_in
        for w in self.widths:
            dims.append((k, w))
            k = w
        return dims


@dataclass
class TopSpec:
    widths: List[int]  # hidden widths followed by 1 (the logit)
    relu: List[bool] | None = None  # hidden layers; the logit layer is linear

    def __post_init__(self):
        if self.widths[-1] != 1:
            raise ValueError("the top model ends in a single logit")
        if self.relu is None:
            self.relu = [True] * (len(self.widths) - 1)


@dataclass
class Workload:
    name: str
    n_rows: int
    dtype: str              # "f32" or "bf16": storage / GEMM operand type
    A: PartySpec
    B: PartySpec
    top: TopSpec
    batch: int              # rows per replica batch
    staleness: int          # s >= 0
    replicas: int           # k >= 1
    lr: float
    clip: float = 0.0       # per-row L2 clip bound C; <= 0: no clip
    sigma: float = 0.0      # noise multiplier; std = sigma * C (C = 1 when no clip)
    noise_emb: bool = False
    noise_grad: bool = False
    clip_emb: bool = False
    clip_grad: bool = False
    fifo_discard: bool = False   # a full channel drops its oldest group
    labels: str = "teacher"  # "logistic" | "teacher" | "bernoulli" | "regression"
    loss: str = "bce"        # "bce" (Eq. 1 on a logit) | "mse" (squared error on a prediction)
    label_p: float = 0.25
    zipf_a: float = 1.1
    id_shift: int = 0        # ids (k * id_stride + id_shift) mod vocab: moves the hot ids
    id_stride: int = 1       # coprime with vocab: scatters the Zipf ranks over the ids (hashed ids)
    data_seed: int = 0
    init_seed: int = 0
    noise_seed: int = 0

    @property
    def rows_per_tick(self) -> int:
        return self.batch * self.replicas

    @property
    def top_in(self) -> int:
        return self.A.d_out + self.B.d_out

    def ticks_per_epoch(self) -> int:
        R = self.rows_per_tick
        return (self.n_rows + R - 1) // R

    def with_rows(self, n_rows: int) -> "Workload":
        w = copy.deepcopy(self)
        w.n_rows = int(n_rows)
        return w

    def replace(self, **kw) -> "Workload":
        w = copy.deepcopy(self)
        for k, v in kw.items():
            if not hasattr(w, k):
                raise AttributeError(k)
            setattr(w, k, v)
        return w

    def to_dict(self):
        return asdict(self)


def _w(i: int, **kw) -> Workload:
    kw.setdefault("data_seed", 1000 + i)
    kw.setdefault("init_seed", 2000 + i)
    kw.setdefault("noise_seed", 0x5EED0000 + i)
    return Workload(**kw)


def tiny_sync() -> Workload:
    """4096 rows, 16 + 16 fp32 features, logistic labels; 16->32->16 bottoms,
    32->16->1 top; batch 256, s=0, k=1, lr 0.05, no noise."""
    return _w(1, name="tiny_sync", n_rows=4096, dtype="f32",
              A=PartySpec(dense=16, widths=[32, 16]),
              B=PartySpec(dense=16, widths=[32, 16]),
              top=TopSpec(widths=[16, 1]),
              batch=256, staleness=0, replicas=1, lr=0.05, labels="logistic")


def dense_tabular() -> Workload:
    """1M rows, 64 + 64 bf16 features, teacher labels; 64->256->128 bottoms,
    256->256->1 top; batch 4096, s=2, k=1."""
    return _w(2, name="dense_tabular", n_rows=1_000_000, dtype="bf16",
              A=PartySpec(dense=64, widths=[256, 128]),
              B=PartySpec(dense=64, widths=[256, 128]),
              top=TopSpec(widths=[256, 1]),
              batch=4096, staleness=2, replicas=1, lr=0.001, labels="teacher")


def ctr() -> Workload:
    """4M rows, 26 categorical fields split 13/13 (vocab 100k, Zipf(1.1) ids,
    16-wide fp32 embeddings) plus 13 dense features on A; bottoms
    concat->256->64, top 128->128->1; batch 8192, s=2, Bernoulli(0.25) labels."""
    return _w(3, name="ctr", n_rows=4_000_000, dtype="f32",
              A=PartySpec(dense=13, n_cat=13, vocab=100_000, emb_dim=16, widths=[256, 64]),
              B=PartySpec(dense=0, n_cat=13, vocab=100_000, emb_dim=16, widths=[256, 64]),
              top=TopSpec(widths=[128, 1]),
              batch=8192, staleness=2, replicas=1, lr=0.001, labels="bernoulli",
              label_p=0.25)


def hetero() -> Workload:
    """2M rows; A 8 features with bottom 8->64, B 500 features with bottom
    500->1024->512->128, bf16; top 192->256->1; batch 8192, s=4, k=4."""
    return _w(4, name="hetero", n_rows=2_000_000, dtype="bf16",
              A=PartySpec(dense=8, widths=[64]),
              B=PartySpec(dense=500, widths=[1024, 512, 128]),
              top=TopSpec(widths=[256, 1]),
              batch=8192, staleness=4, replicas=4, lr=0.001, labels="teacher")


def private() -> Workload:
    """dense_tabular shapes at 10M rows, batch 16384, s=2, k=2; per-row L2
    clip C=1 then Gaussian noise sigma=0.5 on the published embeddings and on
    the returned embedding gradients."""
    return _w(5, name="private", n_rows=10_000_000, dtype="bf16",
              A=PartySpec(dense=64, widths=[256, 128]),
              B=PartySpec(dense=64, widths=[256, 128]),
              top=TopSpec(widths=[256, 1]),
              batch=16384, staleness=2, replicas=2, lr=0.001, labels="teacher",
              clip=1.0, sigma=0.5, clip_emb=True, clip_grad=True,
              noise_emb=True, noise_grad=True)


def regression() -> Workload:
    """Regression with ten-layer MLP bottoms (the paper's bottom model,
    Section 5 "Models"; its regression sets are scored by RMSE): 1M rows,
    140 + 140 bf16 features (the width of a blog-feedback-like table), a
    continuous target from a random teacher; each bottom nine 256-wide ReLU
    layers and a 64-wide cut layer, top 128->64->1 with a linear output and
    the mean squared error; batch 4096, s=2, k=2."""
    return _w(6, name="regression", n_rows=1_000_000, dtype="bf16",
              A=PartySpec(dense=140, widths=[256] * 9 + [64]),
              B=PartySpec(dense=140, widths=[256] * 9 + [64]),
              top=TopSpec(widths=[64, 1]),
              batch=4096, staleness=2, replicas=2, lr=0.001, labels="regression", loss="mse")


ALL = {f.__name__: f for f in (tiny_sync, dense_tabular, ctr, hetero, private, regression)}


def get(name: str) -> Workload:
    return ALL[name]()
