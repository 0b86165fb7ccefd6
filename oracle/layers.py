"""Plain float64 definitions of the pieces one training step is made of.

Test infrastructure only (see ``oracle/__init__.py``).

* Bottom and top models are stacks of fully connected layers,
  y = x W^T + b, W stored [out, in], optionally followed by ReLU (the paper's
  bottom and top models are MLPs, Section 5 "Models").
* The loss is the binary cross-entropy of Eq. (1) on the top model's logit,
  averaged over the rows it is given; for the regression tasks (Section 5,
  "Datasets" and "Evaluation Metrics") the mean squared error of the top
  model's output.
* Categorical inputs look up rows of per-field embedding tables; the bottom
  model's input is the concatenation of the looked-up rows (field order) and
  the dense features.
* The exchanged embedding (and, in the private workload, the returned
  gradient) is clipped per row to L2 norm C before Gaussian noise is added.
  The paper adds Gaussian noise to the passive party's embedding (Appendix
  "Differential Privacy Protocol", Assumption 5); the per-row clip is the
  workload's addition.
"""
from __future__ import annotations

import numpy as np


def linear(x, W, b):
    """Fully connected layer: x [n, in], W [out, in], b [out] -> [n, out]."""
    return x @ W.T + b


def relu(p):
    return np.maximum(p, 0.0)


def relu_mask(a):
    """Derivative of ReLU evaluated through its output: 1 where a > 0, else 0
    (the derivative at the kink is taken as 0)."""
    return (np.asarray(a) > 0.0).astype(np.float64)


def sigmoid(x):
    x = np.asarray(x, dtype=np.float64)
    e = np.exp(-np.abs(x))
    return np.where(x >= 0, 1.0 / (1.0 + e), e / (1.0 + e))


def bce_direct(yhat, y):
    """Eq. (1) per row, written on the predicted probability."""
    return -(y * np.log(yhat) + (1.0 - y) * np.log(1.0 - yhat))


def bce_with_logits(logit, y):
    """Eq. (1) per row with yhat = sigmoid(logit), in the overflow-free form
    max(l, 0) - y l + log(1 + exp(-|l|)) (algebraically identical)."""
    l = np.asarray(logit, dtype=np.float64)
    return np.maximum(l, 0.0) - y * l + np.log1p(np.exp(-np.abs(l)))


def bce_dlogit(logit, y):
    """d/dl of the per-row loss: sigmoid(l) - y."""
    return sigmoid(logit) - y


def mse(pred, y):
    """Squared error of a regression output per row, (pred - y)^2; its mean
    over the rows is the regression loss (scored as RMSE, Section 5
    "Evaluation Metrics")."""
    d = np.asarray(pred, dtype=np.float64) - y
    return d * d


def mse_dpred(pred, y):
    """d/dpred of the per-row squared error: 2 (pred - y)."""
    return 2.0 * (np.asarray(pred, dtype=np.float64) - y)


def clip_rows(v, C):
    """Per-row L2 clip: returns (v * c, n, c) with n = ||v_i||, c = min(1, C/n)
    (c = 1 for n = 0)."""
    v = np.asarray(v, dtype=np.float64)
    n = np.sqrt(np.sum(v * v, axis=1))
    c = np.ones_like(n)
    big = n > C
    c[big] = C / n[big]
    return v * c[:, None], n, c


def clip_rows_backward(g, v, n, c, C):
    """Vector-Jacobian product of ``clip_rows`` at input v: rows with n <= C
    pass g unchanged; otherwise c * (g - u (u . g)) with u = v / n."""
    g = np.array(g, dtype=np.float64, copy=True)
    big = n > C
    if np.any(big):
        u = v[big] / n[big][:, None]
        gb = g[big]
        g[big] = c[big][:, None] * (gb - u * np.sum(u * gb, axis=1, keepdims=True))
    return g


def gather_embeddings(table, ids, vocab):
    """table [n_cat * vocab, E], ids [n, n_cat] -> [n, n_cat * E]: row of
    field f is table[f * vocab + ids[:, f]]."""
    n, n_cat = ids.shape
    rows = ids.astype(np.int64) + vocab * np.arange(n_cat, dtype=np.int64)[None, :]
    return table[rows].reshape(n, -1)


def embedding_grad(g_emb, ids, vocab, table_shape):
    """Dense gradient of the tables for per-row gradient g_emb [n, n_cat * E]:
    sum of the rows' gradients landing on each table row."""
    n, n_cat = ids.shape
    E = table_shape[1]
    rows = ids.astype(np.int64) + vocab * np.arange(n_cat, dtype=np.int64)[None, :]
    out = np.zeros(table_shape, dtype=np.float64)
    np.add.at(out, rows.reshape(-1), np.asarray(g_emb, np.float64).reshape(n * n_cat, E))
    return out
