"""Second, independently written formulation of the training loop, used only
to pin the oracle: PyTorch float64 autograd on the CPU, a full list of party
B's parameter versions instead of a ring, and one big batch per group instead
of per-replica workers.

For batch group u (in order): B's embedding is computed at B's version
max(0, u - s) (the delayed parameter of Assumption 4 / the Theorem's update
rule), optionally clipped per row and noised; A and the top model run at
their current parameters; the loss is the mean BCE of Eq. (1); the gradient
message is the per-row gradient w.r.t. the published embedding, optionally
clipped and noised; B's gradient is the vector-Jacobian product of its
embedding at the delayed version with that message / R; every party takes
one SGD step (Eq. 2).

Dropped channel entries (Section 4.1 "System Design"): for a group whose embedding is
dropped nothing is computed; for one whose gradient is dropped A and the top
model step and B does not.  B's version for the forward of group u is then
the number of B updates applied by the groups g < u - s.

Storage rounding (``rnd``, ``points``): the same named points as the
oracle's emulation modes, placed in the autograd graph rather than in a
hand-written backward.  A value point (inputs, weight operands, layer
outputs, messages) rounds in the forward pass and passes the gradient
through unchanged; a gradient point (a layer's pre-activation) is the
identity forward and rounds the gradient arriving there.  Gradients are
taken of the sum of the per-row losses (the 1/R of the mean goes into the
SGD step), the scale at which the deltas are stored.  The rounding function
here works on the float64 bit pattern (round to nearest even on the low 45
bits for bfloat16), independently of the oracle's.
"""
import numpy as np
import torch

from oracle.philox import gaussian, TAG_EMB, TAG_GRAD


def _t(a):
    return torch.tensor(np.asarray(a, dtype=np.float64))


def bf16_bits(x):
    """float64 -> nearest bfloat16 value (ties to even), on the bit pattern:
    keep the sign, exponent and top 7 fraction bits."""
    b = x.detach().contiguous().view(torch.int64)
    drop = 45
    lsb = (b >> drop) & 1
    b = (b + ((1 << (drop - 1)) - 1) + lsb) & ~((1 << drop) - 1)
    return b.view(torch.float64)


def f32_cast(x):
    return x.detach().to(torch.float32).to(torch.float64)


class _Value(torch.autograd.Function):
    @staticmethod
    def forward(ctx, x, fn):
        return fn(x)

    @staticmethod
    def backward(ctx, g):
        return g, None


class _Grad(torch.autograd.Function):
    @staticmethod
    def forward(ctx, x, fn):
        ctx.fn = fn
        return x.clone()

    @staticmethod
    def backward(ctx, g):
        return ctx.fn(g), None


class _Rounding:
    def __init__(self, rnd, points):
        self.rnd = rnd
        self.points = set(points) if rnd is not None else set()

    def v(self, point, x):
        return _Value.apply(x, self.rnd) if point in self.points else x

    def g(self, point, x):
        return _Grad.apply(x, self.rnd) if point in self.points else x


def _bottom(spec, P, party, x_dense, ids, Q, cut_point):
    xs = []
    if spec.n_cat:
        rows = torch.as_tensor(ids.astype(np.int64)) + spec.vocab * torch.arange(spec.n_cat)[None, :]
        xs.append(P[f"{party}.T"][rows.reshape(-1)].reshape(ids.shape[0], -1))
    if spec.dense:
        xs.append(_t(x_dense))
    a = torch.cat(xs, dim=1) if len(xs) > 1 else xs[0]
    a = Q.v("input", a)
    L = len(spec.widths)
    for l in range(L):
        pre = a @ Q.v("weight", P[f"{party}.W{l}"]).T + P[f"{party}.b{l}"]
        pre = Q.g(cut_point if l == L - 1 else "delta.bottom", pre)
        if spec.relu[l]:
            pre = torch.relu(pre)
        a = Q.v("act.bottom", pre)
    return a


def _clip(v, C):
    n = torch.linalg.norm(v, dim=1, keepdim=True)
    c = torch.where(n > C, C / torch.where(n > 0, n, torch.ones_like(n)), torch.ones_like(n))
    return v * c


def run_history(w, params, data, n_groups, rows_of, discard=None, rnd=None, points=()):
    """Returns (losses per group that A stepped on, final parameters as a
    float64 numpy dict); discard: {group: "emb" | "grad"}; rnd: rounding
    function on float64 tensors (None: no storage rounding) applied at
    ``points``."""
    discard = discard or {}
    Q = _Rounding(rnd, points)
    master = f32_cast if "master" in Q.points else (lambda x: x)
    s = w.staleness
    std = w.sigma * (w.clip if w.clip > 0 else 1.0)
    cur = {k: _t(v) for k, v in params.items()}
    b_keys = [k for k in cur if k.startswith("B.")]
    versions = [{k: cur[k].clone() for k in b_keys}]
    losses = []
    for u in range(n_groups):
        if discard.get(u) == "emb":
            continue
        rows = np.concatenate([np.arange(a, a + c) for a, c in rows_of(u)])
        R = len(rows)
        v_fwd = sum(1 for g in range(max(0, u - s)) if g not in discard)
        PB = {k: versions[v_fwd][k].clone().requires_grad_(True) for k in b_keys}
        PA = {k: v.clone().requires_grad_(True) for k, v in cur.items() if not k.startswith("B.")}
        xb = data["xb"][rows] if data["xb"] is not None else None
        idb = data["idb"][rows] if data["idb"] is not None else None
        z = _bottom(w.B, PB, "B", xb, idb, Q, "delta.cut_b")
        zc = _clip(z, w.clip) if w.clip_emb else z
        if w.noise_emb:
            zc = zc + std * _t(gaussian(w.noise_seed, u, rows, z.shape[1], TAG_EMB))
        if w.clip_emb or w.noise_emb:
            zc = Q.v("msg.emb", zc)
        zhat = zc.detach().requires_grad_(True)
        xa = data["xa"][rows] if data["xa"] is not None else None
        ida = data["ida"][rows] if data["ida"] is not None else None
        za = _bottom(w.A, PA, "A", xa, ida, Q, "delta.cut_a")
        h = torch.cat([za, zhat], dim=1)
        nT = len(w.top.widths)
        for j in range(nT):
            if j < nT - 1:
                h = h @ Q.v("weight", PA[f"top.W{j}"]).T + PA[f"top.b{j}"]
                h = Q.g("delta.top", h)
                if w.top.relu[j]:
                    h = torch.relu(h)
                h = Q.v("act.top", h)
            else:
                h = h @ PA[f"top.W{j}"].T + PA[f"top.b{j}"]     # logit: float32 master weight
        y = _t(data["y"][rows])
        if getattr(w, "loss", "bce") == "mse":
            loss_sum = ((h[:, 0] - y) ** 2).sum()
        else:
            loss_sum = torch.nn.functional.binary_cross_entropy_with_logits(h[:, 0], y, reduction="sum")
        names = list(PA)
        grads = torch.autograd.grad(loss_sum, [PA[k] for k in names] + [zhat])
        gmsg = grads[-1]                            # per-row gradient
        if w.clip_grad:
            gmsg = _clip(gmsg, w.clip)
        if w.noise_grad:
            gmsg = gmsg + std * _t(gaussian(w.noise_seed, u, rows, gmsg.shape[1], TAG_GRAD))
        if "msg.grad" in Q.points:
            gmsg = Q.rnd(gmsg)
        gB = torch.autograd.grad(zc, [PB[k] for k in b_keys], grad_outputs=gmsg, allow_unused=True)
        with torch.no_grad():
            for k, g in zip(names, grads[:-1]):
                cur[k] = master(cur[k] - w.lr * (g / R))
            if discard.get(u) == "grad":
                losses.append(float(loss_sum.detach()) / R)
                continue
            nv = {}
            for k, g in zip(b_keys, gB):
                nv[k] = master(versions[-1][k] - w.lr * ((g if g is not None else 0.0) / R))
            versions.append(nv)
            cur.update(nv)
        losses.append(float(loss_sum.detach()) / R)
    return losses, {k: v.detach().numpy() for k, v in cur.items()}
