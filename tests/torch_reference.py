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

Dropped channel entries (Section 4.2): for a group whose embedding is
dropped nothing is computed; for one whose gradient is dropped A and the top
model step and B does not.  B's version for the forward of group u is then
the number of B updates applied by the groups g < u - s.
"""
import numpy as np
import torch

from oracle.philox import gaussian, TAG_EMB, TAG_GRAD


def _t(a):
    return torch.tensor(np.asarray(a, dtype=np.float64))


def _bottom(spec, P, party, x_dense, ids):
    xs = []
    if spec.n_cat:
        rows = torch.as_tensor(ids.astype(np.int64)) + spec.vocab * torch.arange(spec.n_cat)[None, :]
        xs.append(P[f"{party}.T"][rows.reshape(-1)].reshape(ids.shape[0], -1))
    if spec.dense:
        xs.append(_t(x_dense))
    a = torch.cat(xs, dim=1) if len(xs) > 1 else xs[0]
    for l in range(len(spec.widths)):
        a = a @ P[f"{party}.W{l}"].T + P[f"{party}.b{l}"]
        if spec.relu[l]:
            a = torch.relu(a)
    return a


def _clip(v, C):
    n = torch.linalg.norm(v, dim=1, keepdim=True)
    c = torch.where(n > C, C / torch.where(n > 0, n, torch.ones_like(n)), torch.ones_like(n))
    return v * c


def run_history(w, params, data, n_groups, rows_of, discard=None):
    """Returns (losses per group that A stepped on, final parameters as a
    float64 numpy dict); discard: {group: "emb" | "grad"}."""
    discard = discard or {}
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
        z = _bottom(w.B, PB, "B", xb, idb)
        zc = _clip(z, w.clip) if w.clip_emb else z
        if w.noise_emb:
            zc = zc + std * _t(gaussian(w.noise_seed, u, rows, z.shape[1], TAG_EMB))
        zhat = zc.detach().requires_grad_(True)
        xa = data["xa"][rows] if data["xa"] is not None else None
        ida = data["ida"][rows] if data["ida"] is not None else None
        za = _bottom(w.A, PA, "A", xa, ida)
        h = torch.cat([za, zhat], dim=1)
        nT = len(w.top.widths)
        for j in range(nT):
            h = h @ PA[f"top.W{j}"].T + PA[f"top.b{j}"]
            if j < nT - 1 and w.top.relu[j]:
                h = torch.relu(h)
        y = _t(data["y"][rows])
        loss = torch.nn.functional.binary_cross_entropy_with_logits(h[:, 0], y)
        names = list(PA)
        grads = torch.autograd.grad(loss, [PA[k] for k in names] + [zhat])
        gmsg = grads[-1] * R                        # per-row gradient
        if w.clip_grad:
            gmsg = _clip(gmsg, w.clip)
        if w.noise_grad:
            gmsg = gmsg + std * _t(gaussian(w.noise_seed, u, rows, gmsg.shape[1], TAG_GRAD))
        gB = torch.autograd.grad(zc, [PB[k] for k in b_keys], grad_outputs=gmsg / R,
                                 allow_unused=True)
        with torch.no_grad():
            for k, g in zip(names, grads[:-1]):
                cur[k] = cur[k] - w.lr * g
            if discard.get(u) == "grad":
                losses.append(float(loss.detach()))
                continue
            nv = {}
            for k, g in zip(b_keys, gB):
                nv[k] = versions[-1][k] - w.lr * (g if g is not None else 0.0)
            versions.append(nv)
            cur.update(nv)
        losses.append(float(loss.detach()))
    return losses, {k: v.detach().numpy() for k, v in cur.items()}
