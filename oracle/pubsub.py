"""Plain float64 run of the two-party publisher/subscriber training loop.

Test infrastructure only (see ``oracle/__init__.py``).

The loop follows the phases of the paper's training framework (Algorithm 1,
Appendix) on a deterministic tick schedule (``oracle/schedule.py``):

1. publisher phase, passive party B: each replica (worker) takes its rows of
   batch group t, computes z = f_B(x_B) with B's current parameters,
   optionally clips each row and adds Gaussian noise (GDP protocol), and
   publishes the result to the embedding channel of group t;
2. subscriber phase, active party A, group u = t - s: each replica fetches
   its rows of the published embedding, computes z_A = f_A(x_A), the top
   model on [z_A | z_B] and the loss of Eq. (1) (the mean squared error for
   a regression workload), the gradients of A's and
   the top's parameters and the per-row gradient with respect to the
   published embedding, which (optionally clipped and noised) it publishes
   to the gradient channel of group u;
3. backward phase, party B: fetches the gradient of group u and
   back-propagates it through f_B *at the parameters group u's forward used*
   (the delayed parameter of Assumption 4 / the Theorem's update rule),
   then updates B's current parameters with SGD (Eq. 2);
4. per party, the parameter server averages the replicas' gradients with
   row weights (sum over all rows of the tick divided by their number) and
   makes one SGD step per tick (Eq. 2).  A's and the top's parameters are
   always current (delay 0).

Readings of points the paper leaves open are listed where they are used.
Precision: ``precision='f64'`` computes everything in float64.  ``'bf16'`` and
``'f32'`` additionally round to that storage type at the points named in
``ROUNDING_POINTS`` and keep float32 master parameters; the arithmetic in
between stays float64.  The points are where the values a later product or
the other party reads are stored:

  input         a bottom model's input row (dense features and the looked-up
                embedding rows);
  weight        the weight operand of every bottom and hidden top layer
                (the float32 master, rounded); the logit layer reads its
                float32 master weight unrounded;
  act.bottom    every bottom layer's output;
  act.top       every hidden top layer's output;
  delta.bottom  the gradient at the pre-activation of bottom layers below the
                cut layer;
  delta.top     the gradient at the pre-activation of hidden top layers;
  delta.cut_a   the gradient at A's cut-layer pre-activation;
  delta.cut_b   the gradient at B's cut-layer pre-activation (after the clip
                Jacobian);
  msg.emb       the published embedding when it is clipped or noised (else
                the cut layer's stored output is the message);
  msg.grad      the returned gradient message;
  master        the float32 master parameters after every update.

Deltas are gradients of the *sum* of the per-row losses of a group (the 1/R
of the mean loss is applied in the SGD step), so their rounding does not
depend on the group's size.  ``points`` selects a subset (default: all).
"""
from __future__ import annotations

import numpy as np

from . import layers as L
from .philox import gaussian, TAG_EMB, TAG_GRAD
from .rounding import ROUNDERS, round_f32, identity

ROUNDING_POINTS = ("input", "weight", "act.bottom", "act.top", "delta.bottom", "delta.top",
                   "delta.cut_a", "delta.cut_b", "msg.emb", "msg.grad", "master")


class PubSubOracle:
    """State: float64 master parameters of A, B and the top model; ring of
    s + 1 embedding and gradient slots with headers; B's weight stash and
    activation cache per slot; B's update count (its parameter version)."""

    def __init__(self, w, params: dict, precision: str = "f64", points=None):
        self.w = w
        self.s = int(w.staleness)
        self.prec = precision
        self.rnd = ROUNDERS[precision]
        self.points = frozenset(ROUNDING_POINTS if points is None else points)
        assert self.points <= set(ROUNDING_POINTS), self.points
        self.rnd_master = identity if precision == "f64" or "master" not in self.points else round_f32
        self.p = {k: np.asarray(v, dtype=np.float64).copy() for k, v in params.items()}
        self.nA, self.nB = len(w.A.widths), len(w.B.widths)
        self.nT = len(w.top.widths)
        self.E = [None] * (self.s + 1)      # embedding channel slots
        self.G = [None] * (self.s + 1)      # gradient channel slots
        self.S = [None] * (self.s + 1)      # B's stash: weights + activations
        self.vB = 0                         # B's parameter version
        self.trace = []
        self.noise_std = w.sigma * (w.clip if w.clip > 0 else 1.0)

    # ----------------------------------------------------------- helpers
    def _q(self, point: str, x):
        """Storage rounding at a named point (identity when the point is off
        or the precision is float64)."""
        return self.rnd(x) if point in self.points else identity(x)

    def _weights(self, party: str, n: int):
        """Matrix-product operands: the current master weights rounded to the
        storage type (bf16 copies on the GPU)."""
        return [self._q("weight", self.p[f"{party}.W{l}"]) for l in range(n)]

    def _logit_weight(self):
        """The logit layer's weight row: its float32 master, unrounded."""
        return self.p[f"top.W{self.nT - 1}"][0]

    def _bottom_input(self, party: str, spec, data: dict, rows: np.ndarray):
        xs = []
        ids = None
        if spec.n_cat:
            ids = data["ida" if party == "A" else "idb"][rows]
            xs.append(L.gather_embeddings(self.p[f"{party}.T"], ids, spec.vocab))
        if spec.dense:
            xs.append(data["xa" if party == "A" else "xb"][rows].astype(np.float64))
        x = np.concatenate(xs, axis=1) if len(xs) > 1 else xs[0]
        return self._q("input", x), ids

    def _bottom_forward(self, spec, Wq, bias, x):
        acts = [x]
        a = x
        for l in range(len(Wq)):
            p = L.linear(a, Wq[l], bias[l])
            a = self._q("act.bottom", L.relu(p) if spec.relu[l] else p)
            acts.append(a)
        return acts

    def _bottom_backward(self, spec, Wq, acts, delta_top, ids, party):
        """delta_top: gradient w.r.t. the last layer's pre-activation, per row.
        Returns summed (not averaged) gradients {name: array}."""
        g = {}
        delta = delta_top
        for l in range(len(Wq) - 1, -1, -1):
            g[f"{party}.W{l}"] = delta.T @ acts[l]
            g[f"{party}.b{l}"] = delta.sum(axis=0)
            if l > 0:
                gin = delta @ Wq[l]
                m = L.relu_mask(acts[l]) if spec.relu[l - 1] else 1.0
                delta = self._q("delta.bottom", gin * m)
            elif spec.n_cat:
                gx = delta @ Wq[0]
                ne = spec.n_cat * spec.emb_dim
                g[f"{party}.T"] = L.embedding_grad(gx[:, :ne], ids, spec.vocab,
                                                   self.p[f"{party}.T"].shape)
        return g

    def _sgd(self, grads_sum: dict, n_rows: int):
        """Parameter-server step: row-weighted mean of the replicas' gradient
        sums, then theta <- theta - lr * grad (Eq. 2)."""
        for k, gs in grads_sum.items():
            self.p[k] = self.rnd_master(self.p[k] - self.w.lr * (gs / n_rows))

    @staticmethod
    def _add(acc: dict, g: dict):
        for k, v in g.items():
            acc[k] = acc[k] + v if k in acc else v

    # ------------------------------------------------------------ phases
    def publish(self, g: int, t: int, data: dict, replicas):
        """Publisher phase of batch group g at tick t."""
        w = self.w
        Wq = self._weights("B", self.nB)
        bias = [self.p[f"B.b{l}"].copy() for l in range(self.nB)]
        slot = g % (self.s + 1)
        parts = []
        for start, cnt in replicas:           # one B worker per replica
            rows = np.arange(start, start + cnt)
            x, ids = self._bottom_input("B", w.B, data, rows)
            acts = self._bottom_forward(w.B, Wq, bias, x)
            z = acts[-1]
            if w.clip_emb:
                v, n, c = L.clip_rows(z, w.clip)
            else:
                v, n, c = z, None, None
            if w.noise_emb:
                v = v + self.noise_std * gaussian(w.noise_seed, g, rows, z.shape[1], TAG_EMB)
            zhat = self._q("msg.emb", v) if (w.clip_emb or w.noise_emb) else z
            parts.append(dict(rows=rows, ids=ids, acts=acts, n=n, c=c, zhat=zhat))
        self.S[slot] = dict(group=g, version=self.vB, Wq=Wq, parts=parts)
        self.E[slot] = dict(seq=g, tick=t, version=self.vB,
                            zhat=np.concatenate([q["zhat"] for q in parts]))
        return self.E[slot]

    def active_step(self, u: int, t: int, data: dict, replicas):
        """Subscriber phase of group u at tick t: A's bottom, the top model,
        the loss, A's and the top's update, the gradient message to B."""
        w = self.w
        slot = u % (self.s + 1)
        ent = self.E[slot]
        assert ent is not None and ent["seq"] == u, "embedding of group u not published"
        WqA = self._weights("A", self.nA)
        bA = [self.p[f"A.b{l}"] for l in range(self.nA)]
        WqT = self._weights("top", self.nT - 1)
        bT = [self.p[f"top.b{l}"] for l in range(self.nT - 1)]
        w_out = self._logit_weight()
        b_out = self.p[f"top.b{self.nT - 1}"][0]
        dA = w.A.d_out
        grads = {}
        loss_sum = 0.0
        msgs = []
        off = 0
        for start, cnt in replicas:           # one A worker per replica
            rows = np.arange(start, start + cnt)
            zb = ent["zhat"][off:off + cnt]
            off += cnt
            x, ids = self._bottom_input("A", w.A, data, rows)
            acts = self._bottom_forward(w.A, WqA, bA, x)
            h = [np.concatenate([acts[-1], zb], axis=1)]
            for j in range(self.nT - 1):
                p = L.linear(h[-1], WqT[j], bT[j])
                h.append(self._q("act.top", L.relu(p) if w.top.relu[j] else p))
            logit = h[-1] @ w_out + b_out
            y = data["y"][rows].astype(np.float64)
            if w.loss == "mse":
                loss_sum += L.mse(logit, y).sum()
                dl = L.mse_dpred(logit, y)                 # per row, unscaled
            else:
                loss_sum += L.bce_with_logits(logit, y).sum()
                dl = L.bce_dlogit(logit, y)                # per row, unscaled
            g = {f"top.W{self.nT - 1}": (dl @ h[-1])[None, :],
                 f"top.b{self.nT - 1}": np.array([dl.sum()])}
            gin = dl[:, None] * w_out[None, :]
            for j in range(self.nT - 2, -1, -1):
                m = L.relu_mask(h[j + 1]) if w.top.relu[j] else 1.0
                delta = self._q("delta.top", gin * m)
                g[f"top.W{j}"] = delta.T @ h[j]
                g[f"top.b{j}"] = delta.sum(axis=0)
                gin = delta @ WqT[j]
            gA, GB = gin[:, :dA], gin[:, dA:]
            mA = L.relu_mask(acts[-1]) if w.A.relu[-1] else 1.0
            self._add(g, self._bottom_backward(w.A, WqA, acts, self._q("delta.cut_a", gA * mA), ids, "A"))
            self._add(grads, g)
            # gradient message: per-row gradient w.r.t. the published
            # embedding (no 1/R), optionally clipped and noised
            if w.clip_grad:
                v, _, _ = L.clip_rows(GB, w.clip)
            else:
                v = GB
            if w.noise_grad:
                v = v + self.noise_std * gaussian(w.noise_seed, u, rows, v.shape[1], TAG_GRAD)
            msgs.append(self._q("msg.grad", v))
        R = sum(c for _, c in replicas)
        self._sgd(grads, R)
        self.G[slot] = dict(seq=u, tick=t, version=ent["version"], g=np.concatenate(msgs))
        return loss_sum / R, self.G[slot], grads

    def passive_backward(self, u: int, t: int):
        """Backward phase of group u at tick t on party B."""
        w = self.w
        slot = u % (self.s + 1)
        st, gm = self.S[slot], self.G[slot]
        assert st["group"] == u and gm["seq"] == u
        grads = {}
        off = 0
        R = 0
        for q in st["parts"]:
            cnt = len(q["rows"])
            dz = gm["g"][off:off + cnt]
            off += cnt
            R += cnt
            z = q["acts"][-1]
            if w.clip_emb:
                dz = L.clip_rows_backward(dz, z, q["n"], q["c"], w.clip)
            m = L.relu_mask(z) if w.B.relu[-1] else 1.0
            delta = self._q("delta.cut_b", dz * m)
            self._add(grads, self._bottom_backward(w.B, st["Wq"], q["acts"], delta, q["ids"], "B"))
        self._sgd(grads, R)
        self.vB += 1
        return grads

    # -------------------------------------------------------------- loop
    def tick(self, t: int, data: dict, n_groups: int, group_rows, keep_messages=True,
             keep_grads=False, drop=None):
        """Tick t of the schedule: B publishes group t (t < n_groups); A takes
        group u = t - s and B back-propagates it (0 <= u < n_groups), unless
        ``drop`` ("emb" or "grad", see ``run``) discards group u.  Returns the
        tick's record."""
        s = self.s
        rec = dict(tick=t)
        fwd = bwd = -1
        if t < n_groups:
            fwd = t
            rec["fwd_version"] = self.vB
            ent = self.publish(t, t, data, group_rows(t))
            rec["fwd_slot"] = t % (s + 1)
            if keep_messages:
                rec["zhat"] = ent["zhat"]
            rec["emb_header"] = (ent["seq"], ent["tick"], ent["version"])
        u = t - s
        if 0 <= u < n_groups:
            bwd = u
            rec["bwd_slot"] = u % (s + 1)
            if drop != "emb":
                loss, gm, gA = self.active_step(u, t, data, group_rows(u))
                rec["loss"] = loss
                if keep_messages:
                    rec["gtilde"] = gm["g"]
                rec["grad_header"] = (gm["seq"], gm["tick"], gm["version"])
            gB = self.passive_backward(u, t) if drop is None else {}
            if keep_grads and drop is None:
                rec["grads"] = {**gA, **gB}
        rec["fwd_group"], rec["bwd_group"] = fwd, bwd
        self.trace.append((t, fwd, rec.get("fwd_slot", -1), rec.get("fwd_version", -1),
                           bwd, rec.get("bwd_slot", -1), self.vB if bwd >= 0 else -1))
        return rec

    def run(self, data: dict, n_groups: int, group_rows, snapshot=None,
            keep_messages=True, keep_grads=False, discard=None):
        """Run n_groups batch groups (n_groups + s ticks).

        group_rows(g) -> [(start, count)] per replica.  ``snapshot(t)`` says
        whether to copy the parameters after tick t.  ``discard`` maps a
        group to the channel entry dropped for it (Section 4.1 "System Design": the buffer
        mechanism drops the oldest embedding or gradient of a full channel,
        the waiting deadline a batch whose embedding came too late):
        "emb" -- A never uses the group's embedding, so neither A nor B
        updates on it; "grad" -- A takes its step (and publishes the
        gradient), B drops the gradient and makes no update.  A dropped
        group leaves B's version where it was.  Returns a list of per-tick
        dicts.
        """
        discard = discard or {}
        recs = []
        for t in range(n_groups + self.s):
            rec = self.tick(t, data, n_groups, group_rows, keep_messages, keep_grads,
                            discard.get(t - self.s))
            if snapshot is not None and snapshot(t):
                rec["params"] = {k: v.copy() for k, v in self.p.items()}
            recs.append(rec)
        return recs
