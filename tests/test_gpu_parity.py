"""GPU parity: the HIP path (through the C ABI) against the oracle on the same
seeded inputs, for the five workloads at their real tick shapes, their
full-size ragged epoch tails, odd shapes and the schedule's integer state.
Metrics and tolerances: tests/gpu_harness.py."""
import numpy as np
import pytest

import vfl_synth as S
from vfl_synth.workloads import Workload, PartySpec, TopSpec
from oracle import PubSubOracle
from oracle.philox import philox4x32_10
import gpu_harness as H

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("needs an MI355X")


def _prec(w):
    return "bf16" if w.dtype == "bf16" else "f64"


def _tol(w):
    return H.BF16_THETA_EMU if w.dtype == "bf16" else H.F32_TOL


def _dtol(w):
    return H.BF16_DELTA_TOL if w.dtype == "bf16" else H.F32_TOL


def _check_ints(run, o, recs):
    assert run.mismatches == 0 and run.bad_ids == 0
    assert run.trace == [tuple(r) for r in o.trace]
    for r in recs:
        if "emb_header" in r:
            assert run.msgs[("e", r["fwd_group"])][1] == r["emb_header"]
        if "grad_header" in r:
            assert run.msgs[("g", r["bwd_group"])][1] == r["grad_header"]


def _check_messages(run, recs, w):
    if w.dtype == "bf16":
        tol_elem, frac, l2 = H.BF16_MSG_ELEM, H.BF16_MSG_FRAC, H.BF16_MSG_L2
    else:
        tol_elem, frac, l2 = 1e-4, 2e-3, 1e-4
    for r in recs:
        for key, tag, grp in (("zhat", "e", "fwd_group"), ("gtilde", "g", "bwd_group")):
            if key in r:
                ok, f, e = H.message_ok(run.msgs[(tag, r[grp])][0], r[key], tol_elem, frac, l2)
                H.record(f"{key} bad frac", f, frac, f"t{r['tick']}")
                H.record(f"{key} rel L2", e, l2, f"t{r['tick']}")
                assert ok, (key, r["tick"], f, e)


def _check_losses(run, recs, w):
    tol = H.BF16_LOSS if w.dtype == "bf16" else 1e-4
    ref = np.array([r["loss"] for r in recs if "loss" in r])
    err = np.max(np.abs(run.losses - ref) / np.abs(ref)) if ref.size else 0.0
    H.record("loss rel", err, tol)
    np.testing.assert_allclose(run.losses, ref, rtol=tol)


def _check_params(run, recs, w, per_tick, f64_recs=None, stated=False):
    """theta and delta-theta against the oracle run ``recs`` (the bf16
    emulation for bf16 workloads, float64 otherwise) at every snapshot
    (per_tick) or the last; for bf16 workloads also theta against the plain
    float64 oracle run ``f64_recs``, held to the stated 2e-2 on the named
    workloads (``stated``: their learning rate and shapes) and recorded
    elsewhere (at lr 0.5 the bf16 effect on theta itself reaches 2e-2)."""
    tol, dtol = _tol(w), _dtol(w)
    s = w.staleness
    ticks = sorted(run.snaps) if per_tick else [max(run.snaps)]
    by_tick = {r["tick"]: r for r in recs}
    by_tick64 = {r["tick"]: r for r in f64_recs} if f64_recs else {}
    for t in ticks:
        ref = by_tick[t]["params"]
        n_upd = max(0, t - s + 1)
        for k, v in ref.items():
            g = run.snaps[t][k]
            p0 = run.p0[k].astype(np.float64)
            e = H.rel_inf(g, v)
            H.record("theta rel", e, tol, f"{k} t{t}")
            assert e <= tol, (k, t, e)
            ok, err, bound = H.delta_ok(g, v, p0, dtol, n_upd)
            H.record("dtheta err/bound", err / bound if bound > 0 else 0.0, 1.0, f"{k} t{t}")
            d_ref = np.max(np.abs(v - p0))
            if d_ref > 0:
                H.record("dtheta rel", err / d_ref, dtol,
                         f"{k} t{t} max|dtheta| {d_ref:.2e} ulp {H.ulp32(v):.1e} x {n_upd}")
            assert ok, (k, t, err, bound)
            if t in by_tick64 and "params" in by_tick64[t]:
                v64 = by_tick64[t]["params"][k]
                e64 = H.rel_inf(g, v64)
                if stated:
                    H.record("theta rel vs f64", e64, H.BF16_TOL, f"{k} t{t}")
                    assert e64 <= H.BF16_TOL, (k, t, e64)
                else:
                    H.record("theta rel vs f64 (info)", e64, float("inf"), f"{k} t{t}")
                d64 = np.max(np.abs(v64 - p0))
                if d64 > 0:
                    H.record("dtheta rel vs f64 (info)", np.max(np.abs((g - p0) - (v64 - p0))) / d64,
                             float("inf"), f"{k} t{t}")
                    H.record("emulation dtheta gap to f64 (info)",
                             np.max(np.abs((v - p0) - (v64 - p0))) / d64, float("inf"), f"{k} t{t}")


def _full_check(run, w, per_tick=True, f64=True):
    """Integers, losses, messages and parameters of a run against the
    oracle at the workload's precision (and, for bf16, theta against the
    float64 oracle: the stated bound on the named workloads)."""
    o, recs = run.oracle(_prec(w))
    _check_ints(run, o, recs)
    _check_losses(run, recs, w)
    _check_messages(run, recs, w)
    f64_recs = None
    if w.dtype == "bf16" and f64:
        _, f64_recs = run.oracle("f64", messages=False)
    _check_params(run, recs, w, per_tick, f64_recs, stated=w.name in S.ALL)
    return o, recs


# ------------------------------------------------------------- Philox words
@pytest.mark.parametrize("step,tag,row0", [(0, 0, 0), (305, 1, 9_990_000), (7, 0, 123_456)])
def test_philox_words_bit_exact(step, tag, row0):
    import torch
    from paper_2510_12494_amd import vfl as V
    rows, groups, seed = 4096, 32, 0x5EED0005
    out = torch.zeros(rows * groups * 4, dtype=torch.int32, device="cuda")
    V.vfl_philox(seed, step, tag, row0, rows, groups, out.data_ptr(), 0)
    torch.cuda.synchronize()
    got = out.cpu().numpy().view(np.uint32).reshape(rows, groups, 4)
    r = (np.arange(rows, dtype=np.uint64) + row0)[:, None]
    q = np.arange(groups, dtype=np.uint64)[None, :]
    ref = philox4x32_10(step, r, q, tag, seed & 0xFFFFFFFF, seed >> 32)
    for i in range(4):
        assert np.array_equal(got[:, :, i], ref[i])


# ------------------------------------------------------------ the workloads
def test_tiny_sync_full_epoch():
    """4096 rows, 16 ticks, fp32, s=0: every tick against the float64 oracle."""
    w = S.get("tiny_sync")
    run = H.Run(w, w.n_rows, 16)
    _full_check(run, w)


def test_dense_tabular_100_ticks():
    """bf16, s=2: 100 batch groups (102 ticks) against the bf16-emulating
    oracle, and theta against the float64 oracle within 2e-2."""
    w = S.get("dense_tabular")
    n = 100 * w.rows_per_tick
    last = 100 + w.staleness - 1
    snap = lambda t: t in (10, 50, last)
    run = H.Run(w, n, 100, snap=snap)
    _full_check(run, w)


def test_ctr_per_tick():
    """fp32 with 13 + 13 embedding fields (Zipf ids), s=2: every tick."""
    w = S.get("ctr")
    n = 6 * w.rows_per_tick
    run = H.Run(w, n, 6)
    _full_check(run, w)


@pytest.mark.parametrize("name", ["hetero", "private"])
def test_large_tick_workloads(name):
    """hetero (s=4, k=4) and private (s=2, k=2, clip + noise on both
    messages) at R = 32768 rows per tick."""
    w = S.get(name)
    n = 6 * w.rows_per_tick
    run = H.Run(w, n, 6)
    _full_check(run, w)


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name,batch", [("hetero", 1024), ("private", 4096)])
def test_large_workloads_100_groups(name, batch):
    """hetero and private over 100 batch groups with every width, the
    staleness, replica count, clip and noise of the workload and a smaller
    replica batch (R = 4096 and 8192 rows per tick), so that the float64
    oracle finishes in about a minute: parameters at groups 10, 50 and 100
    against the bf16 emulation, and theta against the float64 oracle within
    2e-2."""
    w = S.get(name).replace(batch=batch)
    n = 100 * w.rows_per_tick
    last = 100 + w.staleness - 1
    snap = lambda t: t in (10, 50, last)
    run = H.Run(w, n, 100, snap=snap)
    _full_check(run, w)


def test_regression_ten_layer_bottoms():
    """The regression workload (ten-layer bottoms, squared-error head, bf16,
    s=2, k=2) at its real tick shape over 6 groups."""
    w = S.get("regression")
    run = H.Run(w, 6 * w.rows_per_tick, 6)
    _full_check(run, w)


@pytest.mark.timeout(900)
def test_regression_100_groups():
    """The regression workload over 100 batch groups at a smaller replica
    batch (R = 2048 rows per tick): parameters at groups 10, 50 and 100
    against the bf16 emulation, and theta against the float64 oracle."""
    w = S.get("regression").replace(batch=1024)
    n = 100 * w.rows_per_tick
    last = 100 + w.staleness - 1
    snap = lambda t: t in (10, 50, last)
    run = H.Run(w, n, 100, snap=snap)
    _full_check(run, w)


@pytest.mark.parametrize("s,k", [(0, 1), (3, 2)])
def test_ten_layer_odd_widths_f32(s, k):
    """Ten-layer bottoms at odd widths with linear layers among the ReLU
    ones, a two-layer top with the squared-error head, float32: every tick
    against the float64 oracle."""
    relu = [True, False, True, True, True, False, True, True, True, True]
    w = Workload(name="deep", n_rows=7 * 130 + 9, dtype="f32",
                 A=PartySpec(dense=19, widths=[40, 33, 24, 17, 40, 9, 28, 31, 12, 8], relu=relu),
                 B=PartySpec(dense=13, n_cat=2, vocab=23, emb_dim=4,
                             widths=[29, 36, 17, 22, 40, 13, 27, 18, 33, 20], relu=relu[::-1]),
                 top=TopSpec(widths=[21, 11, 1]), batch=130 // k, staleness=s, replicas=k,
                 lr=0.01, labels="regression", loss="mse", data_seed=111, init_seed=112,
                 noise_seed=113)
    n_groups = (w.n_rows + w.rows_per_tick - 1) // w.rows_per_tick
    run = H.Run(w, w.n_rows, n_groups)
    _full_check(run, w)


@pytest.mark.parametrize("name", list(S.ALL))
def test_gradient_probe(name):
    """One update per party at lr = 1, so that every parameter change is far
    above float32 resolution: the change equals -grad, compared at the
    workload's tolerance."""
    w = S.get(name).replace(lr=1.0)
    run = H.Run(w, w.rows_per_tick, 1)
    o, recs = run.oracle(_prec(w))
    _check_ints(run, o, recs)
    dtol = _dtol(w)
    for k, v in o.p.items():
        ok, err, bound = H.delta_ok(run.final[k], v, run.p0[k].astype(np.float64), dtol, 1)
        d_ref = np.max(np.abs(v - run.p0[k]))
        if d_ref > 0:
            H.record("grad rel (lr 1)", err / d_ref, dtol, f"{k} max|grad| {d_ref:.2e}")
        assert ok, (k, err, bound)


@pytest.mark.parametrize("name", list(S.ALL))
def test_full_size_epoch_tail(name):
    """The workload's full dataset; the last two groups of its epoch (the
    last one ragged), so row ids, noise counters and tails are those of the
    full size."""
    w = S.get(name)
    T = w.ticks_per_epoch()
    g0 = T - 2
    run = H.Run(w, w.n_rows, 2, g0=g0)
    if w.n_rows % w.rows_per_tick:
        assert sum(c for _, c in run.rows_of(1)) < w.rows_per_tick
    _full_check(run, w)


# ------------------------------------------------------------- odd shapes
def _odd(dtype, s, k, clip):
    return Workload(name="odd", n_rows=1101, dtype=dtype,
                    A=PartySpec(dense=13, widths=[40, 24]),
                    B=PartySpec(dense=21, n_cat=3, vocab=37, emb_dim=4, widths=[33, 17]),
                    top=TopSpec(widths=[19, 1]), batch=100, staleness=s, replicas=k, lr=0.5,
                    clip=1.0 if clip else 0.0, sigma=0.5 if clip else 0.0, clip_emb=clip,
                    clip_grad=clip, noise_emb=clip, noise_grad=clip, labels="bernoulli",
                    label_p=0.4, zipf_a=1.1, data_seed=77, init_seed=78, noise_seed=79)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("s,k,clip", [(0, 1, False), (1, 3, True), (3, 2, False)])
def test_odd_shapes(dtype, s, k, clip):
    """Widths that are not multiples of any tile, 3 embedding fields with an
    input width not a multiple of 16, row counts not multiples of 64 and an
    epoch whose last group holds a single row (1101 = 11 * 100 + 1)."""
    w = _odd(dtype, s, k, clip)
    n_groups = (w.n_rows + w.rows_per_tick - 1) // w.rows_per_tick
    run = H.Run(w, w.n_rows, n_groups)
    _full_check(run, w)


@pytest.mark.parametrize("zipf_a,vocab,shift,stride", [(30.0, 5, 0, 1), (1.1, 3000, 0, 1), (30.0, 40, 17, 1),
                                                      (1.1, 3000, 0, 1009)])
def test_table_sgd_segments(zipf_a, vocab, shift, stride):
    """Sparse table SGD at its extremes: 10,000 rows per tick (two passes of
    the per-field key collection), and either (zipf_a = 30) every sample of
    a field on one id, below 16 (a hot-id workgroup's sum over all rows) or
    at 17 (one id part: the 32-keys-per-thread sort and a segment spanning
    every staged block of both passes, while most parts stay empty), or a
    spread of ids with repeats across parts and hot ids, also with the Zipf
    ranks scattered over the ids (stride 1009, as hashed ids would be: the
    frequent ids are no longer the low ones the hot-id workgroups take).""" 
    w = Workload(name="tables", n_rows=20000, dtype="f32",
                 A=PartySpec(dense=7, n_cat=2, vocab=vocab, emb_dim=16, widths=[24, 16]),
                 B=PartySpec(dense=0, n_cat=3, vocab=vocab, emb_dim=8, widths=[20, 8]),
                 top=TopSpec(widths=[12, 1]), batch=5000, staleness=1, replicas=2, lr=0.5,
                 labels="bernoulli", label_p=0.4, zipf_a=zipf_a, id_shift=shift, id_stride=stride,
                 data_seed=81, init_seed=82, noise_seed=83)
    run = H.Run(w, w.n_rows, 2)
    o, recs = run.oracle("f64")
    _check_ints(run, o, recs)
    _check_losses(run, recs, w)
    _check_params(run, recs, w, per_tick=True)


def test_out_of_range_ids_are_clamped_and_counted():
    """Categorical ids outside [0, vocab) (negative and past the vocabulary,
    on both parties) are read as the nearest valid id and counted: the run
    equals the oracle on the clamped ids, and vfl_check counts each bad id
    once per forward that takes its row (every row here is in exactly one
    group, read by one forward of each party)."""
    w = Workload(name="badids", n_rows=3000, dtype="f32",
                 A=PartySpec(dense=5, n_cat=2, vocab=40, emb_dim=8, widths=[24, 16]),
                 B=PartySpec(dense=0, n_cat=3, vocab=30, emb_dim=4, widths=[20, 8]),
                 top=TopSpec(widths=[12, 1]), batch=500, staleness=1, replicas=2, lr=0.5,
                 labels="bernoulli", label_p=0.4, data_seed=85, init_seed=86, noise_seed=87)
    d = S.generate(w)
    rng = np.random.default_rng(5)
    bad = 0
    clamped = dict(d)
    for key, V in (("ida", w.A.vocab), ("idb", w.B.vocab)):
        ids = d[key].copy()
        m = rng.random(ids.shape) < 0.02
        n = int(m.sum())
        ids[m] = np.where(rng.random(n) < 0.5, -rng.integers(1, 1000, n), V + rng.integers(0, 1000, n))
        d[key] = ids.astype(np.int32)
        clamped[key] = np.clip(ids, 0, V - 1).astype(np.int32)
        bad += n
    assert bad > 50
    n_groups = w.n_rows // w.rows_per_tick
    run = H.Run(w, w.n_rows, n_groups, data=d, messages=False)
    assert run.mismatches == 0 and run.bad_ids == bad
    o = PubSubOracle(w, run.p0, "f64")
    o.run(clamped, n_groups, run.rows_of, keep_messages=False)
    worst = max(H.rel_inf(run.final[k], v) for k, v in o.p.items())
    H.record("theta rel", worst, H.F32_TOL)
    assert worst <= H.F32_TOL


@pytest.mark.parametrize("widths,s,k,clip", [([520, 40], 1, 2, True), ([600, 264, 24], 2, 1, False)])
def test_wide_first_layer_product(widths, s, k, clip):
    """Party B's first layer at least 512 wide (bf16): layer 1's input
    gradient runs as a layer product over the whole group after the chain;
    odd widths (partial 128-output and 256-row tiles), a ragged last group,
    and with two layers the cut-layer delta itself feeds the product."""
    w = Workload(name="wide", n_rows=1401, dtype="bf16",
                 A=PartySpec(dense=24, widths=[32, 16]), B=PartySpec(dense=33, widths=widths),
                 top=TopSpec(widths=[20, 1]), batch=300, staleness=s, replicas=k, lr=0.5,
                 clip=1.0 if clip else 0.0, sigma=0.5 if clip else 0.0, clip_emb=clip,
                 clip_grad=clip, noise_emb=clip, noise_grad=clip, labels="teacher",
                 data_seed=71, init_seed=72, noise_seed=73)
    n_groups = (w.n_rows + w.rows_per_tick - 1) // w.rows_per_tick
    run = H.Run(w, w.n_rows, n_groups)
    _full_check(run, w)


def _wide_three(din, widths, s, k, clip, lr=0.5):
    return Workload(name="widethree", n_rows=1401, dtype="bf16",
                    A=PartySpec(dense=24, widths=[32, 16]), B=PartySpec(dense=din, widths=widths),
                    top=TopSpec(widths=[20, 1]), batch=300, staleness=s, replicas=k, lr=lr,
                    clip=1.0 if clip else 0.0, sigma=0.5 if clip else 0.0, clip_emb=clip,
                    clip_grad=clip, noise_emb=clip, noise_grad=clip, labels="teacher",
                    data_seed=81, init_seed=82, noise_seed=83)


@pytest.mark.parametrize("din,widths,s,k,clip,params", [
    (200, [256, 128, 32], 2, 1, True, True),
    (129, [256, 256, 64], 0, 1, False, True),
    (640, [384, 384, 96], 1, 2, True, False),
    (500, [1024, 512, 128], 4, 2, False, False),
])
def test_wide_three_layer_bottoms(din, widths, s, k, clip, params):
    """Party B's three-layer bf16 bottoms on dense inputs with a wide first
    layer: input widths 129 and 640, output widths that end in a partial
    pass of the chain's 256 columns (384, 96), hetero's bottom, rows per
    tick not a multiple of the block rows and a ragged last group.

    Integers, losses and both messages against the bf16 emulation; with
    `params` also the parameters at every tick.  The last two shapes are
    held to the forward's own outputs only: at a few hundred rows per tick
    their parameter updates are more sensitive to rounding than the
    per-update bound (the emulation itself, with every value perturbed by
    half a float32 ulp before each bf16 rounding, departs from its
    unperturbed run by 3 to 14 times that bound after a single update);
    hetero's bottom is held to the full checks at 4096 and 32768 rows per
    tick by the named-workload tests."""
    w = _wide_three(din, widths, s, k, clip)
    n_groups = (w.n_rows + w.rows_per_tick - 1) // w.rows_per_tick
    run = H.Run(w, w.n_rows, n_groups)
    if params:
        _full_check(run, w)
        return
    o, recs = run.oracle(_prec(w))
    _check_ints(run, o, recs)
    _check_losses(run, recs, w)
    _check_messages(run, recs, w)


@pytest.mark.parametrize("din,widths,s,k,clip", [(200, [256, 128, 32], 2, 1, True),
                                                 (160, [256, 256, 64], 0, 2, False)])
def test_wide_three_layer_gradient_probe(din, widths, s, k, clip):
    """One update per party at lr = 1 on the three-layer bottoms, so that
    every parameter change is -grad far above float32 resolution: B's
    gradients read the forward's RC copies and ReLU bits of both hidden
    layers.  (The 129-wide input of the test above is avoided here: with
    its data one layer-1 pre-activation lies within float32 rounding of
    zero, and the GPU and the emulation take that ReLU decision
    differently, which moves B.W1's gradient by 2 % of its largest entry;
    both stay equally close to the float64 oracle.)"""
    w = _wide_three(din, widths, s, k, clip, lr=1.0)
    run = H.Run(w, w.rows_per_tick, 1)
    o, recs = run.oracle(_prec(w))
    _check_ints(run, o, recs)
    dtol = _dtol(w)
    for key, v in o.p.items():
        ok, err, bound = H.delta_ok(run.final[key], v, run.p0[key].astype(np.float64), dtol, 1)
        d_ref = np.max(np.abs(v - run.p0[key]))
        if d_ref > 0:
            H.record("grad rel (lr 1)", err / d_ref, dtol, f"{key} max|grad| {d_ref:.2e}")
        assert ok, (key, err, bound)


@pytest.mark.parametrize("din", [500, 129])
def test_dense_row_padding_is_never_read(din):
    """Columns of the dense rows past the input width (the row padding up
    to ld) may hold anything: filled with NaN they leave a run bitwise
    unchanged (the chain kernels load whole 16-byte chunks of the rows and
    zero the elements past the width)."""
    import torch
    from paper_2510_12494_amd.session import Session
    w = Workload(name="padding", n_rows=700, dtype="bf16",
                 A=PartySpec(dense=din, widths=[32, 16]), B=PartySpec(dense=din, widths=[256, 128, 32]),
                 top=TopSpec(widths=[20, 1]), batch=300, staleness=1, replicas=1, lr=0.5,
                 labels="teacher", data_seed=91, init_seed=92, noise_seed=93)
    d = S.generate(w)
    p = S.init_params(w)
    n_groups = (w.n_rows + w.rows_per_tick - 1) // w.rows_per_tick
    shapes = {key: v.shape for key, v in p.items()}
    finals = []
    for nan in (False, True):
        sess = Session(w, d, p, lambda g: S.group_rows(w, g, w.n_rows))
        try:
            if nan:
                for key in ("xa", "xb"):
                    assert sess.data[key].shape[1] > din
                    sess.data[key][:, din:] = float("nan")
                torch.cuda.synchronize()
            for t in range(n_groups + w.staleness):
                sess.step(t, n_groups)
            finals.append(sess.params(shapes))
        finally:
            sess.close()
    for key in shapes:
        assert np.array_equal(finals[0][key], finals[1][key]), key


def test_shared_lds_buffers_deep_top():
    """The active kernel shares LDS between buffers that are never live
    together (its input with the second delta buffer, the last top hidden
    output with the gradient-message staging): two hidden top layers (the
    delta chain then writes the second buffer and reads the first hidden
    layer's mask), clip and noise on both messages, two A layers, and groups
    large enough for 32-row blocks."""
    w = Workload(name="deep_top", n_rows=3 * 8192 + 1000, dtype="bf16",
                 A=PartySpec(dense=40, widths=[72, 32]), B=PartySpec(dense=24, widths=[48, 24]),
                 top=TopSpec(widths=[64, 40, 1]), batch=8192, staleness=1, replicas=1, lr=0.2,
                 clip=1.0, sigma=0.5, clip_emb=True, clip_grad=True, noise_emb=True,
                 noise_grad=True, labels="teacher", data_seed=61, init_seed=62, noise_seed=63)
    n_groups = 4
    run = H.Run(w, w.n_rows, n_groups)
    _full_check(run, w)


@pytest.mark.parametrize("dtype,s,discard", [
    ("bf16", 2, {1: "emb", 3: "grad", 5: "emb_fifo"}),
    ("f32", 1, {0: "grad", 3: "emb", 5: "emb_fifo"}),
])
def test_channel_discards(dtype, s, discard):
    """The buffer and waiting-deadline mechanisms (Section 4.1 "System Design"): groups whose
    embedding is dropped (A gives up on the group, or a full FIFO channel
    drops it before A takes it) and groups whose gradient is dropped (a full
    channel after A's step).  Per-tick parameters, the losses of the groups
    A stepped on and every message against the oracle run with the same
    drops; a dropped group never advances B's version (checked through the
    parameters and the slot headers of later forwards)."""
    tables = dtype == "f32"
    w = Workload(name="drops", n_rows=9 * 600, dtype=dtype,
                 A=PartySpec(dense=24, n_cat=2 if tables else 0, vocab=50, emb_dim=8, widths=[32, 16]),
                 B=PartySpec(dense=16, widths=[24, 16]), top=TopSpec(widths=[20, 1]),
                 batch=300, staleness=s, replicas=2, lr=0.5, clip=1.0, sigma=0.5, clip_emb=True,
                 clip_grad=True, noise_emb=True, noise_grad=True, fifo_discard=True,
                 labels="teacher", data_seed=91, init_seed=92, noise_seed=93)
    n_groups = 9
    run = H.Run(w, w.n_rows, n_groups, discard=discard)
    o, recs = run.oracle(_prec(w))
    assert run.mismatches == 0 and run.bad_ids == 0
    for r in recs:
        if "emb_header" in r:
            assert run.msgs[("e", r["fwd_group"])][1] == r["emb_header"]
        if "grad_header" in r:
            assert run.msgs[("g", r["bwd_group"])][1] == r["grad_header"]
    # the schedule trace: every tick run through vfl_step against the
    # oracle's row of that tick (the version columns shift by the drops)
    manual = {u + s for u, k in discard.items() if k in ("emb_fifo", "grad")}
    got_rows = {r[0]: tuple(r) for r in run.trace}
    assert set(got_rows) == set(range(n_groups + s)) - manual
    for r in o.trace:
        if r[0] in got_rows:
            assert got_rows[r[0]] == tuple(r), (r, got_rows[r[0]])
    stepped = [r["bwd_group"] for r in recs if "loss" in r]
    assert sorted(set(range(n_groups)) - set(stepped)) == sorted(
        u for u, k in discard.items() if k in ("emb", "emb_fifo"))
    ref = np.array([r["loss"] for r in recs if "loss" in r])
    got = np.array([run.losses[u] for u in stepped])
    tol = H.BF16_LOSS if dtype == "bf16" else 1e-4
    H.record("loss rel", np.max(np.abs(got - ref) / np.abs(ref)), tol)
    np.testing.assert_allclose(got, ref, rtol=tol)
    _check_messages(run, recs, w)
    _check_params(run, recs, w, per_tick=True)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_limits_of_the_interface(dtype):
    """The largest staleness (s = 4: five channel slots) and replica count
    (k = 8), B's bottom at the 16-layer limit, A's bottom and the top's
    hidden layers at the 16-problem limit of one weight-gradient launch
    (3 + 13), linear layers mixed with ReLU ones (the masks of the
    input-gradient chains skip them), the largest embedding width (16) and
    a ragged last group of 3 rows."""
    w = Workload(name="limits", n_rows=9 * 400 + 3, dtype=dtype,
                 A=PartySpec(dense=11, n_cat=2, vocab=29, emb_dim=16, widths=[36, 20, 16],
                             relu=[True, False, True]),
                 B=PartySpec(dense=9, widths=[24, 18, 30, 12, 26, 16, 20, 10, 14, 22, 9, 17, 25, 11, 19, 10],
                             relu=[True, True, False, True, True, False, True, True] * 2),
                 top=TopSpec(widths=[28, 14, 22, 9, 17, 12, 20, 15, 11, 18, 13, 16, 10, 1],
                             relu=[True, False, True, True, False, True, True, False, True, True,
                                   True, False, True]),
                 batch=50, staleness=4, replicas=8, lr=0.3, clip=1.0, sigma=0.5,
                 clip_emb=True, clip_grad=True, noise_emb=True, noise_grad=True,
                 labels="bernoulli", label_p=0.45, data_seed=101, init_seed=102, noise_seed=103)
    n_groups = (w.n_rows + w.rows_per_tick - 1) // w.rows_per_tick
    run = H.Run(w, w.n_rows, n_groups)
    _full_check(run, w)
