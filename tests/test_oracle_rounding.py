"""Pins for the oracle's storage-rounding (precision emulation) modes.

The bf16 workloads are compared on the GPU with the oracle in its bf16 mode,
which rounds to bfloat16 at the named points of ``oracle.ROUNDING_POINTS``
(inputs, weight operands, layer outputs, pre-activation deltas, messages)
and keeps float32 masters.  Those points are pinned here against the
independently written autograd formulation (tests/torch_reference.py), which
places the same points in its autograd graph and rounds with its own
bit-pattern rounding:

* all points together, and every point alone, agree to float64 rounding;
* dropping any one point from the oracle (or rounding the logit layer's
  weight, which stays float32) breaks the agreement by orders of magnitude
  more than the bound, so each mutation fails the pin;
* the f32 mode agrees in the same way.

The case is small enough to run in a second and has what makes every point
matter: embedding tables on both parties (their looked-up rows are not
bf16-exact), two layers per bottom, two hidden top layers, clip and noise on
both messages, staleness 2 and two replicas with a short last group.
"""
import numpy as np
import pytest
import torch

import vfl_synth as S
from vfl_synth.workloads import Workload, PartySpec, TopSpec
from oracle import PubSubOracle, ROUNDING_POINTS
from oracle.rounding import round_bf16
import oracle.pubsub as PS
from torch_reference import run_history, bf16_bits, f32_cast

TOL_THETA = 1e-10      # relative, on parameters
TOL_DELTA = 1e-8       # relative, on parameter changes theta_t - theta_0
TOL_LOSS = 1e-12


def _case(dtype="bf16"):
    return Workload(name="rounding", n_rows=12 * 5 - 4, dtype=dtype,
                    A=PartySpec(dense=3, n_cat=2, vocab=7, emb_dim=4, widths=[6, 8]),
                    B=PartySpec(dense=5, n_cat=1, vocab=5, emb_dim=4, widths=[7, 4]),
                    top=TopSpec(widths=[6, 5, 1]), batch=6, staleness=2, replicas=2, lr=0.5,
                    clip=0.7, sigma=0.3, clip_emb=True, clip_grad=True, noise_emb=True,
                    noise_grad=True, labels="bernoulli", label_p=0.5, zipf_a=0.8,
                    data_seed=31, init_seed=32, noise_seed=33)


N_GROUPS = 6           # wraps the 5-group epoch (its last group is short)


def _relerr(a, b):
    return np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300)


def _compare(oracle_points, torch_points, precision="bf16", rnd=bf16_bits):
    w = _case()
    d = S.generate(w)
    p = S.init_params(w)
    rows_of = lambda g: S.group_rows(w, g)
    o = PubSubOracle(w, p, precision, points=oracle_points)
    recs = o.run(d, N_GROUPS, rows_of)
    losses, final = run_history(w, p, d, N_GROUPS, rows_of, rnd=rnd, points=torch_points)
    got = [r["loss"] for r in recs if "loss" in r]
    np.testing.assert_allclose(got, losses, rtol=TOL_LOSS)
    for key, v in final.items():
        assert _relerr(o.p[key], v) < TOL_THETA, key
        d0 = p[key].astype(np.float64)
        assert _relerr(o.p[key] - d0, v - d0) < TOL_DELTA, key
    return o, recs


def test_torch_bit_rounding_is_round_to_nearest_even():
    """The torch formulation's rounding: brute-force nearest bfloat16 value
    (ties to the even significand), on random values and on exact ties."""
    rng = np.random.default_rng(5)
    x = rng.standard_normal(4000) * np.exp2(rng.integers(-20, 20, 4000))
    m, e = np.frexp(x)
    ties = np.ldexp(np.floor(m * 256) / 256 + 1 / 512, e)      # midway between neighbours
    for v in np.concatenate([x, ties, -ties]):
        got = float(bf16_bits(torch.tensor([v]))[0])
        mm, ee = np.frexp(v)
        lo = np.ldexp(np.floor(mm * 256) / 256, ee)
        hi = np.ldexp(np.floor(mm * 256) / 256 + 1 / 256, ee)
        if abs(v - lo) != abs(hi - v):
            want = lo if abs(v - lo) < abs(hi - v) else hi
        else:
            want = lo if int(np.floor(mm * 256)) % 2 == 0 else hi
        assert got == want, (v, got, want)


def test_bf16_emulation_equals_history_formulation():
    o, recs = _compare(None, ROUNDING_POINTS)
    for r in recs:
        for key in ("zhat", "gtilde"):
            if key in r:
                assert np.array_equal(round_bf16(r[key]), r[key])


@pytest.mark.parametrize("point", ROUNDING_POINTS)
def test_each_rounding_point_alone(point):
    _compare({point}, {point})


@pytest.mark.parametrize("point", ROUNDING_POINTS)
def test_dropped_rounding_point_is_caught(point):
    """The oracle with one point left out against the formulation with all
    of them: the pin must fail."""
    with pytest.raises(AssertionError):
        _compare(set(ROUNDING_POINTS) - {point}, ROUNDING_POINTS)


def test_bf16_logit_weight_is_caught(monkeypatch):
    """The logit layer reads its float32 master weight; an oracle that
    rounds it to bfloat16 must fail the pin."""
    monkeypatch.setattr(PS.PubSubOracle, "_logit_weight",
                        lambda self: self.rnd(self.p[f"top.W{self.nT - 1}"][0]))
    with pytest.raises(AssertionError):
        _compare(None, ROUNDING_POINTS)


def test_f32_emulation_equals_history_formulation():
    _compare(None, ROUNDING_POINTS, precision="f32", rnd=f32_cast)


def test_emulation_points_change_the_result():
    """Each point moves the result well above the pin's bound (so the pins
    above are not vacuous): the bf16 run with one point on differs from the
    float64 run."""
    w = _case()
    d = S.generate(w)
    p = S.init_params(w)
    rows_of = lambda g: S.group_rows(w, g)
    ref = PubSubOracle(w, p, "f64")
    ref.run(d, N_GROUPS, rows_of, keep_messages=False)
    for point in ROUNDING_POINTS:
        o = PubSubOracle(w, p, "bf16", points={point})
        o.run(d, N_GROUPS, rows_of, keep_messages=False)
        worst = max(_relerr(o.p[k] - p[k].astype(np.float64), ref.p[k] - p[k].astype(np.float64))
                    for k in p)
        assert worst > 100 * TOL_DELTA, (point, worst)
