"""The oracle's pins must catch plausible mistakes: each case plants one in
the oracle (on the CPU, through monkeypatching) and checks that a pin test
then fails."""
import numpy as np
import pytest

import oracle.layers as L
import oracle.pubsub as PS
import test_oracle_step as T


def _fails(fn, *a):
    with pytest.raises(AssertionError):
        fn(*a)


def test_dropped_clip_jacobian_is_caught(monkeypatch):
    monkeypatch.setattr(L, "clip_rows_backward", lambda g, v, n, c, C: g)
    _fails(T.test_finite_differences_whole_step, "bce")


def test_wrong_sign_in_dlogit_is_caught(monkeypatch):
    monkeypatch.setattr(L, "bce_dlogit", lambda l, y: y - L.sigmoid(l))
    _fails(T.test_closed_form_logistic_regression)


def test_backward_at_current_weights_is_caught(monkeypatch):
    """Skipping the weight stash (B's backward at its current parameters
    instead of those its forward used)."""
    orig = PS.PubSubOracle.passive_backward

    def current(self, u, t):
        self.S[u % (self.s + 1)]["Wq"] = self._weights("B", self.nB)
        return orig(self, u, t)
    monkeypatch.setattr(PS.PubSubOracle, "passive_backward", current)
    _fails(T.test_equals_history_formulation, 2, 2, "bce")


def test_swapped_embedding_fields_is_caught(monkeypatch):
    orig = L.embedding_grad
    monkeypatch.setattr(L, "embedding_grad",
                        lambda g, ids, vocab, shape: orig(g, ids[:, ::-1], vocab, shape))
    _fails(T.test_finite_differences_whole_step, "bce")


def test_noise_on_wrong_tag_is_caught(monkeypatch):
    orig = PS.gaussian
    monkeypatch.setattr(PS, "gaussian", lambda seed, step, rows, n, tag: orig(seed, step, rows, n, 0))
    _fails(T.test_equals_history_formulation, 1, 1, "bce")


def test_mean_instead_of_row_weighted_mean_is_caught(monkeypatch):
    """Averaging replica gradients without row weights differs when the
    last group of an epoch is short."""
    orig = PS.PubSubOracle._sgd

    def unweighted(self, grads_sum, n_rows):
        return orig(self, grads_sum, self.w.batch * self.w.replicas)
    monkeypatch.setattr(PS.PubSubOracle, "_sgd", unweighted)
    _fails(T.test_equals_history_formulation, 1, 1, "bce")


def test_squared_error_without_its_factor_two_is_caught(monkeypatch):
    monkeypatch.setattr(L, "mse_dpred", lambda p, y: p - y)
    _fails(T.test_closed_form_linear_regression)


def test_regression_trained_on_bce_is_caught(monkeypatch):
    """The regression head taking the BCE branch (the loss flag ignored)."""
    monkeypatch.setattr(L, "mse", L.bce_with_logits)
    monkeypatch.setattr(L, "mse_dpred", L.bce_dlogit)
    _fails(T.test_equals_history_formulation, 2, 2, "mse")
