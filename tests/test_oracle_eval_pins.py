"""Pins of the oracle's evaluation (the f(t) of Section 4's curves) and of
its temporal efficiency (Eq. 4) against facts fixed by mathematics and by
independent library routines.

A plausible mistake fails one of them: a wrong log-sum-exp (missing max
shift, wrong label column), argmax tie order, a transposed weight, a
dropped bias or ReLU (evaluation); a left or right Riemann sum instead of
the trapezoid, integrating each run over its own length instead of the
minimal shared time, a wrong cut of the segment that straddles it, a
swapped ratio (temporal efficiency).
"""
import math

import numpy as np
import pytest
import torch

from oracle import agn_oracle as O
from oracle import efficiency as TE


def rand_params(dims, rng, scale=0.7):
    return [(rng.standard_normal((dims[l + 1], dims[l])) * scale,
             rng.standard_normal(dims[l + 1]) * 0.3)
            for l in range(len(dims) - 1)]


def torch_mlp_rows(params, X, y):
    """Per-row cross-entropy and argmax of a ReLU MLP with torch's own
    linear, relu and cross_entropy in float64 (an independent
    implementation of the same model)."""
    h = torch.from_numpy(np.asarray(X, dtype=np.float64))
    for l, (W, b) in enumerate(params):
        h = torch.nn.functional.linear(h, torch.from_numpy(W), torch.from_numpy(b))
        if l < len(params) - 1:
            h = torch.relu(h)
    loss = torch.nn.functional.cross_entropy(h, torch.from_numpy(np.asarray(y, dtype=np.int64)),
                                             reduction="none")
    return loss.numpy(), h.numpy()


# --------------------------------------------------------------------------
# evaluation
# --------------------------------------------------------------------------
@pytest.mark.parametrize("dims", [(6, 4), (5, 7, 3), (4, 6, 5, 3)])
def test_evaluate_matches_torch_cross_entropy(dims):
    rng = np.random.default_rng(11)
    params = rand_params(dims, rng)
    X = rng.standard_normal((37, dims[0]))
    y = rng.integers(0, dims[-1], 37)
    row_loss, pred, logits = O.evaluate(params, X, y, dtype=np.float64)
    ref_loss, ref_logits = torch_mlp_rows(params, X, y)
    np.testing.assert_allclose(logits, ref_logits, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(row_loss, ref_loss, rtol=1e-12, atol=1e-12)
    # continuous random logits: no ties, the maximum is unique
    np.testing.assert_array_equal(pred, ref_logits.argmax(axis=1))


def test_evaluate_zero_model_is_uniform():
    """W = 0, b = 0: every logit is 0, the softmax is uniform, the loss of
    every row is log C and the prediction is class 0 (the lowest index of
    the tied maxima)."""
    dims = (5, 4, 7)
    params = [(np.zeros((dims[l + 1], dims[l])), np.zeros(dims[l + 1])) for l in range(2)]
    rng = np.random.default_rng(3)
    X = rng.standard_normal((20, 5))
    y = rng.integers(0, 7, 20)
    row_loss, pred, _ = O.evaluate(params, X, y, dtype=np.float64)
    np.testing.assert_allclose(row_loss, math.log(7), rtol=0, atol=1e-15)
    np.testing.assert_array_equal(pred, 0)


def test_evaluate_planted_classes_closed_form():
    """X row j = s * e_{c_j}, W = I, b = 0: the logits are s * e_{c_j}, the
    prediction is c_j, and the loss is log(e^s + C - 1) - s when the label
    is c_j, log(e^s + C - 1) otherwise."""
    C, s, N = 6, 2.5, 40
    rng = np.random.default_rng(5)
    c = rng.integers(0, C, N)
    y = np.where(rng.random(N) < 0.6, c, (c + 1 + rng.integers(0, C - 1, N)) % C)
    X = s * np.eye(C)[c]
    params = [(np.eye(C), np.zeros(C))]
    row_loss, pred, _ = O.evaluate(params, X, y, dtype=np.float64)
    lse = math.log(math.exp(s) + C - 1)
    np.testing.assert_allclose(row_loss, np.where(y == c, lse - s, lse), rtol=1e-14, atol=0)
    np.testing.assert_array_equal(pred, c)
    assert int((pred == y).sum()) == int((y == c).sum())


def test_evaluate_ties_pick_lowest_index():
    """Two equal largest logits: the lower class index wins."""
    params = [(np.array([[0.0], [1.0], [1.0], [-1.0]]), np.zeros(4))]
    row_loss, pred, _ = O.evaluate(params, np.array([[2.0], [-3.0]]), np.array([2, 3]),
                                   dtype=np.float64)
    np.testing.assert_array_equal(pred, [1, 3])
    # row 0: logits (0, 2, 2, -2), label 2
    np.testing.assert_allclose(row_loss[0], math.log(1 + 2 * math.e ** 2 + math.e ** -2) - 2,
                               rtol=1e-14)


def test_evaluate_mean_is_the_training_loss():
    """The mean of the per-row losses over a batch is the mini-batch loss
    that the training step reports for the same parameters and rows."""
    dims = (8, 6, 5)
    rng = np.random.default_rng(9)
    params = rand_params(dims, rng)
    params32 = [(W.astype(np.float32), b.astype(np.float32)) for W, b in params]
    X = rng.standard_normal((16, 8)).astype(np.float32)
    y = rng.integers(0, 5, 16)
    row_loss, _, _ = O.evaluate(params32, X, y)
    loss, _ = O.loss_and_grads(params32, X, y, O._Prec(np.float32, False))
    assert abs(float(row_loss.mean()) - loss) <= 1e-12 * max(1.0, abs(loss))


# --------------------------------------------------------------------------
# temporal efficiency (Eq. 4)
# --------------------------------------------------------------------------
def test_te_identical_curves_is_one():
    t = [0, 0.5, 1.7, 3.0]
    f = [0.1, 0.4, 0.8, 0.9]
    assert TE.temporal_efficiency(t, f, t, f) == 1.0


def test_te_linear_curves_exact():
    """The trapezoid rule is exact for lines: f_a = 0.3 t sampled at
    irregular times against the constant f_b = 0.6 gives
    (0.3 m^2 / 2) / (0.6 m) = m / 4 over the shared time m."""
    ta = [0.0, 0.13, 0.9, 1.05, 2.4, 4.0]
    fa = [0.3 * t for t in ta]
    tb = [0.0, 1.1, 3.0]
    fb = [0.6] * 3
    assert TE.temporal_efficiency(ta, fa, tb, fb) == pytest.approx(3.0 / 4, rel=1e-14)
    assert TE.temporal_efficiency(tb, fb, ta, fa) == pytest.approx(4.0 / 3, rel=1e-14)


def test_te_cut_at_the_minimal_shared_time():
    """a: f = t on [0, 2]; b: f = 1 on [0, 1].  m = 1 cuts a's only
    segment in its middle: int_0^1 t dt = 1/2, so E(a, b) = 1/2; values of
    a after m change nothing."""
    assert TE.temporal_efficiency([0, 2], [0, 2], [0, 1], [1, 1]) == pytest.approx(0.5, rel=1e-15)
    assert TE.temporal_efficiency([0, 2, 9], [0, 2, -50], [0, 1], [1, 1]) == pytest.approx(0.5, rel=1e-15)


def test_te_quadratic_within_trapezoid_bound():
    """f_a = t^2 sampled every h on [0, m], f_b = 1: the trapezoid area
    exceeds m^3 / 3 by exactly m h^2 / 6 (the error term (m h^2 / 12) f'')."""
    m, k = 2.0, 50
    h = m / k
    t = [i * h for i in range(k + 1)]
    e = TE.temporal_efficiency(t, [v * v for v in t], [0, m], [1, 1])
    assert e * m == pytest.approx(m ** 3 / 3 + m * h * h / 6, rel=1e-12)


def test_te_reciprocal_and_scale_invariant():
    rng = np.random.default_rng(2)
    ta = np.concatenate([[0.0], np.cumsum(rng.random(30) + 0.01)])
    tb = np.concatenate([[0.0], np.cumsum(rng.random(20) + 0.05)])
    fa, fb = rng.random(31), rng.random(21)
    e = TE.temporal_efficiency(ta, fa, tb, fb)
    assert e * TE.temporal_efficiency(tb, fb, ta, fa) == pytest.approx(1.0, rel=1e-13)
    assert TE.temporal_efficiency(ta, 3 * fa, tb, 3 * fb) == pytest.approx(e, rel=1e-13)


@pytest.mark.parametrize("ta,fa", [
    ([0.0], [1.0]),                 # one sample
    ([0.5, 1.0], [1.0, 1.0]),       # does not start at 0
    ([0.0, 1.0, 1.0], [1, 1, 1]),   # times not increasing
    ([0.0, 1.0], [1.0]),            # length mismatch
    ([0.0, 1.0], [1.0, np.nan]),    # not finite
])
def test_te_rejects_bad_curves(ta, fa):
    with pytest.raises(ValueError):
        TE.temporal_efficiency(ta, fa, [0, 1], [1, 1])


def test_te_rejects_zero_reference_area():
    with pytest.raises(ValueError):
        TE.temporal_efficiency([0, 1], [1, 1], [0, 1], [0, 0])
