"""Pins for the loss derivatives, the prediction update and the boosting loop (Section 2, eq. 2).

Expected values come from the losses themselves, not from the derivative
formulas the oracle implements:
- gradients and hessian diagonals equal central finite differences of the
  loss (softmax cross-entropy, sigmoid binary cross-entropy);
- softmax gradients sum to zero over the outputs of a row;
- the update is checked on a hand example;
- Newton boosting with lambda > 0 and a small learning rate lowers the
  training loss at every step.
A mutation check plants plausible mistakes and shows the pins catch each.
"""
import math

import numpy as np
import pytest

import oracle
from oracle import boost


def _fd_grad_hess(loss_fn, F, target, eps=1e-4):
    """Central differences of the per-row loss in every output: (gradient, hessian diagonal)."""
    n, d = F.shape
    g = np.zeros((n, d))
    h = np.zeros((n, d))
    l0 = loss_fn(F, target)
    for j in range(d):
        Fp, Fm = F.copy(), F.copy()
        Fp[:, j] += eps
        Fm[:, j] -= eps
        lp, lm = loss_fn(Fp, target), loss_fn(Fm, target)
        g[:, j] = (lp - lm) / (2 * eps)
        h[:, j] = (lp - 2 * l0 + lm) / (eps * eps)
    return g, h


def test_losses_hand_values():
    """Hand values of the two cross-entropies (Section 4 uses them).

    Softmax: equal scores over d classes give p = 1/d, so the loss is log d;
    scores (log 3, 0) give p = (3/4, 1/4), so label 1 costs -log(1/4) = log 4
    and label 0 costs log(4/3).  Sigmoid: a = 0 gives s = 1/2 (log 2 per
    output, whatever the target); a = log 3 gives s = 3/4, so target 1 costs
    log(4/3) and target 0 costs log 4.
    """
    F = np.zeros((1, 4))
    F2 = np.array([[0.0, 0.0], [math.log(3.0), 0.0], [math.log(3.0), 0.0]])
    got = oracle.boost.softmax_ce_loss(F2, np.array([0, 1, 0]))
    assert got == pytest.approx([math.log(2.0), math.log(4.0), math.log(4.0 / 3.0)], rel=1e-14)
    assert oracle.boost.softmax_ce_loss(F[:1], np.array([2]))[0] == pytest.approx(math.log(4.0), rel=1e-14)
    Fs = np.array([[0.0, 0.0], [math.log(3.0), math.log(3.0)]])
    Ys = np.array([[1, 0], [1, 0]], dtype=np.uint8)
    got = oracle.boost.sigmoid_bce_loss(Fs, Ys)
    assert got == pytest.approx([2 * math.log(2.0), math.log(4.0 / 3.0) + math.log(4.0)], rel=1e-14)


def test_softmax_derivatives_match_finite_differences():
    rng = np.random.default_rng(1)
    F = rng.standard_normal((50, 6)) * 2.0
    y = rng.integers(0, 6, 50)
    g, h = boost.softmax_ce_derivatives(F, y)
    g_fd, h_fd = _fd_grad_hess(boost.softmax_ce_loss, F, y)
    assert np.allclose(g, g_fd, atol=1e-8)
    assert np.allclose(h, h_fd, atol=1e-5)
    assert np.allclose(g.sum(axis=1), 0.0, atol=1e-15)
    assert np.all((h >= 0) & (h <= 0.25))


def test_sigmoid_derivatives_match_finite_differences():
    rng = np.random.default_rng(2)
    F = rng.standard_normal((40, 5)) * 3.0
    Y = (rng.random((40, 5)) < 0.3).astype(np.uint8)
    g, h = boost.sigmoid_bce_derivatives(F, Y)
    g_fd, h_fd = _fd_grad_hess(boost.sigmoid_bce_loss, F, Y)
    assert np.allclose(g, g_fd, atol=1e-8)
    assert np.allclose(h, h_fd, atol=1e-5)


def test_gradient_pass_outputs():
    rng = np.random.default_rng(3)
    F = rng.standard_normal((30, 4)).astype(np.float32)
    Y = (rng.random((30, 4)) < 0.5).astype(np.uint8)
    G, Hd, h_row, n2 = boost.gradients("sigmoid", F, Y)
    assert G.dtype == np.float32 and Hd.dtype == np.float32
    assert np.allclose(h_row, Hd.astype(np.float64).mean(axis=1), rtol=1e-6)
    assert np.array_equal(n2, oracle.column_norms2(G))
    with pytest.raises(ValueError):
        boost.gradients("hinge", F, Y)


def test_update_hand_example():
    F = np.array([[1.0, 0.0], [0.5, 0.5], [0.0, -1.0]], dtype=np.float32)
    row_idx = np.array([2, 0, 1], dtype=np.int32)   # leaf 0 = {2}, leaf 1 = {0, 1}
    leaf_off = np.array([0, 1, 3], dtype=np.int32)
    V = np.array([[4.0, -2.0], [1.0, 0.5]])
    got = boost.update_predictions(F, row_idx, leaf_off, V, 0.5)
    want = np.array([[1.5, 0.25], [1.0, 0.75], [2.0, -2.0]], dtype=np.float32)
    assert np.array_equal(got, want)
    assert np.array_equal(boost.update_predictions(F, row_idx, leaf_off, V, 0.0), F)


def _problem(loss, n=600, m=4, d=4, seed=5):
    rng = np.random.default_rng(seed)
    bins = rng.integers(0, 16, (n, m), dtype=np.uint8)
    if loss == "softmax":
        target = (bins[:, 0] // 4 + (bins[:, 1] > 9)) % d      # labels that the features explain
    else:
        target = np.stack([(bins[:, j % m] > 7 + j) for j in range(d)], axis=1).astype(np.uint8)
    return bins, target


@pytest.mark.parametrize("loss,kind,k", [("softmax", "identity", 4), ("softmax", "top_outputs", 2),
                                         ("sigmoid", "identity", 4)])
def test_boosting_lowers_the_training_loss(loss, kind, k):
    bins, target = _problem(loss)
    loss_fn = boost.softmax_ce_loss if loss == "softmax" else boost.sigmoid_bce_loss
    F = np.zeros((bins.shape[0], 4), dtype=np.float32)
    prev = loss_fn(F, target).mean()
    for _ in range(4):
        F, _ = boost.boost(bins, 16, F, target, loss, 1, 0.3, kind, k, 3, 1.0)
        cur = loss_fn(F, target).mean()
        assert cur < prev
        prev = cur


def test_boost_pins_catch_planted_mistakes(monkeypatch):
    rng = np.random.default_rng(7)
    F = rng.standard_normal((30, 5)) * 2.0
    y = rng.integers(0, 5, 30)
    g_fd, h_fd = _fd_grad_hess(boost.softmax_ce_loss, F, y)
    g, h = boost.softmax_ce_derivatives(F, y)
    planted = {
        "gradient sign": (-g, h),
        "hessian p instead of p(1-p)": (g, g + np.eye(5)[y]),
        "label column not subtracted": (g + np.eye(5)[y], h),
    }
    for name, (gb, hb) in planted.items():
        assert not (np.allclose(gb, g_fd, atol=1e-8) and np.allclose(hb, h_fd, atol=1e-5)), name
    # an update in the wrong direction raises the loss
    bins, target = _problem("softmax")
    good = boost.update_predictions
    monkeypatch.setattr(boost, "update_predictions", lambda F, r, o, V, lr: good(F, r, o, V, -lr))
    F0 = np.zeros((bins.shape[0], 4), dtype=np.float32)
    F1, _ = boost.boost(bins, 16, F0, target, "softmax", 1, 0.3, "identity", 4, 3, 1.0)
    assert boost.softmax_ce_loss(F1, target).mean() > boost.softmax_ce_loss(F0, target).mean()
