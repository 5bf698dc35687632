"""Pins of the exit-head training oracle (Sec. IV-A, Eq. (22), (23)):
a first descent step worked by hand, the loss gradient against finite
differences, separable data, and argmax ties."""
import math

import numpy as np
import pytest

from oracle import exit_head as X


def test_argmax_and_ties():
    W = np.array([[1.0, 0.0], [0.0, 1.0], [1.0, 0.0]])   # rows 0 and 2 equal
    H = np.array([[2.0, 1.0], [1.0, 3.0], [1.0, 1.0]])
    idx, margin = X.head_argmax(W, H)
    assert idx.tolist() == [0, 1, 0]                  # tie 0 / 2 -> 0
    assert margin.tolist() == [0.0, 2.0, 0.0]         # a tie has no margin
    assert X.consistency_labels([0, 1, 2], [0, 2, 2]).tolist() == [1, 0, 1]


def test_first_step_by_hand():
    # H = [[1, 0], [0, 2]], labels (1, 0), start at zero: xi = 1/2 for both,
    # residuals (-1/2, 1/2); gradient of w = ((-1/2)(1, 0) + (1/2)(0, 2)) / 2
    # = (-1/4, 1/2), of c = 0; loss ln 2.  With lr 0.4: w = (0.1, -0.2).
    w, c, losses = X.train_exit_head([[1.0, 0.0], [0.0, 2.0]], [1, 0], 1, 0.4)
    assert w.tolist() == pytest.approx([0.1, -0.2], abs=1e-15) and c == 0.0
    assert losses[0] == pytest.approx(math.log(2.0), abs=1e-15)


def test_step_is_the_loss_gradient():
    rng = np.random.default_rng(2)
    Q, d = 40, 5
    H = rng.normal(size=(Q, d))
    y = (rng.uniform(size=Q) < 0.4).astype(float)
    w0, c0 = rng.normal(size=d) * 0.3, 0.2
    lr = 1e-3
    w1, c1, _ = X.train_exit_head(H, y, 1, lr, w0, c0)
    g = -(w1 - w0) / lr
    gc = -(c1 - c0) / lr
    eps = 1e-6
    for i in range(d):
        e = np.zeros(d)
        e[i] = eps
        num = (X.bce_loss(H @ (w0 + e) + c0, y) - X.bce_loss(H @ (w0 - e) + c0, y)) / (2 * eps)
        assert g[i] == pytest.approx(num, rel=1e-6, abs=1e-9)
    num = (X.bce_loss(H @ w0 + c0 + eps, y) - X.bce_loss(H @ w0 + c0 - eps, y)) / (2 * eps)
    assert gc == pytest.approx(num, rel=1e-6, abs=1e-9)


def test_separable_data_is_learned():
    rng = np.random.default_rng(4)
    H = rng.normal(size=(200, 3))
    y = (H @ np.array([1.5, -2.0, 0.5]) + 0.3 > 0).astype(float)
    w, c, losses = X.train_exit_head(H, y, 400, 0.5)
    assert np.all(np.diff(losses) <= 1e-12)            # full-batch descent, small step
    assert losses[-1] < 0.15
    assert np.mean(((H @ w + c) > 0) == (y > 0)) > 0.97


def test_loss_is_stable_for_large_logits():
    assert X.bce_loss([800.0, -800.0], [1, 0]) == pytest.approx(0.0, abs=1e-300)
    assert X.bce_loss([800.0], [0]) == pytest.approx(800.0)
