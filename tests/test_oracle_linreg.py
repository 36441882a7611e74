"""Pins of the oracle's linear-regression gradient-descent step (Section 2.4; reading:
MC residual, K-split r^T X and r . r, ScalingN by fl(2/n), the leading component as the
plain gradient, Grow-ExpN update):
  * nc = 1: every MC step is one rounded operation, so the step equals a numpy
    evaluation in the component format (sequential linear layer, the K-split tree sums
    written independently in numpy);
  * an exactly fitted model is a fixed point: r = 0, so W is unchanged and the loss is 0;
  * the loss equals (1/n) sum r_i^2 of the MC residual (exact rationals) within the
    rounding of fl(1/n) and the MC sum;
  * gradient descent converges towards W*: the loss falls by orders of magnitude.
"""
from fractions import Fraction

import numpy as np
import pytest

from paper_2207_08867_amd import inputs
from test_oracle_splitk import _np_splitk_nc1


def _bits(a):
    a = np.asarray(a)
    return a.view(np.uint16 if a.dtype == np.float16 else np.uint32)


@pytest.mark.parametrize("dt", [np.float16, np.float32])
def test_nc1_is_plain_float_step(orc, dt):
    n, d, Sg, Sl, lr = 301, 3, 7, 5, 0.05
    X, y_neg, W, _ = inputs.linreg_inputs(n, d, 1, dt, seed=70)
    W_new, loss = orc.linreg_gd_step(X, y_neg, W, lr, slices_g=Sg, slices_l=Sl)
    with np.errstate(all="ignore"):
        acc = (X[:, 0] * W[0, 0]).astype(dt)
        for j in range(1, d):
            acc = (acc + (X[:, j] * W[0, j]).astype(dt)).astype(dt)
        r = (acc + y_neg).astype(dt)
        G = _np_splitk_nc1(r[None, :], X, Sg)[0]
        RR = _np_splitk_nc1(r[None, :], r[:, None], Sl)[0, 0]
        g = (G * dt(2.0 / n)).astype(dt)
        step = (dt(-lr) * g).astype(dt)
        W_ref = (W[0] + step).astype(dt)
        loss_ref = dt(RR * dt(1.0 / n))
    assert np.array_equal(_bits(W_new[0]), _bits(W_ref))
    assert _bits(loss[0]) == _bits(np.array([loss_ref], dt))[0]


@pytest.mark.parametrize("dt", [np.float16, np.float32])
@pytest.mark.parametrize("nc", [1, 2, 3])
def test_exact_fit_is_fixed_point(orc, dt, nc):
    g = np.random.default_rng(71)
    n, d = 200, 2
    X = g.integers(-4, 5, (n, d)).astype(dt)
    w_star = np.array([0.75, -1.25])
    y = X.astype(np.float64) @ w_star
    assert np.array_equal(y.astype(dt).astype(np.float64), y)  # the targets are exact
    W = np.zeros((nc, d), dt)
    W[0] = w_star
    W_new, loss = orc.linreg_gd_step(X, (-y).astype(dt), W, 0.05, slices_g=9, slices_l=4)
    assert np.array_equal(W_new.astype(np.float64), W.astype(np.float64))
    assert not loss.astype(np.float64).any()


@pytest.mark.parametrize("dt", [np.float16, np.float32])
@pytest.mark.parametrize("nc", [2, 3])
def test_loss_is_mean_square_of_residual(orc, dt, nc):
    n, d = 400, 2
    X, y_neg, W, _ = inputs.linreg_inputs(n, d, nc, dt, seed=72)
    _, loss = orc.linreg_gd_step(X, y_neg, W, 0.05, slices_g=11, slices_l=13)
    yhat = orc.linear(X, W.reshape(nc, 1, d), nc=nc).reshape(nc, n)
    r = orc.add(yhat, y_neg, nc=nc, y_mc=False)
    F = lambda v: Fraction(float(v))
    exact = sum(sum(F(r[c, i]) for c in range(nc)) ** 2 for i in range(n)) / n
    got = sum(F(v) for v in loss)
    u = 2.0 ** -11 if dt == np.float16 else 2.0 ** -24
    assert abs(got - exact) <= Fraction(3 * u) * exact


def test_gradient_descent_converges(orc):
    n, d = 500, 2
    X, y_neg, W, w_star = inputs.linreg_inputs(n, d, 2, np.float32, seed=73)
    losses = []
    for _ in range(300):
        W, loss = orc.linreg_gd_step(X, y_neg, W, 0.05, slices_g=62, slices_l=62)
        losses.append(float(loss.astype(np.float64).sum()))
    assert losses[-1] < 1e-4 * losses[0]
    w = W.astype(np.float64).sum(axis=0)
    assert np.abs(w - w_star).max() < 1e-2
