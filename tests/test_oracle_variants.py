"""Pins of the oracle's Mult-MCN-Slow and Square-MCN (Appendix A.2.1).

Mult-MCN-Slow:
  * nc = 1: the first digit fl(x y) is the result whenever it is non-zero (numpy);
  * y = (2^k, 0, ...): every remainder step is exact, so the result is x 2^k exactly;
  * against the exact product (Python fractions): every element within 4u and the
    median within 2 u^nc (binary32), the same classes as Div-MCN, whose remainder
    steps it shares.
Square-MCN (first step read as fl(x_0 x_0)):
  * nc = 1: fl(x_0^2) (numpy);
  * nc >= 2: the Grow-ExpN of (a, 0, ..., 0) and b, a = fl(x_0^2), b = fl(2 x_0 x_1),
    passes b through the zero components unchanged and ends in Two-Sum(a, b), so
    the result is (fl(a + b), a + b - fl(a + b), 0, ...): checked with numpy's
    rounding and remainders computed with exact rationals.
"""
from fractions import Fraction

import numpy as np
import pytest

from paper_2207_08867_amd import inputs

U = {np.float16: 2.0 ** -11, np.float32: 2.0 ** -24}


@pytest.mark.parametrize("dt", [np.float16, np.float32])
def test_mul_slow_nc1(orc, dt):
    x, y = inputs.elementwise_inputs("mul", 20000, 1, dt, seed=21)
    got = orc.mul_slow(x, y, nc=1)
    want = (x[0] * y[0]).astype(dt)
    nz = want != 0
    assert nz.mean() > 0.99
    assert np.array_equal(got[0][nz], want[nz])


@pytest.mark.parametrize("dt", [np.float16, np.float32])
@pytest.mark.parametrize("nc", [2, 3, 4])
def test_mul_slow_power_of_two(orc, dt, nc):
    x, _ = inputs.elementwise_inputs("mul", 5000, nc, dt, seed=22)
    g = np.random.default_rng(23)
    k = g.integers(-3, 4, x.shape[1])
    y = np.zeros_like(x)
    y[0] = np.exp2(k).astype(dt)
    got = orc.mul_slow(x, y, nc=nc)
    want = (x.astype(np.float64) * np.exp2(k)[None]).astype(dt)
    if dt == np.float16:  # keep elements whose scaled components stay normal or exactly subnormal
        ok = np.all((want.astype(np.float64) == x.astype(np.float64) * np.exp2(k)[None]), axis=0)
    else:
        ok = np.ones(x.shape[1], bool)
    assert ok.mean() > 0.6  # binary16 second components are often subnormal: 2^-k loses bits
    assert np.array_equal(got[:, ok], want[:, ok])


@pytest.mark.parametrize("dt", [np.float16, np.float32])
@pytest.mark.parametrize("nc", [2, 3])
def test_mul_slow_accuracy(orc, dt, nc):
    n = 2000
    x, y = inputs.elementwise_inputs("mul", n, nc, dt, seed=24)
    got = orc.mul_slow(x, y, nc=nc)
    F = lambda v: Fraction(float(v))
    rel = []
    for i in range(n):
        X = sum(F(v) for v in x[:, i])
        Y = sum(F(v) for v in y[:, i])
        R = sum(F(v) for v in got[:, i])
        rel.append(float(abs(R - X * Y) / abs(X * Y)))
    rel = np.array(rel)
    u = U[dt]
    assert rel.max() <= 4 * u
    if dt == np.float32 or nc == 2:
        assert np.median(rel) <= 2 * u ** nc


@pytest.mark.parametrize("dt", [np.float16, np.float32])
@pytest.mark.parametrize("nc", [1, 2, 3, 4])
def test_square_closed_form(orc, dt, nc):
    x, _ = inputs.elementwise_inputs("mul", 20000, nc, dt, seed=25)
    got = orc.square(x, nc=nc)
    a = (x[0] * x[0]).astype(dt)
    if nc == 1:
        assert np.array_equal(got[0], a)
        return
    b = ((dt(2) * x[0]).astype(dt) * x[1]).astype(dt)
    s = (a + b).astype(dt)
    # the exact remainder a + b - s (a float of the format, by the Two-Sum theorem)
    er = [Fraction(float(ai)) + Fraction(float(bi)) - Fraction(float(si)) for ai, bi, si in zip(a, b, s)]
    e = np.array([float(v) for v in er]).astype(dt)
    assert all(Fraction(float(ei)) == v for ei, v in zip(e, er))
    # Simple-Renorm: (s, e) when s is non-zero, (e, 0) otherwise (a + b = 0 exactly gives zeros)
    first = np.where(s != 0, s, e)
    second = np.where(s != 0, e, dt(0))
    assert np.array_equal(got[0], first)
    assert np.array_equal(got[1], second)
    assert not got[2:].any()
