"""Pins of the oracle with binary64 components (the paper's MC float64, used for its
hyperbolic models), against references that share none of its code:
  * nc = 1: every MC operation is one rounded binary64 operation (numpy float64);
  * the error-free transformations are exact (Python fractions);
  * nc = 2, 3, against exact rationals (u = 2^-53): Add-MCN and ScalingN within
    4 u^nc on every element; Div-MCN and Mult-MCN within 4u on every element and 2 u^nc
    at the median (the accuracy classes of these division-based algorithms);
  * MM-MCN at nc = 1 is the sequential binary64 GEMM; the K-split product at nc = 1 is
    the numpy tree; MC x MC within 4 K u^nc of the exact product, checked both by the
    oracle's exact checker (its binary64 path splits each product with fma) and by
    fractions on a small case;
  * the binary64 component exponential against decimal arithmetic (the whole range,
    subnormal results, boundaries, arguments within 2^-72 of a rounding boundary), and
    Exp-MCN over it (nc = 1, zero tails, the exact product of the component
    exponentials within 8 u^nc).
"""
from fractions import Fraction

import os

import numpy as np
import pytest

from test_oracle_splitk import _np_splitk_nc1

U = 2.0 ** -53
F = lambda v: Fraction(float(v))


def mc64(g, shape, nc, scale=1.0):
    """Canonical binary64 expansions: each part below a quarter ulp of the one before."""
    out = np.zeros((nc,) + shape)
    out[0] = g.normal(0, scale, shape)
    for c in range(1, nc):
        ulp = np.exp2(np.floor(np.log2(np.abs(out[c - 1]) + 1e-300)) - 52)
        out[c] = g.uniform(-0.25, 0.25, shape) * ulp
    return out


def val(x, i):
    return sum(F(x[c].flat[i]) for c in range(x.shape[0]))


def test_nc1_is_binary64(orc):
    g = np.random.default_rng(80)
    x = g.normal(0, 1, (1, 5000)) * np.exp2(g.integers(-40, 40, (1, 5000)))
    y = g.normal(0, 1, (1, 5000)) * np.exp2(g.integers(-40, 40, (1, 5000)))
    assert np.array_equal(orc.add(x, y, nc=1), x + y)
    assert np.array_equal(orc.add(x, y[0], nc=1, y_mc=False), x + y)
    assert np.array_equal(orc.mul(x, y[0], nc=1, y_mc=False), x * y)
    assert np.array_equal(orc.div(x, y, nc=1), x / y)


def test_eft_exact(orc):
    g = np.random.default_rng(81)
    a = g.normal(0, 1, 3000) * np.exp2(g.integers(-60, 60, 3000))
    b = g.normal(0, 1, 3000) * np.exp2(g.integers(-60, 60, 3000))
    s, e = orc.two_sum(orc.F64, a, b)
    p, f = orc.two_prod(orc.F64, a, b)
    for i in range(3000):
        assert F(s[i]) + F(e[i]) == F(a[i]) + F(b[i])
        assert F(p[i]) + F(f[i]) == F(a[i]) * F(b[i])
        assert s[i] == a[i] + b[i] and p[i] == a[i] * b[i]


@pytest.mark.parametrize("nc", [2, 3])
def test_mc_accuracy(orc, nc):
    g = np.random.default_rng(82 + nc)
    n = 1500
    x = mc64(g, (n,), nc)
    y = mc64(g, (n,), nc)
    y[0] = np.abs(y[0]) + 0.5  # divisors away from zero
    v = g.normal(0, 1, n)
    add = orc.add(x, y, nc=nc)
    scl = orc.mul(x, v, nc=nc, y_mc=False)
    div = orc.div(x, y, nc=nc)
    mul = orc.mul(x, y, nc=nc)
    rel = {"div": [], "mul": []}
    for i in range(n):
        X, Y, V = val(x, i), val(y, i), F(v[i])
        # Add-MCN and ScalingN: every element within 4 u^nc
        for got, exact, mag in ((val(add, i), X + Y, abs(X) + abs(Y)), (val(scl, i), X * V, abs(X * V))):
            assert abs(got - exact) <= 4 * Fraction(U) ** nc * mag + Fraction(2) ** -1070, i
        rel["div"].append(float(abs(val(div, i) - X / Y) / abs(X / Y)))
        rel["mul"].append(float(abs(val(mul, i) - X * Y) / abs(X * Y)))
    # Div-MCN and Mult-MCN (division-based): every element within 4u, the median within
    # 2 u^nc -- the accuracy classes the binary32 pins establish for these algorithms
    for k, r in rel.items():
        assert max(r) <= 4 * U, k
        assert np.median(r) <= 2 * U ** nc, k


def test_matmul_nc1_and_splitk_nc1(orc):
    g = np.random.default_rng(85)
    M, N, K = 6, 7, 45
    A = g.normal(0, 1, (M, K)) * np.exp2(g.integers(-20, 20, (M, K)))
    B = g.normal(0, 1, (K, N))
    acc = A[:, 0, None] * B[None, 0, :]
    for k in range(1, K):
        acc = acc + A[:, k, None] * B[None, k, :]
    assert np.array_equal(orc.matmul(A[None], B[None], nc=1), acc[None])
    for S in (2, 5, 13):
        got = orc.matmul_splitk(A[None], B[None], nc=1, slices=S, b_mc=False)[0]
        assert np.array_equal(got, _np_splitk_nc1(A, B, S))


@pytest.mark.parametrize("nc", [2, 3])
def test_matmul_mc_bound(orc, nc):
    g = np.random.default_rng(86 + nc)
    M, N, K = 5, 4, 30
    A = mc64(g, (M, K), nc)
    B = mc64(g, (K, N), nc)
    C = orc.matmul(A, B, nc=nc)
    err, absab, _ = orc.matmul_exact_err(A, B, C)
    assert np.all(np.abs(err) <= 4 * K * U ** nc * absab)
    # the checker's binary64 path (fma-split products) against fractions
    for i in range(M):
        for j in range(N):
            exact = sum(val(A[:, i:i + 1, k:k + 1], 0) * val(B[:, k:k + 1, j:j + 1], 0) for k in range(K))
            e = sum(F(C[c, i, j]) for c in range(nc)) - exact
            assert abs(float(e) - err[i * N + j]) <= 2.0 ** -50 * abs(float(e)) + 1e-300


def _decimal_exp(x):
    """e^x from 90-digit decimal arithmetic, converted to binary64 (both steps correctly
    rounded; the arguments used here are not within 10^-80 of a rounding boundary)."""
    import decimal

    with decimal.localcontext() as ctx:
        ctx.prec = 90
        ctx.Emin, ctx.Emax = -999999, 999999
        return float(decimal.Decimal(float(x)).exp())


def test_exp64_correctly_rounded_sample(orc):
    """The binary64 component exponential against decimal arithmetic: the whole finite
    range, the subnormal results, tiny arguments, boundaries and special values."""
    g = np.random.default_rng(40)
    xs = np.concatenate([g.uniform(-745.2, 709.8, 6000), g.uniform(-1, 1, 3000), g.uniform(-746, -708, 2000),
                         g.normal(0, 1, 2000) * np.exp2(g.integers(-80, 0, 2000)),
                         [0.0, -0.0, 709.782712893384, 709.7827128933841, -745.1332191019411,
                          -745.1332191019412, -708.3964185322641, 1e-300, -1e-300, 2.0 ** -53, -(2.0 ** -54)]])
    got = orc.fl_exp64(xs)
    want = np.array([_decimal_exp(x) for x in xs])
    assert np.array_equal(got, want)
    assert not np.signbit(got).any()
    sp = orc.fl_exp64(np.array([np.inf, -np.inf, np.nan, 800.0, -800.0]))
    assert sp[0] == np.inf and sp[1] == 0.0 and np.isnan(sp[2]) and sp[3] == np.inf and sp[4] == 0.0


def test_exp64_near_rounding_boundaries(orc):
    """Arguments whose e^x lies within 2^-72 of a rounding boundary (the fixture written
    by tests/golden/make_exp64_near_midpoints.py) are rounded as decimal arithmetic
    rounds them."""
    path = os.path.join(os.path.dirname(__file__), "golden", "exp64_near_midpoints.txt")
    xs = np.array([float.fromhex(l) for l in open(path) if l.strip() and not l.startswith("#")])
    assert len(xs) > 200
    assert np.array_equal(orc.fl_exp64(xs), np.array([_decimal_exp(x) for x in xs]))


def test_exp_mcn_binary64(orc):
    """Exp-MCN over binary64 components: nc = 1 is the correctly rounded exponential;
    exp((x_0, 0, ...)) = (e^x_0, 0, ...); and the result equals the exact product of the
    component exponentials up to the carry roundings of the ScalingN chain."""
    g = np.random.default_rng(41)
    n = 1500
    x1 = g.uniform(-20, 20, (1, n))
    assert np.array_equal(orc.exp(x1, nc=1)[0], orc.fl_exp64(x1[0]))
    x = np.zeros((3, n))
    x[0] = x1[0]
    r = orc.exp(x, nc=3)
    assert np.array_equal(r[0], orc.fl_exp64(x1[0])) and not r[1:].any()
    for nc in (2, 3):
        x = np.zeros((nc, n))
        x[0] = g.uniform(-20, 20, n)
        for c in range(1, nc):
            x[c] = g.uniform(-1, 1, n) * np.exp2(-20 * c)
        r = orc.exp(x, nc=nc)
        E = orc.fl_exp64(x)
        u = Fraction(2) ** -53
        for i in range(n):
            prod = Fraction(1)
            for c in range(nc):
                prod *= Fraction(float(E[c, i]))
            got = sum(Fraction(float(r[c, i])) for c in range(nc))
            assert abs(got - prod) <= 8 * u ** nc * prod, i
