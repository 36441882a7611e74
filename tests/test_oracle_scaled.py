"""Pins for the oracle's binary16 arithmetic with scaled low components (reading SC1:
component c stands for 2^(-11 c) times its stored binary16 value, and every rounding
of the paper's algorithms is taken in the binary16 format of its level).

Checked against facts that do not come from the oracle:
  * nc = 1 is plain binary16 arithmetic (numpy float16 operations and the sequential
    float16 GEMM);
  * nc = 2 closed forms: Add-MCN of two one-term values is (RN(a+b), the exact rounding
    error) and ScalingN of a one-term value is (RN(ab), ab - RN(ab)), the error stored
    one level down -- so, unlike plain binary16, the pair holds a b exactly even when
    the error lies below the binary16 subnormal grid;
  * error bounds against the exact value of the inputs (Python Fractions and the
    exact fixed-point checker) with NO subnormal floor -- the stated 4 K u^nc for the
    products -- on data where the plain binary16 format provably cannot meet them;
  * structural identities (a product with one reduction step is ScalingN; MC x MC with
    zero low components of B is MC x plain).
"""
from fractions import Fraction

import numpy as np
import pytest

from paper_2207_08867_amd import inputs

U16 = 2.0 ** -11


def _seq_f16_matmul(A, B):
    """Plain binary16 product, k sequential, one rounding per operation."""
    M, K = A.shape
    acc = np.outer(A[:, 0], B[0, :]).astype(np.float16)
    for k in range(1, K):
        acc = (acc + np.outer(A[:, k], B[k, :]).astype(np.float16)).astype(np.float16)
    return acc


def _exact(planes, i):
    return sum(Fraction(float(planes[c, i])) for c in range(planes.shape[0]))


def test_split_scaled_levels():
    g = np.random.default_rng(1)
    x = g.normal(0.0, 1 / 32, 5000)
    s = inputs.split_scaled(x, 4)
    # level c holds the next binary16 precision: four components keep 44 bits of every x
    # whose leading component is a normal binary16 number
    val = sum(np.ldexp(s[c].astype(np.float64), -11 * c) for c in range(4))
    big = np.abs(x) >= 2.0 ** -13
    assert np.all(np.abs(val - x)[big] <= np.abs(x)[big] * 2.0 ** -43)
    assert np.count_nonzero(s[2]) > 4900  # unlike plain binary16, the third component is in use


def test_nc1_is_plain_binary16(orc):
    g = np.random.default_rng(2)
    x = g.uniform(-2, 2, 3001).astype(np.float16)
    y = g.uniform(-2, 2, 3001).astype(np.float16)
    assert np.array_equal(orc.scaled_add(x[None], y[None], nc=1)[0], (x + y).astype(np.float16))
    assert np.array_equal(orc.scaled_mul(x[None], y[None], nc=1)[0], (x * y).astype(np.float16))
    A = g.uniform(-1, 1, (13, 37)).astype(np.float16)
    B = g.uniform(-1, 1, (37, 11)).astype(np.float16)
    ref = _seq_f16_matmul(A, B)
    assert np.array_equal(orc.scaled_matmul(A[None], B[None], nc=1)[0], ref)
    assert np.array_equal(orc.scaled_matmul(A[None], B[None], nc=1, a_mc=False)[0], ref)
    assert np.array_equal(orc.scaled_linear(A, np.ascontiguousarray(B.T)[None], nc=1)[0], ref)


def test_nc2_two_sum_closed_form(orc):
    """Add-MCN((a, 0), (b, 0)) = (s, e) with s = RN(a + b) and e = a + b - s exactly,
    e stored at level 1 (times 2^11)."""
    g = np.random.default_rng(3)
    a = g.normal(0, 1, 4000).astype(np.float16)
    b = (g.normal(0, 1, 4000) * np.exp2(g.integers(-14, 1, 4000))).astype(np.float16)
    s = (a.astype(np.float64) + b).astype(np.float16)
    keep = s != 0
    a, b, s = a[keep], b[keep], s[keep]
    e = a.astype(np.float64) + b.astype(np.float64) - s.astype(np.float64)
    z = np.zeros_like(a)
    got = orc.scaled_add(np.stack([a, z]), np.stack([b, z]), nc=2)
    assert np.array_equal(got[0], s)
    assert np.array_equal(got[1].astype(np.float64), np.ldexp(e, 11).astype(np.float16).astype(np.float64))
    # the pair is exact: a + b = s + 2^-11 got[1]
    assert np.array_equal(s.astype(np.float64) + np.ldexp(got[1].astype(np.float64), -11),
                          a.astype(np.float64) + b.astype(np.float64))


def test_nc2_two_prod_exact_below_the_subnormal_grid(orc):
    """ScalingN((a, 0), b) = (p, e) with p = RN(ab) and e = ab - p at level 1: for a
    normal p (|ab| >= 2^-14) the pair holds ab exactly, also where ab - p lies below
    2^-24 (plain binary16 loses it)."""
    g = np.random.default_rng(4)
    a = (g.uniform(0.5, 1, 4000) * np.exp2(g.integers(-6, 2, 4000)) * g.choice([-1, 1], 4000)).astype(np.float16)
    v = (g.uniform(0.5, 1, 4000) * np.exp2(g.integers(-6, 2, 4000))).astype(np.float16)
    ab = a.astype(np.float64) * v.astype(np.float64)
    p = ab.astype(np.float16)
    got = orc.scaled_mul(np.stack([a, np.zeros_like(a)]), v[None], nc=2)
    assert np.array_equal(got[0], p)
    assert np.array_equal(p.astype(np.float64) + np.ldexp(got[1].astype(np.float64), -11), ab)
    lost = (ab - p.astype(np.float64)) != (ab - p.astype(np.float64)).astype(np.float16).astype(np.float64)
    assert lost.sum() > 1000  # cases where plain binary16 cannot hold the error


@pytest.mark.parametrize("nc", [2, 3])
def test_add_and_scaling_bounds_without_floor(orc, nc):
    """|Add-MCN(x, y) - (x + y)| <= 8 u^nc (|x| + |y|) and |ScalingN(x, v) - x v| <=
    8 u^nc |x| |v| exactly (Fractions), at magnitudes 2^-8 .. 1 (products 2^-12 .. 1:
    leading terms stay normal binary16 numbers) where plain binary16 components cannot
    reach u^3 (their last level would need bits below 2^-24)."""
    g = np.random.default_rng(10 + nc)
    n = 600
    mag = np.exp2(g.integers(-8, 1, n))
    x = inputs.split_scaled(g.uniform(0.5, 1, n) * g.choice([-1, 1], n) * mag, nc)
    y = inputs.split_scaled(g.uniform(-1, 1, n) * mag, nc)
    v = (g.uniform(0.5, 1, n) * g.choice([-1, 1], n) * np.exp2(g.integers(-3, 1, n))).astype(np.float16)
    xs, ys = orc.unscale(x), orc.unscale(y)
    add = orc.unscale(orc.scaled_add(x, y, nc=nc))
    mul = orc.unscale(orc.scaled_mul(x, v[None], nc=nc))
    lim = Fraction(8) * Fraction(U16) ** nc
    for i in range(n):
        X, Y, V = _exact(xs, i), _exact(ys, i), Fraction(float(v[i]))
        assert abs(_exact(add, i) - (X + Y)) <= lim * (abs(X) + abs(Y)), i
        assert abs(_exact(mul, i) - X * V) <= lim * abs(X) * abs(V), i


def _literal_ratio(orc, A, B, C, nc, K, bias=None):
    err, absab, _ = orc.matmul_exact_err(orc.unscale(A), orc.unscale(B), orc.unscale(C),
                                         bias=None if bias is None else orc.unscale(bias))
    return float(np.max(np.abs(err) / absab)) / (4 * K * U16 ** nc)


@pytest.mark.parametrize("nc", [2, 3])
@pytest.mark.parametrize("kinds", [(True, True), (True, False), (False, True)])
def test_product_literal_bound(orc, nc, kinds):
    """The stated tolerance |C - C*| <= 4 K u^nc (|A||B|), as written, for every
    output (entries N(0, 1/K), K = 512) -- which plain binary16 components miss at
    nc = 3 on the same values."""
    a_mc, b_mc = kinds
    M, N, K = 24, 20, 512
    A, B = inputs.matmul_normal_scaled(M, N, K, nc, seed=20 + nc)
    A = A if a_mc else A[:1]
    B = B if b_mc else B[:1]
    C = orc.scaled_matmul(A, B, nc=nc, a_mc=a_mc, b_mc=b_mc)
    assert _literal_ratio(orc, A, B, C, nc, K) <= 1.0
    if nc == 3 and a_mc and b_mc:
        Ap, Bp = inputs.matmul_normal(M, N, K, nc, np.float16, seed=20 + nc)
        Cp = orc.matmul(Ap, Bp, nc=nc)
        err, absab, _ = orc.matmul_exact_err(Ap, Bp, Cp)
        assert float(np.max(np.abs(err) / absab)) > 4 * K * U16 ** 3


def test_linear_literal_bound(orc):
    x, W, b = next(inputs.linear_inputs_scaled(40, 256, 24, 3, seed=5))
    Y = orc.scaled_linear(x, W, b, nc=3)
    Wt = np.ascontiguousarray(W.transpose(0, 2, 1))
    assert _literal_ratio(orc, x[None], Wt, Y, 3, 256, bias=b) <= 1.0


def test_one_step_product_is_scaling(orc):
    g = np.random.default_rng(6)
    A = inputs.split_scaled(g.normal(0, 0.1, (9, 1)), 3)
    B = g.normal(0, 0.1, (1, 7)).astype(np.float16)
    C = orc.scaled_matmul(A, B[None], nc=3, b_mc=False)
    ref = orc.scaled_mul(np.repeat(A[:, :, 0:1], 7, axis=2).reshape(3, -1), np.tile(B, (9, 1)).reshape(1, -1),
                         nc=3)
    assert np.array_equal(C.reshape(3, -1).view(np.uint16), ref.view(np.uint16))


def test_mc_by_mc_with_zero_low_components_is_mc_by_plain(orc):
    A, B = inputs.matmul_normal_scaled(11, 13, 70, 3, seed=7)
    Bz = B.copy()
    Bz[1:] = 0
    C = orc.scaled_matmul(A, Bz, nc=3)
    ref = orc.scaled_matmul(A, B[:1], nc=3, b_mc=False)
    assert np.array_equal(C.view(np.uint16), ref.view(np.uint16))


def test_positions_match_full(orc):
    A, B = inputs.matmul_normal_scaled(9, 8, 33, 2, seed=8)
    full = orc.scaled_matmul(A, B, nc=2)
    rows = np.array([0, 8, 3, 5])
    cols = np.array([7, 0, 3, 2])
    assert np.array_equal(orc.scaled_matmul(A, B, nc=2, rows=rows, cols=cols).view(np.uint16),
                          full[:, rows, cols].view(np.uint16))
