"""Pins for the oracle's matrix products (Appendix A.2.2; MC-Linear of Section 2.3)
and for its exact-arithmetic checker.

  * nc = 1: MM-MCN collapses to the plain sequential float product with one
    rounding per multiply and per add, evaluated here with numpy.
  * K = 1: the product is ScalingN of each MC entry by the plain entry.
  * Transposition: (A B)^T computed as B^T A^T with the operand roles swapped gives
    the same components (same terms, same order), which pins the index handling.
  * MC x MC with a B whose lower components are zero equals MC x plain.
  * Error bound against exact rational arithmetic: |C - C*| <= 4 K u^nc (|A||B|)
    plus, in binary16, a floor of nA nB K eta for Two-Prod errors that fall below
    the subnormal grid.
  * MC-Linear equals the product with the transposed weight followed by Add-MCN.
  * The exact checker itself against Python Fractions.
"""
from fractions import Fraction

import numpy as np
import pytest

from paper_2207_08867_amd import inputs

U = {np.float16: 2.0 ** -11, np.float32: 2.0 ** -24}
ETA16 = 2.0 ** -25


def _seq_plain_matmul(A, B):
    """Plain product, k sequential, one rounding per operation (numpy scalar-type arrays)."""
    dt = A.dtype.type
    M, K = A.shape
    acc = np.outer(A[:, 0], B[0, :]).astype(dt) if K else np.zeros((M, B.shape[1]), dt)
    with np.errstate(all="ignore"):
        for k in range(1, K):
            acc = (acc + np.outer(A[:, k], B[k, :]).astype(dt)).astype(dt)
    return acc


@pytest.mark.parametrize("dt", [np.float16, np.float32])
def test_nc1_is_sequential_float_gemm(orc, dt):
    g = np.random.default_rng(30)
    A = g.uniform(-1, 1, (13, 37)).astype(dt)
    B = g.uniform(-1, 1, (37, 11)).astype(dt)
    C = orc.matmul(A[None], B[None], nc=1)[0]
    ref = _seq_plain_matmul(A, B)
    assert np.array_equal(C.astype(np.float64), ref.astype(np.float64))
    C2 = orc.matmul(A[None], B[None], nc=1, a_mc=False)[0]
    assert np.array_equal(C2.astype(np.float64), ref.astype(np.float64))


@pytest.mark.parametrize("dt,nc", [(np.float32, 2), (np.float32, 3), (np.float16, 3)])
def test_k1_is_scaling(orc, dt, nc):
    g = np.random.default_rng(31)
    M, N = 9, 7
    A = inputs.split(g.uniform(-1, 1, (M, 1)), nc, dt)
    B = g.uniform(-1, 1, (1, N)).astype(dt)
    C = orc.matmul(A, B[None], nc=nc, b_mc=False)
    for j in range(N):
        ref = orc.mul(A[:, :, 0], np.full(M, B[0, j], dtype=dt), nc=nc, y_mc=False)
        assert np.array_equal(C[:, :, j], ref)


@pytest.mark.parametrize("dt,nc", [(np.float32, 2), (np.float16, 3)])
def test_transpose_swaps_roles(orc, dt, nc):
    g = np.random.default_rng(32)
    M, N, K = 11, 6, 29
    A = inputs.split(g.normal(0, 1, (M, K)), nc, dt)
    B = g.normal(0, 1, (K, N)).astype(dt)
    C = orc.matmul(A, B[None], nc=nc, b_mc=False)
    At = np.ascontiguousarray(A.transpose(0, 2, 1))
    Bt = np.ascontiguousarray(B.T)
    Ct = orc.matmul(Bt[None], At, nc=nc, a_mc=False)
    assert np.array_equal(C, Ct.transpose(0, 2, 1))


def test_mcxmc_with_plain_b_equals_mcxplain(orc):
    g = np.random.default_rng(33)
    nc, dt = 3, np.float32
    A = inputs.split(g.normal(0, 1, (8, 20)), nc, dt)
    B0 = g.normal(0, 1, (20, 5)).astype(dt)
    B = np.zeros((nc, 20, 5), dtype=dt)
    B[0] = B0
    assert np.array_equal(orc.matmul(A, B, nc=nc), orc.matmul(A, B0[None], nc=nc, b_mc=False))


def _fr_matrix(P):
    return [[Fraction(float(v)) for v in row] for row in P]


def _exact_product(A, B):
    """Exact rational product of the MC inputs (planes summed exactly)."""
    Af = sum(np.array(_fr_matrix(A[c]), dtype=object) for c in range(A.shape[0]))
    Bf = sum(np.array(_fr_matrix(B[c]), dtype=object) for c in range(B.shape[0]))
    return Af.dot(Bf), np.abs(Af).dot(np.abs(Bf))


@pytest.mark.parametrize("dt,nc,a_mc,b_mc", [
    (np.float32, 2, True, True), (np.float32, 3, True, True), (np.float32, 3, True, False),
    (np.float32, 2, False, True), (np.float16, 2, True, True), (np.float16, 3, True, True),
])
def test_bound_vs_exact_fractions(orc, dt, nc, a_mc, b_mc):
    g = np.random.default_rng(34)
    M, N, K = 6, 5, 24
    A = inputs.split(g.normal(0, 1 / np.sqrt(K), (M, K)), nc if a_mc else 1, dt)
    B = inputs.split(g.normal(0, 1 / np.sqrt(K), (K, N)), nc if b_mc else 1, dt)
    C = orc.matmul(A, B, nc=nc, a_mc=a_mc, b_mc=b_mc)
    exact, absab = _exact_product(A, B)
    Cf = sum(np.array(_fr_matrix(C[c]), dtype=object) for c in range(nc))
    u = Fraction(U[dt])
    floor = Fraction(A.shape[0] * B.shape[0] * K) * Fraction(ETA16) if dt == np.float16 else 0
    for i in range(M):
        for j in range(N):
            assert abs(Cf[i, j] - exact[i, j]) <= 4 * K * u ** nc * absab[i, j] + floor


def test_exact_checker_vs_fractions(orc):
    """The C exact checker (fixed-point accumulator) against Fractions, with wide
    exponent ranges and subnormal components."""
    g = np.random.default_rng(35)
    for dt, nc in ((np.float32, 3), (np.float16, 3), (np.float32, 2)):
        M, N, K = 5, 4, 17
        sc = np.exp2(g.integers(-30, 30, (M, K))) if dt == np.float32 else np.exp2(g.integers(-8, 8, (M, K)))
        A = inputs.split(g.normal(0, 1, (M, K)) * sc, nc, dt)
        B = inputs.split(g.normal(0, 1, (K, N)), nc, dt)
        C = orc.matmul(A, B, nc=nc)
        bias = inputs.split(g.normal(0, 1, N), nc, dt)
        exact, absab = _exact_product(A, B)
        bf = [sum(Fraction(float(bias[c, j])) for c in range(nc)) for j in range(N)]
        err, ab, ex = orc.matmul_exact_err(A, B, C, bias=bias)
        Cf = sum(np.array(_fr_matrix(C[c]), dtype=object) for c in range(nc))
        for i in range(M):
            for j in range(N):
                t = i * N + j
                want = Cf[i, j] - exact[i, j] - bf[j]
                assert abs(Fraction(err[t]) - want) <= abs(want) * Fraction(2) ** -50
                assert abs(Fraction(ex[t]) - (exact[i, j] + bf[j])) <= abs(exact[i, j] + bf[j]) * Fraction(2) ** -50
                want_ab = absab[i, j] + abs(bf[j])
                assert abs(Fraction(ab[t]) - want_ab) <= want_ab * Fraction(2) ** -40


def test_exact_checker_cancellation(orc):
    """Exact sums that cancel to tiny or zero values."""
    dt = np.float32
    x = np.array([[1.0, -1.0, 2.0 ** -100], [2.0 ** -149, 0.0, 3.0]], dtype=dt).reshape(2, 3)
    y = np.array([[1.0, -1.0, 2.0 ** -100]], dtype=dt)
    d = orc.exact_diff(x, y)
    assert d[0] == 2.0 ** -149 and d[1] == 0.0 and d[2] == 3.0


def test_positions_match_full(orc):
    g = np.random.default_rng(36)
    nc, dt = 3, np.float32
    A, B = inputs.matmul_normal(17, 23, 31, nc, dt, seed=36)
    C = orc.matmul(A, B, nc=nc)
    rows = g.integers(0, 17, 40)
    cols = g.integers(0, 23, 40)
    Cs = orc.matmul(A, B, nc=nc, rows=rows, cols=cols)
    assert np.array_equal(Cs, C[:, rows, cols])


@pytest.mark.parametrize("bias", [True, False])
def test_linear_is_product_then_add(orc, bias):
    nc, dt = 3, np.float16
    x, W, b = next(inputs.linear_inputs(19, 33, 14, nc, dt, seed=37))
    Y = orc.linear(x, W, b if bias else None, nc=nc)
    P = orc.matmul(x[None], np.ascontiguousarray(W.transpose(0, 2, 1)), nc=nc, a_mc=False)
    if bias:
        P = orc.add(P, np.broadcast_to(b[:, None, :], P.shape).copy(), nc=nc)
    assert np.array_equal(Y, P)


def test_degenerate_sizes(orc):
    nc, dt = 2, np.float32
    A = np.zeros((nc, 3, 0), dtype=dt)
    B = np.zeros((nc, 0, 4), dtype=dt)
    C = orc.matmul(A, B, nc=nc)
    assert C.shape == (nc, 3, 4) and (C == 0).all() and not np.signbit(C).any()


# ---------------------------------------------------------------------------------
# pruned MC x MC product
# ---------------------------------------------------------------------------------

def _seq_gemm(A, B, dt):
    acc = (A[:, 0][:, None] * B[0][None, :]).astype(dt)
    for k in range(1, A.shape[1]):
        acc = (acc + (A[:, k][:, None] * B[k][None, :]).astype(dt)).astype(dt)
    return acc


@pytest.mark.parametrize("dt", [np.float16, np.float32])
def test_pruned_nc1_and_nc2_structure(orc, dt):
    """nc = 1: nothing is pruned (the product is MM-MCN).  nc = 2: the pruned product
    is Add-MCN(MM-MCN(A, B^(0)), (G, 0)) with G the sequential float GEMM of A^(0) and
    B^(1), evaluated by numpy."""
    A, B = inputs.matmul_normal(9, 7, 11, 1, dt, seed=31)
    assert np.array_equal(orc.matmul_pruned(A, B, nc=1), orc.matmul(A, B, nc=1))
    A, B = inputs.matmul_normal(9, 7, 11, 2, dt, seed=32)
    P0 = orc.matmul(A, B[:1], nc=2, a_mc=True, b_mc=False)
    G = _seq_gemm(A[0], B[1], dt)
    want = orc.add(P0, np.stack([G, np.zeros_like(G)]), nc=2)
    assert np.array_equal(orc.matmul_pruned(A, B, nc=2), want)


@pytest.mark.parametrize("dt", [np.float16, np.float32])
@pytest.mark.parametrize("nc", [2, 3, 4])
def test_pruned_zero_low_components_of_b(orc, dt, nc):
    """When B's low components are zero, nothing is left out: the pruned product is
    MM-MCN bit for bit."""
    A, B = inputs.matmul_normal(12, 10, 9, nc, dt, seed=33)
    B[1:] = 0
    assert np.array_equal(orc.matmul_pruned(A, B, nc=nc), orc.matmul(A, B, nc=nc))


@pytest.mark.parametrize("dt", [np.float16, np.float32])
@pytest.mark.parametrize("nc", [2, 3, 4])
def test_pruned_exact_bound(orc, dt, nc):
    """Within 4 K u^min(nc,3) (|A||B|) (+ the binary16 floor) of the exact product."""
    for M, N, K, gen in ((16, 12, 300, "normal"), (8, 8, 64, "uniform")):
        if gen == "normal":
            A, B = inputs.matmul_normal(M, N, K, nc, dt, seed=34)
        else:
            A, B = inputs.matmul_uniform(M, N, K, nc, dt, seed=34)
        C = orc.matmul_pruned(A, B, nc=nc)
        err, absab, _ = orc.matmul_exact_err(A, B, C)
        u = U[dt]
        floor = nc * nc * K * 2.0 ** -25 if dt == np.float16 else 0.0
        assert (np.abs(err) <= 4 * K * u ** min(nc, 3) * absab + floor).all()
