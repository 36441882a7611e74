"""Pins of the oracle's batched product (BMM-MCN / 4DMM-MCN) and AddMM-MCN
(Appendix A.2.2) against references that do not use the oracle's code:

* nc = 1 reduces every MC step to one rounded operation (ScalingN -> fl(x v),
  Add-MCN -> fl(x + y)), so the batched product is the sequential float GEMM and
  AddMM is fl(fl(alpha P) + fl(beta Y)); numpy evaluates both in the component
  format, with its own broadcasting of the batch dimensions;
* AddMM with alpha = 2^k and beta = 0 is 2^k times MM-MCN exactly (ScalingN by a
  power of two multiplies every component exactly; ScalingN by 0 gives zeros, and
  Add-MCN with zeros returns its compact operand unchanged);
* the AddMM result lies within 4 K u^nc (|alpha| |A||B| + |beta| |Y|) (+ a few u^nc
  for the final scalings and addition) of the exact alpha A B + beta Y, computed
  with Python fractions.
"""
from fractions import Fraction

import numpy as np
import pytest

from paper_2207_08867_amd import inputs


def seq_gemm(A, B, dt):
    """Sequential float GEMM in format dt with numpy broadcasting over leading
    dimensions: acc = fl(a_0 b_0), acc = fl(acc + fl(a_k b_k))."""
    A = A.astype(dt)
    B = B.astype(dt)
    acc = (A[..., :, 0][..., :, None] * B[..., 0, :][..., None, :]).astype(dt)
    for k in range(1, A.shape[-1]):
        acc = (acc + (A[..., :, k][..., :, None] * B[..., k, :][..., None, :]).astype(dt)).astype(dt)
    return acc


@pytest.mark.parametrize("dt", [np.float16, np.float32])
@pytest.mark.parametrize("shapes", [((3, 5, 4), (3, 4, 6)),
                                    ((2, 1, 5, 4), (1, 3, 4, 6)),
                                    ((4, 5, 4), (2, 4, 4, 6)),
                                    ((1, 5, 4), (3, 4, 6))])
def test_batched_nc1_is_sequential_gemm(orc, dt, shapes):
    sa, sb = shapes
    g = np.random.default_rng(11)
    A = g.uniform(-1, 1, sa).astype(dt)
    B = g.uniform(-1, 1, sb).astype(dt)
    got = orc.matmul_batched(A[None], B[None], nc=1)
    assert got.shape == (1,) + np.matmul(np.zeros(sa), np.zeros(sb)).shape
    want = seq_gemm(A, B, dt)
    assert np.array_equal(got[0].view(np.uint16 if dt == np.float16 else np.uint32),
                          np.broadcast_to(want, got.shape[1:]).view(np.uint16 if dt == np.float16 else np.uint32))


@pytest.mark.parametrize("dt", [np.float16, np.float32])
@pytest.mark.parametrize("y_full", [True, False])
def test_addmm_nc1_closed_form(orc, dt, y_full):
    g = np.random.default_rng(12)
    M, N, K = 7, 6, 9
    A = g.uniform(-1, 1, (M, K)).astype(dt)
    B = g.uniform(-1, 1, (K, N)).astype(dt)
    Y = g.uniform(-1, 1, (M, N) if y_full else (N,)).astype(dt)
    alpha, beta = dt(0.75), dt(-1.5)
    got = orc.addmm(A[None], B[None], Y[None], float(alpha), float(beta), nc=1, a_mc=True, b_mc=False)
    P = seq_gemm(A, B, dt)
    want = ((alpha * P).astype(dt) + (beta * np.broadcast_to(Y, (M, N))).astype(dt)).astype(dt)
    assert np.array_equal(got[0], want)


@pytest.mark.parametrize("dt", [np.float16, np.float32])
@pytest.mark.parametrize("nc", [2, 3])
def test_addmm_power_of_two_scaling(orc, dt, nc):
    A, B = inputs.matmul_normal(9, 8, 12, nc, dt, seed=13)
    Y = inputs.split(np.random.default_rng(14).normal(size=(9, 8)), nc, dt)
    P = orc.matmul(A, B[:1], nc=nc, a_mc=True, b_mc=False)
    got = orc.addmm(A, B[:1], Y, 4.0, 0.0, nc=nc)
    want = (P.astype(np.float64) * 4).astype(dt)
    assert np.array_equal(got, want)


@pytest.mark.parametrize("nc", [2, 3])
def test_addmm_row_bias_is_full_bias(orc, nc):
    """A bias of one row (nc, N) means the same as that row repeated for every output
    row (nc, M, N) -- the zero-product case makes it checkable exactly: with alpha = 0
    and beta = 1 the result is Add-MCN(0, Y) = Y for every row (Y compact)."""
    g = np.random.default_rng(18)
    A, B = inputs.matmul_normal(5, 7, 4, nc, np.float32, seed=19)
    Yrow = inputs.split(g.normal(size=(7,)), nc, np.float32)
    got_row = orc.addmm(A, B[:1], Yrow, 0.0, 1.0, nc=nc)
    assert np.array_equal(got_row, np.broadcast_to(Yrow[:, None, :], (nc, 5, 7)))
    Yfull = np.ascontiguousarray(np.broadcast_to(Yrow[:, None, :], (nc, 5, 7)))
    assert np.array_equal(orc.addmm(A, B[:1], Yrow, 0.5, -2.0, nc=nc), orc.addmm(A, B[:1], Yfull, 0.5, -2.0, nc=nc))


@pytest.mark.parametrize("dt", [np.float16, np.float32])
@pytest.mark.parametrize("nc", [2, 3])
def test_addmm_exact_bound(orc, dt, nc):
    M, N, K = 4, 3, 6
    A, B = inputs.matmul_normal(M, N, K, nc, dt, seed=15)
    Y = inputs.split(np.random.default_rng(16).normal(0, 0.3, (M, N)), nc, dt)
    alpha, beta = 0.375, -1.25
    got = orc.addmm(A, B, Y, alpha, beta, nc=nc, a_mc=True, b_mc=True)
    u = 2.0 ** -11 if dt == np.float16 else 2.0 ** -24
    floor = 2 * nc * nc * K * 2.0 ** -25 if dt == np.float16 else 0.0
    F = lambda v: Fraction(float(v))
    for i in range(M):
        for j in range(N):
            ab = sum(sum(F(A[c, i, k]) for c in range(nc)) * sum(F(B[c, k, j]) for c in range(nc)) for k in range(K))
            y = sum(F(Y[c, i, j]) for c in range(nc))
            exact = F(alpha) * ab + F(beta) * y
            absab = sum(abs(sum(F(A[c, i, k]) for c in range(nc))) * abs(sum(F(B[c, k, j]) for c in range(nc)))
                        for k in range(K))
            mag = abs(F(alpha)) * absab + abs(F(beta)) * abs(y)
            err = abs(sum(F(got[c, i, j]) for c in range(nc)) - exact)
            lim = (4 * K + 8) * Fraction(u) ** min(nc, 3) * mag + Fraction(floor)
            assert err <= lim, (i, j, float(err), float(lim))


@pytest.mark.parametrize("nc", [2, 3])
def test_batched_missing_batch_dims_mc(orc, nc):
    """An MC operand with fewer batch dimensions than the result: its planes axis
    stays the planes axis (the result's batch (i1, i2) uses A's matrix i2 for every
    i1), checked slice by slice against the 2-D product on explicitly chosen slices."""
    g = np.random.default_rng(17)
    A = inputs.split(g.normal(size=(4, 6, 5)), nc, np.float32)          # batch (4,)
    B = inputs.split(g.normal(size=(nc, 4, 5, 3)), nc, np.float32)      # batch (nc, 4)
    got = orc.matmul_batched(A, B, nc=nc)
    assert got.shape == (nc, nc, 4, 6, 3)
    for i1 in range(nc):
        for i2 in range(4):
            want = orc.matmul(np.ascontiguousarray(A[:, i2]), np.ascontiguousarray(B[:, i1, i2]), nc=nc)
            assert np.array_equal(got[:, i1, i2], want)
