"""Pins for the oracle's K-split matrix product.

The K-split product deals the reduction steps round-robin to S slices, sums each
slice in MM-MCN order (Appendix A.2.2) and combines the slice sums with a pairwise
tree of Add-MCN -- a reading of the remark in Section 2.2 that an accurate sum of N
MC values needs depth O(nc log N).  Pins:

  * S = 1 is MM-MCN itself, and so is S = K = 2 (a tree of two leaves is one Add-MCN
    after the first term);
  * nc = 1: every step is one rounding, so the result is a plain float computation
    -- products, slice sums in order, pairwise tree with the odd entry moved up --
    evaluated here with numpy, independently of the oracle; the data are chosen so
    that other slice assignments or tree shapes give different roundings;
  * the error bound against exact rational arithmetic, as for MM-MCN;
  * sampled positions agree with the full product; K = 0 gives +0.
"""
from fractions import Fraction

import numpy as np
import pytest

from paper_2207_08867_amd import inputs

U = {np.float16: 2.0 ** -11, np.float32: 2.0 ** -24}
ETA16 = 2.0 ** -25


def _bits(a):
    a = np.ascontiguousarray(a)
    return a.view(np.uint16 if a.dtype == np.float16 else np.uint32)


@pytest.mark.parametrize("dt,nc,a_mc,b_mc", [
    (np.float32, 2, True, True), (np.float32, 3, True, False), (np.float16, 3, False, True),
])
def test_one_slice_is_mm(orc, dt, nc, a_mc, b_mc):
    g = np.random.default_rng(60)
    M, N, K = 7, 9, 41
    A = inputs.split(g.normal(0, 1, (M, K)), nc if a_mc else 1, dt)
    B = inputs.split(g.normal(0, 1, (K, N)), nc if b_mc else 1, dt)
    ref = orc.matmul(A, B, nc=nc, a_mc=a_mc, b_mc=b_mc)
    got = orc.matmul_splitk(A, B, nc=nc, slices=1, a_mc=a_mc, b_mc=b_mc)
    assert np.array_equal(_bits(got), _bits(ref))


@pytest.mark.parametrize("dt,nc", [(np.float32, 3), (np.float16, 2)])
def test_two_terms_two_slices_is_mm(orc, dt, nc):
    g = np.random.default_rng(61)
    A = inputs.split(g.normal(0, 1, (6, 2)), nc, dt)
    B = inputs.split(g.normal(0, 1, (2, 5)), nc, dt)
    ref = orc.matmul(A, B, nc=nc)
    for S in (2, 3, 100):  # S is capped at K
        assert np.array_equal(_bits(orc.matmul_splitk(A, B, nc=nc, slices=S)), _bits(ref))


def _np_splitk_nc1(A, B, S, tree=True):
    """Plain float K-split product: one rounding per multiply and add (numpy)."""
    dt = A.dtype.type
    M, K = A.shape
    S = min(S, K)
    with np.errstate(all="ignore"):
        parts = []
        for s in range(S):
            acc = None
            for k in range(s, K, S):
                p = (A[:, k, None] * B[None, k, :]).astype(dt)
                acc = p if acc is None else (acc + p).astype(dt)
            parts.append(acc)
        if not tree:  # an alternative combination, to show the data tell orders apart
            acc = parts[0]
            for p in parts[1:]:
                acc = (acc + p).astype(dt)
            return acc
        while len(parts) > 1:
            nxt = [(parts[q] + parts[q + 1]).astype(dt) for q in range(0, len(parts) - 1, 2)]
            if len(parts) % 2:
                nxt.append(parts[-1])
            parts = nxt
    return parts[0]


@pytest.mark.parametrize("dt", [np.float16, np.float32])
def test_nc1_is_plain_float_tree(orc, dt):
    g = np.random.default_rng(62)
    M, N, K = 9, 8, 53
    # mixed magnitudes so that the rounding of each sum depends on the order
    A = (g.uniform(-1, 1, (M, K)) * np.exp2(g.integers(-6, 7, (M, K)))).astype(dt)
    B = g.uniform(-1, 1, (K, N)).astype(dt)
    for S in (2, 3, 5, 7, 8, 13, 53, 80):
        ref = _np_splitk_nc1(A, B, S)
        got = orc.matmul_splitk(A[None], B[None], nc=1, slices=S, b_mc=False)[0]
        assert np.array_equal(_bits(got), _bits(ref)), S
        got2 = orc.matmul_splitk(A[None], B[None], nc=1, slices=S, a_mc=False)[0]
        assert np.array_equal(_bits(got2), _bits(ref)), S
        if S in (5, 13):
            # another tree shape or slice assignment rounds differently on these data
            assert not np.array_equal(_bits(_np_splitk_nc1(A, B, S, tree=False)), _bits(ref))
            assert not np.array_equal(_bits(_np_splitk_nc1(A, B, S + 1)), _bits(ref))


def _fr_sum_planes(P):
    out = np.zeros(P.shape[1:], dtype=object)
    for c in range(P.shape[0]):
        out = out + np.vectorize(lambda v: Fraction(float(v)), otypes=[object])(P[c])
    return out


@pytest.mark.parametrize("dt,nc,S", [
    (np.float32, 2, 3), (np.float32, 3, 8), (np.float32, 3, 30), (np.float16, 2, 5), (np.float16, 3, 8),
])
def test_bound_vs_exact_fractions(orc, dt, nc, S):
    g = np.random.default_rng(63)
    M, N, K = 5, 4, 30
    A = inputs.split(g.normal(0, 1 / np.sqrt(K), (M, K)), nc, dt)
    B = inputs.split(g.normal(0, 1 / np.sqrt(K), (K, N)), nc, dt)
    C = orc.matmul_splitk(A, B, nc=nc, slices=S)
    Af, Bf = _fr_sum_planes(A), _fr_sum_planes(B)
    exact, absab = Af.dot(Bf), np.abs(Af).dot(np.abs(Bf))
    Cf = _fr_sum_planes(C)
    u = Fraction(U[dt])
    floor = Fraction(nc * nc * K) * Fraction(ETA16) if dt == np.float16 else 0
    for i in range(M):
        for j in range(N):
            assert abs(Cf[i, j] - exact[i, j]) <= 4 * K * u ** min(nc, 3) * absab[i, j] + floor


def test_positions_and_empty(orc):
    g = np.random.default_rng(64)
    nc, dt = 3, np.float32
    A, B = inputs.matmul_normal(13, 11, 70, nc, dt, seed=64)
    C = orc.matmul_splitk(A, B, nc=nc, slices=6)
    rows, cols = g.integers(0, 13, 30), g.integers(0, 11, 30)
    assert np.array_equal(_bits(orc.matmul_splitk(A, B, nc=nc, slices=6, rows=rows, cols=cols)),
                          _bits(C[:, rows, cols]))
    Z = orc.matmul_splitk(np.zeros((nc, 3, 0), dt), np.zeros((nc, 0, 4), dt), nc=nc, slices=4)
    assert Z.shape == (nc, 3, 4) and (Z == 0).all() and not np.signbit(Z).any()
