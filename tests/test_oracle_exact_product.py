"""Pins of the exact-product oracle (the MC product rounded into nc binary16
components by successive rounding), against references that share none of its code:

* the rounding: numpy's float64 -> float16 conversion (IEEE round-to-nearest-even
  with gradual underflow) on values that are exact in float64, including ties,
  the subnormal range and the overflow threshold;
* the exact sums: Python fractions over the components, term by term;
* identity: I x B returns B's components whenever B is a canonical expansion
  (each later part below a quarter ulp of the one before);
* the successive split: exact when P has at most 11 nc significant bits in range,
  otherwise within half an ulp of the last component, never overlapping;
* the paper's MM-MCN bound (4 K u^nc sum |A||B|, Section 2.4) holds with large
  room, and the MM-MCN oracle agrees within that bound;
* non-finite inputs and overflow follow the stated readings.
"""
from fractions import Fraction

import numpy as np
import pytest

from oracle import exact_product as xp
from paper_2207_08867_amd import inputs

U = 2.0 ** -11


def f16_bits(v):
    return np.array([v], dtype=np.float16).view(np.uint16)[0]


def test_round_matches_numpy_on_exact_doubles():
    g = np.random.default_rng(1)
    vals = []
    for _ in range(20000):
        m = int(g.integers(1, 1 << 53))
        if g.random() < 0.3:
            m >>= int(g.integers(0, 50))
            m = max(m, 1)
        s = int(g.integers(0, 45))
        v = m << s
        vals.append(-v if g.random() < 0.5 else v)
    # ties at every quantum, the subnormal floor and the overflow threshold
    for qe in range(24, 70):
        for n in (1, 2, 3, 1023, 1024, 2047):
            vals += [(2 * n + 1) << (qe - 1), -((2 * n + 1) << (qe - 1))]
    vals += [1 << 23, 3 << 23, (1 << 23) - 1, (1 << 23) + 1, 65504 << 48, 65519 << 48, 65520 << 48]
    for v in vals:
        assert (abs(v) >> max(abs(v).bit_length() - 53, 0)) << max(abs(v).bit_length() - 53, 0) == abs(v)
        bits, val = xp.round_units48(v)
        with np.errstate(over="ignore"):
            want = f16_bits(float(v) * 2.0 ** -48)
        assert bits == want, (v, hex(bits), hex(want))
        if val is not None:
            assert Fraction(val, 1 << 48) == Fraction(float(np.array([bits], np.uint16).view(np.float16)[0]))
    # values with more bits than float64 holds, on either side of the overflow threshold
    assert xp.round_units48((65520 << 48) - 1) == (0x7BFF, 65504 << 48)
    assert xp.round_units48(-((65520 << 48) - 1)) == (0xFBFF, -(65504 << 48))
    assert xp.round_units48(1 << 100)[0] == 0x7C00 and xp.round_units48(-(1 << 100))[0] == 0xFC00
    # 2^14 (1 + 2^-11 + 2^-62): just above a tie, by a bit float64 would drop -> rounds up
    assert xp.round_units48((1 << 62) + (1 << 51) + 1) == (0x7401, 1025 << 52)
    assert xp.round_units48((1 << 62) + (1 << 51)) == (0x7400, 1 << 62)  # the tie itself goes to even


def test_exact_sums_against_fractions():
    g = np.random.default_rng(2)
    for nc in (1, 2, 3, 4):
        A = inputs.split(g.normal(0, 3.0, (3, 5)) * np.exp2(g.integers(-20, 8, (3, 5))), nc, np.float16)
        B = inputs.split(g.normal(0, 1.0, (5, 4)) * np.exp2(g.integers(-20, 8, (5, 4))), nc, np.float16)
        P, rb, cb = xp.exact_sums(A, B)
        assert not rb.any() and not cb.any()
        for i in range(3):
            for j in range(4):
                want = sum(Fraction(float(A[a, i, k])) * Fraction(float(B[b, k, j]))
                           for k in range(5) for a in range(nc) for b in range(nc))
                assert Fraction(P[i, j], 1 << 48) == want


def canonical(g, shape, nc):
    """Expansions whose later parts stay below a quarter ulp of the part before."""
    out = np.zeros((nc,) + shape, dtype=np.float16)
    out[0] = g.uniform(-4, 4, shape).astype(np.float16)
    for c in range(1, nc):
        prev = out[c - 1].astype(np.float64)
        ulp = np.exp2(np.floor(np.log2(np.maximum(np.abs(prev), 2.0 ** -14))) - 10)
        v = (g.uniform(-0.25, 0.25, shape) * ulp).astype(np.float16)
        v = np.where(np.abs(v.astype(np.float64)) < 0.25 * ulp, v, np.float16(0))
        out[c] = np.where(prev == 0, np.float16(0), v)
    return out + np.float16(0)  # -0 + +0 = +0: an exact zero part is +0


@pytest.mark.parametrize("nc", [1, 2, 3])
def test_identity_returns_canonical_expansions(nc):
    g = np.random.default_rng(3)
    B = canonical(g, (6, 7), nc)
    A = np.zeros((nc, 6, 6), dtype=np.float16)
    A[0] = np.eye(6, dtype=np.float16)
    got = xp.matmul_exact(A, B, nc=nc)
    assert np.array_equal(got.view(np.uint16), B.view(np.uint16))


def frac16(v):
    return Fraction(float(v))


def ulp16(v):
    a = abs(float(v))
    if a < 2.0 ** -14:
        return Fraction(1, 1 << 24)
    e = int(np.floor(np.log2(a)))
    return Fraction(2) ** (e - 10)


@pytest.mark.parametrize("nc", [1, 2, 3, 4])
def test_split_properties_and_paper_bound(orc, nc):
    M, N, K = 6, 5, 40
    A, B = inputs.matmul_normal(M, N, K, nc, np.float16, seed=4)
    got = xp.matmul_exact(A, B, nc=nc)
    mm = orc.matmul(A, B, nc=nc)
    P, _, _ = xp.exact_sums(A, B)
    for i in range(M):
        for j in range(N):
            exact = Fraction(P[i, j], 1 << 48)
            comps = [frac16(got[c, i, j]) for c in range(nc)]
            err = abs(sum(comps) - exact)
            # within half an ulp of the last component (or the half subnormal quantum)
            assert err <= ulp16(got[nc - 1, i, j]) / 2
            # non-overlapping: each component at most half an ulp of the one before
            for c in range(1, nc):
                if comps[c] != 0:
                    assert abs(comps[c]) <= ulp16(got[c - 1, i, j]) / 2
            absab = sum(abs(sum(frac16(A[c, i, k]) for c in range(nc))) * abs(sum(frac16(B[c, k, j]) for c in range(nc)))
                        for k in range(K))
            bound = 4 * K * Fraction(U) ** nc * absab + nc * K * Fraction(1, 1 << 25)
            assert err <= bound / 64
            mm_err = abs(sum(frac16(mm[c, i, j]) for c in range(nc)) - exact)
            assert mm_err <= bound


@pytest.mark.parametrize("nc", [2, 3])
def test_exact_when_representable(nc):
    """Small integers: P is an integer of a few bits, so c_0 = P and the rest are +0."""
    g = np.random.default_rng(5)
    A = np.zeros((nc, 5, 9), np.float16)
    B = np.zeros((nc, 9, 4), np.float16)
    A[0] = g.integers(-8, 9, (5, 9))
    B[0] = g.integers(-8, 9, (9, 4))
    got = xp.matmul_exact(A, B, nc=nc)
    want = A[0].astype(np.float64) @ B[0].astype(np.float64)
    assert np.array_equal(got[0].astype(np.float64), want)
    assert np.array_equal(got[1:].view(np.uint16), np.zeros_like(got[1:]).view(np.uint16))


def test_two_components_hold_22_bits():
    """1 + 2^-20 needs two binary16 components: (1, 2^-20); with nc = 1 it rounds to 1."""
    A = np.zeros((2, 1, 2), np.float16)
    B = np.zeros((2, 2, 1), np.float16)
    A[0, 0] = [1.0, 2.0 ** -10]
    B[0, :, 0] = [1.0, 2.0 ** -10]
    got = xp.matmul_exact(A, B, nc=2)
    assert got[0, 0, 0] == 1.0 and got[1, 0, 0] == np.float16(2.0 ** -20)
    got1 = xp.matmul_exact(A[:1], B[:1], nc=1)
    assert got1[0, 0, 0] == 1.0


def test_nonfinite_and_overflow():
    A = np.ones((2, 3, 4), np.float16) * np.float16(0.5)
    A[1] = 0
    B = np.ones((2, 4, 3), np.float16)
    B[1] = 0
    A[1, 1, 2] = np.inf         # row 1 of A
    B[0, 3, 2] = np.nan         # column 2 of B
    got = xp.matmul_exact(A, B, nc=2)
    nan = np.isnan(got)
    want = np.zeros((3, 3), bool)
    want[1, :] = True
    want[:, 2] = True
    assert np.array_equal(nan[0], want) and np.array_equal(nan[1], want)
    assert np.all(got[0][~want] == 2.0) and np.all(got[1][~want] == 0)
    big = np.full((1, 2, 3), 60000, np.float16)
    got = xp.matmul_exact(big, np.full((1, 3, 2), 2, np.float16), nc=3, a_mc=False, b_mc=False)
    assert np.all(np.isposinf(got[0])) and not got[1:].any()


def test_positions_match_full():
    A, B = inputs.matmul_normal(7, 9, 33, 3, np.float16, seed=6)
    full = xp.matmul_exact(A, B, nc=3)
    r = np.array([0, 6, 3, 2])
    c = np.array([8, 0, 4, 4])
    part = xp.matmul_exact(A, B, nc=3, rows=r, cols=c)
    assert np.array_equal(part.view(np.uint16), full[:, r, c].view(np.uint16))


def test_plain_operands():
    """A plain (one-component) operand is the MC operand with zero later components."""
    A, B = inputs.matmul_normal(4, 5, 12, 3, np.float16, seed=7)
    A1 = A.copy()
    A1[1:] = 0
    got = xp.matmul_exact(A[:1], B, nc=3, a_mc=False)
    assert np.array_equal(got.view(np.uint16), xp.matmul_exact(A1, B, nc=3).view(np.uint16))


@pytest.mark.parametrize("nc", [1, 2, 3])
def test_bias_alone_returns_canonical_bias(nc):
    """A = 0: the exact value is the bias itself, split back into its own components."""
    g = np.random.default_rng(8)
    b = canonical(g, (9,), nc)
    A = np.zeros((nc, 4, 6), np.float16)
    B = canonical(g, (6, 9), nc)
    got = xp.matmul_exact(A, B, nc=nc, bias=b)
    assert np.array_equal(got.view(np.uint16), np.broadcast_to(b[:, None, :], got.shape).view(np.uint16))


@pytest.mark.parametrize("nc", [2, 3])
def test_bias_is_an_extra_reduction_term(nc):
    """x W^T + b equals the bias-free exact product of [A | 1] and [B ; b]."""
    A, B = inputs.matmul_normal(5, 7, 11, nc, np.float16, seed=9)
    b = inputs.split(np.random.default_rng(10).normal(0, 0.5, 7), nc, np.float16)
    b[:, 2] = [np.float16(3000.0)] + [np.float16(0)] * (nc - 1)
    A1 = np.concatenate([A, np.zeros((nc, 5, 1), np.float16)], axis=2)
    A1[0, :, -1] = 1
    B1 = np.concatenate([B, b[:, None, :]], axis=1)
    got = xp.matmul_exact(A, B, nc=nc, bias=b)
    assert np.array_equal(got.view(np.uint16), xp.matmul_exact(A1, B1, nc=nc).view(np.uint16))
    r, c = np.array([0, 4, 2]), np.array([6, 2, 0])
    assert np.array_equal(xp.matmul_exact(A, B, nc=nc, bias=b, rows=r, cols=c).view(np.uint16),
                          got[:, r, c].view(np.uint16))


def test_nonfinite_bias_column():
    A, B = inputs.matmul_normal(3, 4, 5, 2, np.float16, seed=11)
    b = np.zeros((2, 4), np.float16)
    b[1, 3] = np.inf
    got = xp.matmul_exact(A, B, nc=2, bias=b)
    assert np.isnan(got[:, :, 3]).all() and not np.isnan(got[:, :, :3]).any()
