"""Pins for the oracle's error-free transformations and component exponential.

Two-Sum and Two-Prod (Appendix A.2.1) have closed forms: s = fl(a+b) with
e = (a+b) - s exactly, and p = fl(a*b) with e = fl(a*b - p).  These are checked
against numpy rounding and exact float64 / Fraction arithmetic, exhaustively over
one operand in binary16.  The component exponential is pinned against a 50-digit
decimal exponential over every binary16 input, with a margin check against ties.
"""
import decimal
import math
import os
import re
from fractions import Fraction

import numpy as np
import pytest

F16, F32 = 0, 1
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def parse_value(tok: str) -> float:
    """Parse exact binary expressions such as 1+2^-11, -3*2^-26, -(2-2^-23)."""
    expr = tok.replace("^", "**")
    if not re.fullmatch(r"[0-9+\-*/().e ]+", expr):
        raise ValueError(tok)
    v = eval(expr, {"__builtins__": {}}, {})  # arithmetic only, checked above
    return float(Fraction(v)) if not isinstance(v, float) else v


def _all_finite_f16():
    v = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16).view(np.float16)
    return v[np.isfinite(v)].astype(np.float64)


def test_two_sum_golden_f16(orc):
    rows = []
    for line in open(os.path.join(GOLDEN, "two_sum_f16.txt")):
        line = line.split("#")[0].strip()
        if line:
            rows.append([parse_value(t) for t in line.split()])
    rows = np.array(rows)
    s, e = orc.two_sum(F16, rows[:, 0], rows[:, 1])
    assert (s == rows[:, 2]).all(), (s, rows[:, 2])
    assert (e == rows[:, 3]).all(), (e, rows[:, 3])


def test_two_sum_closed_form_f16(orc):
    """s = fl(a+b) and s + e = a + b exactly, over all finite a and 400 random b."""
    g = np.random.default_rng(10)
    a = _all_finite_f16()
    b = g.choice(a, 400)
    A, B = np.repeat(a, b.size), np.tile(b, a.size)
    with np.errstate(all="ignore"):
        ref_s = (A + B).astype(np.float16).astype(np.float64)
    keep = np.isfinite(ref_s)
    A, B, ref_s = A[keep], B[keep], ref_s[keep]
    s, e = orc.two_sum(F16, A, B)
    assert (s == ref_s).all()
    assert (s + e == A + B).all()  # both sides exact in float64 for binary16 operands
    # and e itself is a binary16 value
    assert (e.astype(np.float16).astype(np.float64) == e).all()


def test_two_sum_closed_form_f32(orc):
    g = np.random.default_rng(11)
    n = 400_000
    a = (np.exp2(g.uniform(-140, 60, n)) * g.choice([-1.0, 1.0], n)).astype(np.float32).astype(np.float64)
    b = (np.exp2(g.uniform(-140, 60, n)) * g.choice([-1.0, 1.0], n)).astype(np.float32).astype(np.float64)
    b[: n // 4] = (a[: n // 4] * np.exp2(-g.integers(0, 40, n // 4))).astype(np.float32)
    s, e = orc.two_sum(F32, a, b)
    ref_s = (a.astype(np.float32) + b.astype(np.float32)).astype(np.float64)
    assert (s == ref_s).all()
    # exactness with rationals on a sample (float64 sums of binary32 may round)
    for i in g.choice(n, 4000, replace=False):
        assert Fraction(s[i]) + Fraction(e[i]) == Fraction(a[i]) + Fraction(b[i])


def test_two_prod_exact_when_representable(orc):
    """a*b = p + e exactly unless the error falls below the subnormal grid."""
    g = np.random.default_rng(12)
    for fmt, dt, lo, hi, tiny in ((F16, np.float16, -6, 6, 2.0 ** -24), (F32, np.float32, -50, 50, 2.0 ** -149)):
        a = (np.exp2(g.uniform(lo, hi, 200_000)) * g.choice([-1.0, 1.0], 200_000)).astype(dt).astype(np.float64)
        b = (np.exp2(g.uniform(lo, hi, 200_000)) * g.choice([-1.0, 1.0], 200_000)).astype(dt).astype(np.float64)
        p, e = orc.two_prod(fmt, a, b)
        exact = a * b  # exact in float64
        rep = np.abs(exact - p) >= tiny * 2 ** 11 if fmt == F16 else np.abs(exact - p) >= tiny * 2 ** 24
        assert (p + e == exact)[rep].all()
        # otherwise e is the rounded error and |a*b - p - e| is at most half the subnormal step
        assert (np.abs(exact - p - e) <= tiny / 2).all()


def _exp16_reference(x: float) -> float:
    """Round e^x to binary16 from a 50-digit decimal exponential, asserting that
    e^x is not within 1e-30 (relative) of a rounding boundary."""
    with decimal.localcontext() as ctx:
        ctx.prec = 50
        E = decimal.Decimal(x).exp()
    Ef = Fraction(E)
    if Ef >= Fraction(65520):
        return math.inf
    # candidates: binary16 values around float(E)
    f = np.float16(float(E))
    cands = set()
    for v in (f, np.nextafter(f, np.float16(np.inf)), np.nextafter(f, np.float16(0))):
        if np.isfinite(v):
            cands.add(Fraction(float(v)))
    best = min(cands, key=lambda c: abs(c - Ef))
    # margin: no other candidate within 1e-30 relative of the same distance
    for c in cands:
        if c != best:
            assert abs(abs(c - Ef) - abs(best - Ef)) > Fraction(1, 10 ** 30) * Ef
    return float(best)


def test_exp_f16_exhaustive_correctly_rounded(orc):
    x = _all_finite_f16()
    got = orc.fl_exp(F16, x)
    # inputs below -17.4 give e^x < 2^-25 (rounds to 0); above 11.1 overflow.  Check
    # every input in between against the decimal reference, and the tails by class.
    mid = (x > -17.5) & (x < 11.2)
    for xi, gi in zip(x[mid], got[mid]):
        assert gi == _exp16_reference(float(xi)), xi
    assert (got[x <= -17.5] == 0).all()
    assert np.isinf(got[x >= 11.2]).all()


def test_exp_f32_sample_correctly_rounded(orc):
    """Binary32 exponential: sample of inputs against the decimal reference."""
    g = np.random.default_rng(13)
    x = g.uniform(-100, 88, 3000).astype(np.float32).astype(np.float64)
    x = np.concatenate([x, g.uniform(-1e-3, 1e-3, 1000).astype(np.float32).astype(np.float64)])
    got = orc.fl_exp(F32, x)
    with decimal.localcontext() as ctx:
        ctx.prec = 60
        for xi, gi in zip(x, got):
            E = Fraction(decimal.Decimal(float(xi)).exp())
            f = np.float32(float(E))
            cands = [Fraction(float(v)) for v in (f, np.nextafter(f, np.float32(np.inf)), np.nextafter(f, np.float32(0)))]
            best = min(cands, key=lambda c: abs(c - E))
            assert Fraction(gi) == best, xi


def test_exp_f32_exhaustive(orc):
    """Every binary32 input with 2^-30 <= |x| <= 105 (outside that range e^x rounds
    to 1, 0 or infinity far from any rounding boundary): the oracle rounds expl's
    long double e^x, whose error (a few long double ulps, about 2^-62 relative) can
    only matter where e^x lies that close to a binary32 rounding boundary.  The scan
    lists every input whose expl value is within 2^-44 of one; all other inputs
    round correctly, and the listed ones are checked against a 60-digit decimal
    exponential, which also shows none lies within 2^-58."""
    n, pats = orc.exp32_near_ties(2.0 ** -44, max_out=8192)
    assert 0 < n <= 8192
    x = pats.view(np.float32).astype(np.float64)
    got = orc.fl_exp(F32, x)
    closest = 1.0
    with decimal.localcontext() as ctx:
        ctx.prec = 60
        for xi, gi in zip(x, got):
            E = Fraction(decimal.Decimal(float(xi)).exp())
            f = np.float32(float(E))
            cands = sorted({Fraction(float(v)) for v in (np.nextafter(f, np.float32(0)), f,
                                                         np.nextafter(f, np.float32(np.inf)))})
            best = min(cands, key=lambda c: abs(c - E))
            assert Fraction(gi) == best, xi
            mids = [(a + b) / 2 for a, b in zip(cands, cands[1:])]
            closest = min(closest, float(min(abs(m - E) for m in mids) / E))
    assert closest > 2.0 ** -58
