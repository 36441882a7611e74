"""Pins for the oracle's number model (component rounding and basic operations).

The oracle rounds every step into the component format itself (round_to() in
oracle/mcf_oracle.c, written from the IEEE-754 definition).  These tests pin it to
independent library routines:
  * numpy's float64 -> float16 / float32 conversion (round to nearest even, gradual
    underflow, overflow to inf);
  * numpy's float16 / float32 array arithmetic (IEEE + - * / on x86 SSE; float16
    ops are evaluated in float32 and rounded, which is innocuous for these four
    operations because 24 >= 2*11 + 2);
  * exact float64 arithmetic for the Two-Prod error.
"""
import numpy as np
import pytest

F16, F32 = 0, 1


def _same(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    both_nan = np.isnan(a) & np.isnan(b)
    eq = (a == b) & (np.signbit(a) == np.signbit(b))
    return eq | both_nan


def _all_f16():
    return np.arange(1 << 16, dtype=np.uint32).astype(np.uint16).view(np.float16)


def test_f16_decode_encode_all_encodings(orc):
    L = orc.lib()
    h = np.arange(1 << 16, dtype=np.uint32)
    dec = np.array([L.mcf_oracle_f16_decode(int(v)) for v in h])
    ref = h.astype(np.uint16).view(np.float16).astype(np.float64)
    assert _same(dec, ref).all()
    fin = np.isfinite(ref) | np.isinf(ref)
    enc = np.array([L.mcf_oracle_f16_encode(float(v)) for v in ref[fin]], dtype=np.uint32)
    assert (enc == h[fin]).all()


def test_round_f16_every_value_and_midpoint(orc):
    v = _all_f16().astype(np.float64)
    v = v[np.isfinite(v)]
    assert _same(orc.fl_round(F16, v), v).all()
    # midpoints between consecutive non-negative finite binary16 values, both signs,
    # and points a hair above / below each midpoint
    pos = np.unique(np.abs(v))
    mids = (pos[:-1] + pos[1:]) / 2  # exact in float64
    for pts in (mids, np.nextafter(mids, np.inf), np.nextafter(mids, -np.inf)):
        for s in (1.0, -1.0):
            x = s * pts
            with np.errstate(over="ignore"):
                ref = x.astype(np.float16).astype(np.float64)
            assert _same(orc.fl_round(F16, x), ref).all()
    # overflow threshold: 65520 is the tie between 65504 and 2^16 -> inf
    assert np.isinf(orc.fl_round(F16, [65520.0]))[0]
    assert orc.fl_round(F16, [np.nextafter(65520.0, 0)])[0] == 65504.0


def test_round_f16_random_log_uniform(orc):
    g = np.random.default_rng(1)
    x = np.exp2(g.uniform(-30, 17, 2_000_000)) * g.choice([-1.0, 1.0], 2_000_000)
    with np.errstate(over="ignore"):
        ref = x.astype(np.float16).astype(np.float64)
    assert _same(orc.fl_round(F16, x), ref).all()


def test_round_f32_random_and_midpoints(orc):
    g = np.random.default_rng(2)
    x = np.exp2(g.uniform(-160, 130, 2_000_000)) * g.choice([-1.0, 1.0], 2_000_000)
    with np.errstate(over="ignore"):
        ref = x.astype(np.float32).astype(np.float64)
    assert _same(orc.fl_round(F32, x), ref).all()
    # exact ties between random neighbouring binary32 values (normal and subnormal)
    bits = g.integers(0, 0x7F7FFFFF, 1_000_000, dtype=np.int64).astype(np.uint32)
    a = bits.view(np.float32).astype(np.float64)
    b = (bits + 1).view(np.float32).astype(np.float64)
    mids = (a + b) / 2
    for pts in (mids, np.nextafter(mids, np.inf), np.nextafter(mids, -np.inf)):
        with np.errstate(over="ignore"):
            ref = pts.astype(np.float32).astype(np.float64)
        assert _same(orc.fl_round(F32, pts), ref).all()
        assert _same(orc.fl_round(F32, -pts), -ref).all()


def _finite_f16_sample(g, n):
    v = g.integers(0, 1 << 16, n, dtype=np.int64).astype(np.uint16).view(np.float16)
    return v[np.isfinite(v)]


@pytest.mark.parametrize("op", ["add", "sub", "mul", "div"])
def test_f16_ops_vs_numpy(orc, op):
    g = np.random.default_rng(3)
    a = _all_f16()
    a = a[np.isfinite(a)]
    b = _finite_f16_sample(g, 300)
    A = np.repeat(a, b.size)
    B = np.tile(b, a.size)
    if op == "div":
        keep = B != 0
        A, B = A[keep], B[keep]
    with np.errstate(all="ignore"):
        ref = {"add": A + B, "sub": A - B, "mul": A * B, "div": A / B}[op].astype(np.float64)
    fn = {"add": orc.fl_add, "sub": orc.fl_sub, "mul": orc.fl_mul, "div": orc.fl_div}[op]
    got = fn(F16, A.astype(np.float64), B.astype(np.float64))
    assert _same(got, ref).all()


@pytest.mark.parametrize("op", ["add", "sub", "mul", "div"])
def test_f32_ops_vs_numpy(orc, op):
    g = np.random.default_rng(4)
    n = 2_000_000
    # mixed exponents, subnormals included
    a = (np.exp2(g.uniform(-150, 60, n)) * g.choice([-1.0, 1.0], n)).astype(np.float32)
    b = (np.exp2(g.uniform(-150, 60, n)) * g.choice([-1.0, 1.0], n)).astype(np.float32)
    # and near-cancelling pairs
    b[: n // 4] = -a[: n // 4] * (1 + np.float32(2.0 ** -20) * g.integers(-8, 8, n // 4).astype(np.float32))
    with np.errstate(all="ignore"):
        ref = {"add": a + b, "sub": a - b, "mul": a * b, "div": a / b}[op].astype(np.float64)
    fn = {"add": orc.fl_add, "sub": orc.fl_sub, "mul": orc.fl_mul, "div": orc.fl_div}[op]
    got = fn(F32, a.astype(np.float64), b.astype(np.float64))
    assert _same(got, ref).all()


def test_two_prod_error_f16(orc):
    """e = fl(a*b - fl(a*b)): a*b and a*b - p are exact in float64 for binary16."""
    g = np.random.default_rng(5)
    a = _all_f16()
    a = a[np.isfinite(a)]
    b = _finite_f16_sample(g, 200)
    A = np.repeat(a, b.size).astype(np.float64)
    B = np.tile(b, a.size).astype(np.float64)
    with np.errstate(all="ignore"):
        p = (A * B).astype(np.float16).astype(np.float64)
        keep = np.isfinite(p)
        A, B, p = A[keep], B[keep], p[keep]
        ref = (A * B - p).astype(np.float16).astype(np.float64)
    assert _same(orc.two_prod_err(F16, A, B), ref).all()


def test_two_prod_error_f32(orc):
    """For binary32, a*b (48 bits) and a*b - p are exact in float64."""
    g = np.random.default_rng(6)
    n = 2_000_000
    a = (np.exp2(g.uniform(-100, 50, n)) * g.choice([-1.0, 1.0], n)).astype(np.float32).astype(np.float64)
    b = (np.exp2(g.uniform(-100, 50, n)) * g.choice([-1.0, 1.0], n)).astype(np.float32).astype(np.float64)
    with np.errstate(all="ignore"):
        p = (a * b).astype(np.float32).astype(np.float64)
        keep = np.isfinite(p)
        a, b, p = a[keep], b[keep], p[keep]
        ref = (a * b - p).astype(np.float32).astype(np.float64)
    assert _same(orc.two_prod_err(F32, a, b), ref).all()


def test_fma_tie_uses_remainder(orc):
    """fl(fma(a, b, c)) when the double sum a*b + c rounds onto a binary32 tie.

    a = 3 and b = 5592407 * 2^-24 give a*b = 1 + 2^-22 + 2^-24 exactly, the tie
    between 1 + 2^-22 (even) and 1 + 2^-22 + 2^-23.  Adding c = +-2^-100 leaves the
    double sum on the tie, so only the remainder can decide the direction."""
    fma = orc.lib().mcf_oracle_fl_fma
    a, b = 3.0, 5592407 * 2.0 ** -24
    assert a * b == 1 + 2.0 ** -22 + 2.0 ** -24
    assert fma(F32, a, b, 0.0) == 1 + 2.0 ** -22  # tie, to even
    assert fma(F32, a, b, 2.0 ** -100) == 1 + 2.0 ** -22 + 2.0 ** -23
    assert fma(F32, a, b, -(2.0 ** -100)) == 1 + 2.0 ** -22
    assert fma(F32, -a, b, -(2.0 ** -100)) == -(1 + 2.0 ** -22 + 2.0 ** -23)
