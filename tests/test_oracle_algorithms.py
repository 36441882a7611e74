"""Pins for the oracle's MC algorithms (Appendix A.2.1 and Section 2.1).

Each algorithm is checked against facts that do not come from the oracle itself:
  * brute force of a trivial specification (Simple-Renorm);
  * textbook reductions at nc = 1 and nc = 2 (Add-MCN, Grow-ExpN, ScalingN,
    Div-MCN, Mult-MCN, Exp-MCN collapse to a single rounded operation, Two-Sum or
    Two-Prod, evaluated here with numpy);
  * exact identities (division and multiplication by powers of two, x/x, exp of a
    one-component value);
  * error bounds against exact rational arithmetic (Python Fractions), at input
    magnitudes where the component format's subnormal floor does not mask a
    dropped or mis-indexed term;
  * invariants of Renormalize (exact sum preservation, non-overlap) and the
    hand-derived fixtures in tests/golden/.
"""
import itertools
import os
from fractions import Fraction

import numpy as np
import pytest

from paper_2207_08867_amd.inputs import split

F16, F32 = 0, 1
U = {np.float16: 2.0 ** -11, np.float32: 2.0 ** -24}
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _fr(v) -> Fraction:
    return Fraction(float(v))


def exact_vals(planar, idx):
    """Exact value (Fraction) of elements idx of a planar MC array."""
    return [sum((_fr(planar[c, i]) for c in range(planar.shape[0])), Fraction(0)) for i in idx]


def bits_equal(a, b):
    a = np.asarray(a)
    b = np.asarray(b)
    ua = a.view(np.uint16 if a.dtype == np.float16 else np.uint32)
    ub = b.view(np.uint16 if b.dtype == np.float16 else np.uint32)
    return np.array_equal(ua, ub)


def value_equal(a, b):
    """Componentwise equality with +0 == -0 (zero signs are not part of the contract)."""
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return bool(((a == b) | (np.isnan(a) & np.isnan(b))).all())


# ---------------------------------------------------------------------------------
# Simple-Renorm
# ---------------------------------------------------------------------------------

@pytest.mark.parametrize("m", [1, 2, 3, 4, 5])
def test_simple_renorm_brute_force(orc, m):
    g = np.random.default_rng(20)
    pats = list(itertools.product([0, 1], repeat=m))
    h = np.zeros((m, len(pats)), dtype=np.float32)
    for j, p in enumerate(pats):
        for i, nz in enumerate(p):
            h[i, j] = np.float32(g.uniform(0.5, 2.0) * g.choice([-1, 1])) if nz else (np.float32(-0.0) if (i + j) % 2 else 0)
    for r in range(1, m + 1):
        out = orc.renorm(h, nc=m, nc_out=r, mode=1)
        for j in range(len(pats)):
            nz = [float(h[i, j]) for i in range(m) if h[i, j] != 0][:r]
            spec = nz + [0.0] * (r - len(nz))
            assert list(out[:, j].astype(np.float64)) == spec
            # padding is +0
            assert not np.signbit(out[len(nz):, j]).any()


# ---------------------------------------------------------------------------------
# nc = 1 and nc = 2 reductions
# ---------------------------------------------------------------------------------

@pytest.mark.parametrize("dt", [np.float16, np.float32])
def test_nc1_reductions(orc, dt):
    g = np.random.default_rng(21)
    n = 200_000
    x = g.uniform(-4, 4, n).astype(dt)
    y = g.uniform(0.25, 4, n).astype(dt) * g.choice([-1, 1], n).astype(dt)
    X, Y = x[None], y[None]
    with np.errstate(all="ignore"):
        assert value_equal(orc.add(X, Y, nc=1)[0], x + y)
        assert value_equal(orc.add(X, y, nc=1, y_mc=False)[0], x + y)
        assert value_equal(orc.add(x, Y, nc=1, x_mc=False)[0], x + y)
        assert value_equal(orc.mul(X, y, nc=1, y_mc=False)[0], x * y)
        assert value_equal(orc.div(X, Y, nc=1)[0], x / y)
        # Mult-MCN at nc = 1 is x / fl(1/y), not fl(x*y)
        assert value_equal(orc.mul(X, Y, nc=1)[0], x / (dt(1) / y))
        assert value_equal(orc.exp(X, nc=1)[0], orc.fl_exp(F16 if dt == np.float16 else F32, x).astype(dt))
        assert value_equal(orc.renorm(X, nc=1)[0], x)


@pytest.mark.parametrize("dt,fmt", [(np.float16, F16), (np.float32, F32)])
def test_nc2_reduce_to_eft(orc, dt, fmt):
    g = np.random.default_rng(22)
    n = 100_000
    a = (g.uniform(-8, 8, n) * np.exp2(g.integers(-6, 6, n))).astype(dt)
    b = (g.uniform(-8, 8, n) * np.exp2(g.integers(-6, 6, n))).astype(dt)
    A = np.stack([a, np.zeros_like(a)])
    B = np.stack([b, np.zeros_like(b)])
    s, e = orc.two_sum(fmt, a, b)
    ts = np.stack([np.where(s != 0, s, e), np.where(s != 0, e, 0)]).astype(dt)
    assert value_equal(orc.add(A, B, nc=2), ts)
    assert value_equal(orc.add(A, b, nc=2, y_mc=False), ts)
    p, pe = orc.two_prod(fmt, a, b)
    tp = np.stack([np.where(p != 0, p, pe), np.where(p != 0, pe, 0)]).astype(dt)
    assert value_equal(orc.mul(A, b, nc=2, y_mc=False), tp)
    assert value_equal(orc.mul(a, B, nc=2, x_mc=False), tp)


# ---------------------------------------------------------------------------------
# exact identities
# ---------------------------------------------------------------------------------

@pytest.mark.parametrize("dt,nc", [(np.float32, 2), (np.float32, 3), (np.float16, 2), (np.float16, 3)])
def test_identities(orc, dt, nc):
    g = np.random.default_rng(23)
    n = 20_000
    scale = 100.0 if dt == np.float32 else 20000.0  # keeps most binary16 third components normal
    x = split(g.uniform(-scale, scale, n), nc, dt)
    # Mult-MCN ends with Renormalize, which rewrites a representation whose next
    # component is exactly half an ulp of the previous one (a tie) into the even
    # neighbour: same value, other components.  Those elements are compared by value.
    tie = np.zeros(n, dtype=bool)
    for c in range(nc - 1):
        tie |= np.abs(x[c + 1].astype(np.float64)) == _ulp(x[c], dt) / 2
    tiny = np.finfo(dt).tiny  # scaling below the normal range would round the identity away
    for k in ((-3, 0, 2) if dt == np.float32 else (-1, 0, 1)):  # binary16: stay below 65504
        p2 = np.zeros((nc, n), dtype=dt)
        p2[0] = dt(2.0 ** k)
        ok = ~((np.abs(x.astype(np.float64)) * 2.0 ** -abs(k) < tiny) & (x != 0)).any(0)
        d = orc.div(x, p2, nc=nc)
        assert value_equal(d[:, ok], (x.astype(np.float64) * 2.0 ** -k).astype(dt)[:, ok])
        m = orc.mul(x, p2, nc=nc)
        ref = (x.astype(np.float64) * 2.0 ** k).astype(dt)
        assert value_equal(m[:, ok & ~tie], ref[:, ok & ~tie])
        t = np.where(ok & tie)[0]
        assert exact_vals(m, t) == exact_vals(ref, t)
        assert ok.sum() > n // 2
    one = np.zeros((nc, n), dtype=dt)
    one[0] = 1
    assert value_equal(orc.div(x, x, nc=nc), one)
    zero = np.zeros((nc, n), dtype=dt)
    assert value_equal(orc.add(x, zero, nc=nc), x)
    e0 = np.zeros((nc, n), dtype=dt)
    e0[0] = g.uniform(-4, 4, n).astype(dt)
    ref = np.zeros((nc, n), dtype=dt)
    ref[0] = orc.fl_exp(F16 if dt == np.float16 else F32, e0[0]).astype(dt)
    assert value_equal(orc.exp(e0, nc=nc), ref)


# ---------------------------------------------------------------------------------
# error bounds against exact arithmetic
# ---------------------------------------------------------------------------------

# Magnitudes keep every component well above the subnormal floor, so a dropped or
# mis-indexed term shows up as an error of order u^(nc-1) instead of u^nc.
CASES = [(np.float32, 2, 1.0), (np.float32, 3, 1.0), (np.float16, 2, 3000.0), (np.float16, 3, 3000.0)]


def _mc(g, n, nc, dt, scale, lo=None):
    v = g.uniform(-scale, scale, n)
    if lo is not None:
        v = np.sign(v) * (lo + np.abs(v))
    return split(v, nc, dt)


@pytest.mark.parametrize("dt,nc,scale", CASES)
def test_add_scaling_error_bounds(orc, dt, nc, scale):
    """Add-MCN and ScalingN drop only their final carry (order u^nc of the inputs)
    plus carry roundings of smaller order."""
    g = np.random.default_rng(24)
    n = 3000
    u = Fraction(U[dt])
    x = _mc(g, n, nc, dt, scale)
    y = _mc(g, n, nc, dt, scale)
    v = g.uniform(-4, 4, n).astype(dt)
    idx = range(n)
    X, Y = exact_vals(x, idx), exact_vals(y, idx)
    V = [_fr(t) for t in v]
    r_add = exact_vals(orc.add(x, y, nc=nc), idx)
    r_scal = exact_vals(orc.mul(x, v, nc=nc, y_mc=False), idx)
    r_scal2 = exact_vals(orc.mul(v, x, nc=nc, x_mc=False), idx)
    # binary16: a Two-Prod error below the subnormal grid is lost (at most half the
    # smallest subnormal, eta = 2^-25, per component product)
    eta = Fraction(2) ** -25 if dt == np.float16 else Fraction(0)
    worst = 0
    for i in idx:
        assert abs(r_add[i] - (X[i] + Y[i])) <= 8 * u ** nc * (abs(X[i]) + abs(Y[i])), i
        assert abs(r_scal[i] - X[i] * V[i]) <= 8 * u ** nc * abs(X[i] * V[i]) + nc * eta, i
        assert r_scal2[i] == r_scal[i]
        if X[i] * V[i]:
            worst = max(worst, abs(r_scal[i] - X[i] * V[i]) / abs(X[i] * V[i]) / u ** nc)
    assert worst > Fraction(1, 100)  # the bound is within a small factor of what occurs


@pytest.mark.parametrize("dt,nc,scale", CASES)
def test_grow_expn_drops_only_last_term(orc, dt, nc, scale):
    """Grow-ExpN is a chain of exact Two-Sums from the last component up; Simple-Renorm
    then keeps the first nc of the nc+1 terms, so the only loss is the error term of
    Two-Sum(x_{nc-1}, v), at most u |x_{nc-1} + v| (none when a term is zero).  Two
    regimes of v: comparable to x, and far below x_0 (where dropping any other term
    would exceed the bound by orders of magnitude)."""
    g = np.random.default_rng(29)
    n = 3000
    u = Fraction(U[dt])
    x = _mc(g, n, nc, dt, scale)
    for vscale in (scale, scale * 2.0 ** -8):
        v = g.uniform(-vscale, vscale, n).astype(dt)
        r = orc.add(x, v, nc=nc, y_mc=False)
        assert np.array_equal(r, orc.add(v, x, nc=nc, x_mc=False))
        got = exact_vals(r, range(n))
        X = exact_vals(x, range(n))
        for i in range(n):
            ex = X[i] + _fr(v[i])
            assert abs(got[i] - ex) <= u * abs(_fr(x[nc - 1, i]) + _fr(v[i])), i


@pytest.mark.parametrize("dt,nc", [(np.float32, 2), (np.float32, 3), (np.float16, 2)])
def test_div_mult_error_bounds(orc, dt, nc):
    """Div-MCN as printed divides only the leading remainder component by y_0, and
    Add-MCN / Simple-Renorm leave the remainder's components overlapping, so a
    fraction of the inputs come out only about u-accurate (at most a few u) while
    the typical element reaches u^nc.  Pinned: every element within 4u of x/y (resp.
    x*y), the median within 2 u^nc, and DivN equal to Div-MCN with a zero-padded
    dividend.  A dropped digit, a wrong sign or index moves the median by orders
    of magnitude."""
    g = np.random.default_rng(25)
    n = 4000
    u = U[dt]
    sx, sy = (1.0, 1.0) if dt == np.float32 else (8.0, 4.0)
    x = _mc(g, n, nc, dt, sx)
    y = _mc(g, n, nc, dt, sy * 0.5, lo=sy * 0.5)
    X = orc.exact_diff(x)
    Y = orc.exact_diff(y)
    for res, ref in ((orc.div(x, y, nc=nc), X / Y), (orc.mul(x, y, nc=nc), X * Y)):
        rel = np.abs(orc.exact_diff(res) - ref) / np.abs(ref)
        assert rel.max() <= 4 * u
        assert np.median(rel) <= 2 * u ** nc
    # exact check of the worst element with rationals (the float64 quotient above is
    # itself rounded at 2^-53 relative, below u^nc only for binary16)
    q = orc.div(x, y, nc=nc)
    k = int(np.argmax(np.abs(orc.exact_diff(q) - X / Y) / np.abs(X / Y)))
    ex = exact_vals(x, [k])[0] / exact_vals(y, [k])[0]
    assert abs(exact_vals(q, [k])[0] - ex) <= 4 * Fraction(u) * abs(ex)
    v = g.uniform(1, 3, n).astype(dt)
    padded = np.zeros((nc, n), dtype=dt)
    padded[0] = v
    assert np.array_equal(orc.div(v, y, nc=nc, x_mc=False), orc.div(padded, y, nc=nc))


@pytest.mark.parametrize("dt,nc", [(np.float32, 2), (np.float32, 3), (np.float16, 2), (np.float16, 3)])
def test_exp_error_bound(orc, dt, nc):
    """Exp-MCN equals the product of the component exponentials up to the carry
    roundings of the ScalingN chain."""
    g = np.random.default_rng(26)
    n = 2000
    fmt = F16 if dt == np.float16 else F32
    x = split(g.uniform(-4, 4, n), nc, dt)
    if dt == np.float16:  # make lower components large enough that exp(x_i) != 1
        x[1:] = g.uniform(-0.5, 0.5, (nc - 1, n)).astype(dt)
    r = exact_vals(orc.exp(x, nc=nc), range(n))
    u = Fraction(U[dt])
    eta = Fraction(2) ** -25 if dt == np.float16 else Fraction(0)  # binary16 subnormal floor
    E = [orc.fl_exp(fmt, x[c]) for c in range(nc)]
    for i in range(n):
        prod = Fraction(1)
        for c in range(nc):
            prod *= _fr(E[c][i])
        assert abs(r[i] - prod) <= 8 * u ** nc * prod + nc * eta, i


# ---------------------------------------------------------------------------------
# Renormalize
# ---------------------------------------------------------------------------------

def _ulp(v, dt):
    v = np.abs(np.asarray(v, dtype=dt))
    return (np.nextafter(v, dt(np.inf)) - v).astype(np.float64)


def test_renormalize_golden(orc):
    for line in open(os.path.join(GOLDEN, "renormalize_f32.txt")):
        line = line.split("#")[0].strip()
        if not line:
            continue
        from test_oracle_eft import parse_value

        lhs, rhs = line.split(";")
        xin = [parse_value(t) for t in lhs.split()]
        want = [parse_value(t) for t in rhs.split()]
        x = np.array(xin, dtype=np.float32)[:, None]
        got = orc.renorm(x, nc=len(xin), mode=0)[:, 0]
        assert list(got.astype(np.float64)) == want, (xin, got)


@pytest.mark.parametrize("dt,nc", [(np.float32, 2), (np.float32, 3), (np.float32, 4), (np.float16, 3)])
def test_renormalize_invariants(orc, dt, nc):
    g = np.random.default_rng(27)
    n = 4000
    scale = 1.0 if dt == np.float32 else 3000.0
    # class (a): successive-rounding splits; class (b): raw ScalingN-with-expand output
    xa = split(g.uniform(-scale, scale, n), nc, dt)
    xb = orc.scaling_expand(split(g.uniform(-scale, scale, n), nc - 1, dt), g.uniform(-3, 3, n).astype(dt), nc=nc - 1)
    for x in (xa, xb):
        r = orc.renorm(x, nc=nc, mode=0)
        # exact sum preserved (at most nc values are ever emitted when r = nc)
        assert exact_vals(r, range(n)) == exact_vals(x, range(n))
        # zeros only trailing, and ulp-non-overlapping
        for c in range(nc - 1):
            assert ((r[c + 1] == 0) | (r[c] != 0)).all()
            assert (np.abs(r[c + 1].astype(np.float64)) <= _ulp(r[c], dt)).all()
    # idempotent on class (a) away from exact half-ulp ties
    r = orc.renorm(xa, nc=nc, mode=0)
    strict = np.ones(n, dtype=bool)
    for c in range(nc - 1):
        strict &= np.abs(xa[c + 1].astype(np.float64)) < _ulp(xa[c], dt) / 2
    assert value_equal(r[:, strict], xa[:, strict])


def test_renormalize_truncation(orc):
    """r < nc keeps the leading part: error below the last kept component's ulp."""
    g = np.random.default_rng(28)
    n = 2000
    x = split(g.uniform(-1, 1, n), 3, np.float32)
    r = orc.renorm(x, nc=3, nc_out=2, mode=0)
    ex = exact_vals(x, range(n))
    got = exact_vals(r, range(n))
    u = Fraction(2) ** -24
    for i in range(n):
        assert abs(got[i] - ex[i]) <= 2 * u * u * abs(ex[i])
