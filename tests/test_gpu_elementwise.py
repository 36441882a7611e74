"""GPU parity of the elementwise MC operations against the CPU oracle (bitwise).

Inputs come from paper_2207_08867_amd.inputs (seeded); the oracle sees the same host
arrays.  Components are compared bit for bit (binary16 / binary32 patterns), NaNs
by class.  Sizes are ragged (not multiples of the 16-byte vector width) so both
the vector path and the scalar tail run; the full 2^26-element workload is checked
on a random sample of elements, which the oracle evaluates one by one.
"""
import numpy as np
import pytest

from paper_2207_08867_amd import inputs

pytestmark = pytest.mark.gpu

DTS = [np.float16, np.float32]


def to_dev(a):
    import torch

    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def to_host(t):
    return t.cpu().numpy()


def assert_bits(got, want, what=""):
    got = np.asarray(got)
    want = np.asarray(want)
    assert got.shape == want.shape, (got.shape, want.shape)
    u = {2: np.uint16, 4: np.uint32, 8: np.uint64}[got.dtype.itemsize]
    gb, wb = got.view(u), want.view(u)
    nan = np.isnan(got.astype(np.float64)) & np.isnan(want.astype(np.float64))
    bad = (gb != wb) & ~nan
    if bad.any():
        idx = np.argwhere(bad)[:5]
        raise AssertionError(f"{what}: {int(bad.sum())} component mismatches, e.g. at {idx.tolist()}: "
                             f"got {[got[tuple(i)] for i in idx]} want {[want[tuple(i)] for i in idx]}")


@pytest.fixture(scope="module")
def mcf():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2207_08867_amd as m

    m.lib()
    return m


def _operands(op, n, nc, dt, seed):
    x, y = inputs.elementwise_inputs(op, n, nc, dt, seed=seed)
    return x, y


@pytest.mark.parametrize("dt", DTS)
@pytest.mark.parametrize("nc", [1, 2, 3, 4])
@pytest.mark.parametrize("op", ["add", "mul", "div"])
@pytest.mark.parametrize("kinds", [(True, True), (True, False), (False, True)])
def test_binary_parity(mcf, orc, dt, nc, op, kinds):
    n = 40_003
    x_mc, y_mc = kinds
    x, y = _operands(op, n, nc, dt, seed=100 + nc)
    xa = x if x_mc else x[:1]
    ya = y if y_mc else y[:1]
    fn = {"add": (mcf.mc_add, orc.add), "mul": (mcf.mc_mul, orc.mul), "div": (mcf.mc_div, orc.div)}[op]
    got = to_host(fn[0](to_dev(xa), to_dev(ya), nc=nc, x_mc=x_mc, y_mc=y_mc))
    want = fn[1](xa, ya, nc=nc, x_mc=x_mc, y_mc=y_mc)
    assert_bits(got, want, f"{op} {dt.__name__} nc={nc} kinds={kinds}")


@pytest.mark.parametrize("dt", DTS)
@pytest.mark.parametrize("nc", [1, 2, 3, 4])
@pytest.mark.parametrize("mode", [0, 1])
def test_renorm_parity(mcf, orc, dt, nc, mode):
    n = 30_011
    g = np.random.default_rng(7 + nc)
    # overlapping inputs: raw sums of independent draws, plus planted zeros
    x = np.stack([g.uniform(-1, 1, n) * 2.0 ** (-12 * c * (dt == np.float32) - 5 * c * (dt == np.float16))
                  for c in range(nc)]).astype(dt)
    x[:, g.random(n) < 0.2] = 0
    x[g.integers(0, nc, n), np.arange(n)] = 0
    for nc_out in range(1, nc + 1):
        got = to_host(mcf.mc_renorm(to_dev(x), nc_out=nc_out, mode=mode))
        want = orc.renorm(x, nc=nc, nc_out=nc_out, mode=mode)
        assert_bits(got, want, f"renorm mode={mode} {dt.__name__} {nc}->{nc_out}")


@pytest.mark.parametrize("dt", DTS)
@pytest.mark.parametrize("nc", [1, 2, 3, 4])
def test_exp_parity(mcf, orc, dt, nc):
    n = 50_001
    x, _ = inputs.elementwise_inputs("exp", n, nc, dt, seed=300 + nc)
    got = to_host(mcf.mc_exp(to_dev(x), nc=nc))
    assert_bits(got, orc.exp(x, nc=nc), f"exp {dt.__name__} nc={nc}")


def test_exp32_component_exhaustive(mcf, orc):
    """The binary32 component exponential (Exp-MCN at nc = 1) on every binary32 input
    with 2^-30 <= |x| <= 105 -- the range where e^x is neither 1, 0 nor infinite
    after rounding, and where inputs whose binary64 e^x lies close to a rounding
    boundary take the double-double path -- in chunks of 2^26, plus every 997th bit
    pattern over the whole encoding space (zeros, subnormals, huge, infinities,
    NaNs)."""
    lo, hi = 0x30800000, 0x42D20001  # 2^-30 .. 105.0
    chunk = 1 << 26
    for sign in (0, 0x80000000):
        for start in range(lo, hi, chunk):
            bits = np.arange(start, min(start + chunk, hi), dtype=np.uint32) | np.uint32(sign)
            x = bits.view(np.float32)[None]
            print(f"exp32 exhaustive: sign {sign >> 31} patterns {start:#x}..", flush=True)
            got = to_host(mcf.mc_exp(to_dev(x), nc=1))
            assert_bits(got, orc.exp(x, nc=1), f"exp32 from {start | sign:#x}")
    bits = np.arange(0, 1 << 32, 997, dtype=np.uint64).astype(np.uint32)
    x = bits.view(np.float32)[None]
    got = to_host(mcf.mc_exp(to_dev(x), nc=1))
    assert_bits(got, orc.exp(x, nc=1), "exp32 strided")


def test_exp_component_exhaustive(mcf, orc):
    """The component exponential on every binary16 encoding (nc = 1 is exactly the
    correctly rounded exponential)."""
    x = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16).view(np.float16)[None].copy()
    got = to_host(mcf.mc_exp(to_dev(x), nc=1))
    assert_bits(got, orc.exp(x, nc=1), "exp16 exhaustive")
    # every encoding as the second and as the third component (the lower components'
    # exponentials: arithmetic for |x| <= 2^-9, the table otherwise)
    for nc in (2, 3):
        y = np.zeros((nc, 1 << 16), dtype=np.float16)
        y[0] = np.float16(0.75)
        y[nc - 1] = x[0]
        if nc == 3:
            y[1] = np.float16(-2.0 ** -10)
        assert_bits(to_host(mcf.mc_exp(to_dev(y), nc=nc)), orc.exp(y, nc=nc), f"exp16 exhaustive, component {nc - 1}")


def test_div_f16_component_strided_exhaustive(mcf, orc):
    """Correctly rounded binary16 division: every dividend against 2048 divisors."""
    a = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16).view(np.float16)
    b = a[np.isfinite(a) & (a != 0)][::30][:2048]
    A = np.repeat(a, b.size)[None].copy()
    B = np.tile(b, a.size)[None].copy()
    got = to_host(mcf.mc_div(to_dev(A), to_dev(B), nc=1))
    assert_bits(got, orc.div(A, B, nc=1), "div16")


def test_special_values(mcf, orc):
    """Subnormal components, signed zeros and values near the binary16 range."""
    g = np.random.default_rng(9)
    n = 4099
    for dt in DTS:
        tiny = np.finfo(dt).smallest_subnormal
        x = np.stack([g.integers(-64, 64, n) * tiny, g.integers(-8, 8, n) * tiny, np.zeros(n)]).astype(dt)
        x[2, ::7] = -0.0
        y = np.stack([g.uniform(-1e-3, 1e-3, n), g.integers(-4, 4, n) * tiny, np.zeros(n)]).astype(dt)
        for fn, ofn in ((mcf.mc_add, orc.add), (mcf.mc_mul, orc.mul)):
            assert_bits(to_host(fn(to_dev(x), to_dev(y), nc=3, y_mc=True)), ofn(x, y, nc=3), "special")
            assert_bits(to_host(fn(to_dev(x), to_dev(y[:1]), nc=3, y_mc=False)), ofn(x, y[:1], nc=3, y_mc=False),
                        "special")


@pytest.mark.parametrize("dt", DTS)
def test_overflow_from_finite_operands(mcf, orc, dt):
    """Leading sums and products that overflow although every operand is finite
    (|x| in [0.3, 1] of the format's largest value, plain factors in [1, 4]):
    ScalingN, Add-MCN and Grow-ExpN agree with the algorithm bit for bit -- the
    infinite leading component and the NaN carries the Two-Sums leave behind it."""
    g = np.random.default_rng(15)
    n = 4099
    big = float(np.finfo(dt).max)

    def sign():
        return g.choice([-1.0, 1.0], n)

    x = inputs.split(sign() * g.uniform(0.3, 1.0, n) * big, 3, dt)
    y = inputs.split(sign() * g.uniform(0.3, 1.0, n) * big, 3, dt)
    v = (sign() * g.uniform(1.0, 4.0, n)).astype(dt)[None]
    w = (sign() * g.uniform(0.3, 1.0, n) * big).astype(dt)[None]
    tx, ty, tv, tw = to_dev(x), to_dev(y), to_dev(v), to_dev(w)
    cases = (
        ("ScalingN (MC,T)", mcf.mc_mul(tx, tv, nc=3, y_mc=False), orc.mul(x, v, nc=3, y_mc=False)),
        ("ScalingN (T,MC)", mcf.mc_mul(tv, tx, nc=3, x_mc=False), orc.mul(v, x, nc=3, x_mc=False)),
        ("Add-MCN", mcf.mc_add(tx, ty, nc=3), orc.add(x, y, nc=3)),
        ("Grow-ExpN", mcf.mc_add(tx, tw, nc=3, y_mc=False), orc.add(x, w, nc=3, y_mc=False)),
    )
    for what, got, want in cases:
        lead = want[0].astype(np.float64)
        assert np.isinf(lead).any() and np.isfinite(lead).any(), what  # both kinds occur
        assert_bits(to_host(got), want, f"{what} overflow")


def test_literal_mult_inputs_overflow_class(mcf, orc):
    """Mult-MCN with divisors drawn from U[-1/2, 1/2] (the literal elementwise input
    range): tiny divisors overflow the reciprocal.  Elements whose result is finite on
    both sides agree bit for bit; the others are non-finite on both sides."""
    n = 1 << 18
    x, _ = inputs.elementwise_inputs("add", n, 3, np.float16, seed=11)
    _, y = inputs.elementwise_inputs("add", n, 3, np.float16, seed=12)
    got = to_host(mcf.mc_mul(to_dev(x), to_dev(y), nc=3))
    want = orc.mul(x, y, nc=3)
    gfin = np.isfinite(got.astype(np.float64)).all(0)
    wfin = np.isfinite(want.astype(np.float64)).all(0)
    assert np.array_equal(gfin, wfin)
    assert (~wfin).sum() > 0  # the case does occur (about 2^-15 of the elements)
    assert_bits(got[:, wfin], want[:, wfin], "mult literal range")


def test_in_place_and_empty(mcf, orc):
    import torch

    x, y = inputs.elementwise_inputs("add", 1000, 3, np.float32, seed=13)
    want = orc.add(x, y, nc=3)
    tx = to_dev(x)
    mcf.mc_add(tx, to_dev(y), nc=3, out=tx)
    assert_bits(to_host(tx), want, "in place")
    e = torch.empty((3, 0), dtype=torch.float32, device="cuda")
    assert mcf.mc_add(e, e, nc=3).shape == (3, 0)


@pytest.mark.parametrize("op", ["add", "mul", "div", "exp", "renorm"])
def test_full_size_sampled(mcf, orc, op):
    """The 2^26-element binary16 nc=3 workload, in the launch configuration the
    benchmark uses, checked on a random sample of 2^16 elements plus both ends."""
    n = 1 << 26
    nc = 3
    x, y = inputs.elementwise_inputs(op, n, nc, np.float16, seed=0)
    if op == "exp":
        out = mcf.mc_exp(to_dev(x), nc=nc)
    elif op == "renorm":
        out = mcf.mc_renorm(to_dev(x), mode=0)
    else:
        f = {"add": mcf.mc_add, "mul": mcf.mc_mul, "div": mcf.mc_div}[op]
        out = f(to_dev(x), to_dev(y), nc=nc)
    got = to_host(out)
    g = np.random.default_rng(14)
    idx = np.unique(np.concatenate([g.integers(0, n, 1 << 16), np.arange(64), np.arange(n - 64, n)]))
    xs = np.ascontiguousarray(x[:, idx])
    if op == "exp":
        want = orc.exp(xs, nc=nc)
    elif op == "renorm":
        want = orc.renorm(xs, nc=nc, mode=0)
    else:
        ys = np.ascontiguousarray(y[:, idx])
        want = {"add": orc.add, "mul": orc.mul, "div": orc.div}[op](xs, ys, nc=nc)
    assert_bits(got[:, idx], want, f"{op} full size")


def test_deterministic(mcf):
    x, y = inputs.elementwise_inputs("mul", 1 << 20, 3, np.float16, seed=15)
    tx, ty = to_dev(x), to_dev(y)
    a = to_host(mcf.mc_mul(tx, ty, nc=3))
    b = to_host(mcf.mc_mul(tx, ty, nc=3))
    assert_bits(a, b, "repeat")


@pytest.mark.parametrize("dt", DTS)
@pytest.mark.parametrize("nc", [2, 3, 4])
@pytest.mark.parametrize("op", ["mul", "div"])
def test_div_mult_spread_and_zero_components(mcf, orc, dt, nc, op):
    """Div-MCN and Mult-MCN on operands with magnitudes spread over 2^-20 .. 2^6 and
    about a quarter of all components (leading ones included) set to +0 or -0, so
    that ScalingN terms have zeros before non-zeros, quotient digits are zero and the
    per-lane tests of the fast steps fail both ways.  Non-finite results (zero
    divisors) compare by class, finite ones bit for bit."""
    n = 20_011
    g = np.random.default_rng(500 + nc + 10 * (op == "mul") + 20 * (dt == np.float32))
    def operand():
        v = g.normal(0.0, 1.0, n) * np.exp2(g.integers(-20, 7, n))
        X = inputs.split(v, nc, dt)
        kill = g.random(X.shape) < 0.25
        X[kill] = np.where(g.random(kill.sum()) < 0.5, dt(0.0), dt(-0.0))
        return X
    x, y = operand(), operand()
    fn = {"mul": (mcf.mc_mul, orc.mul), "div": (mcf.mc_div, orc.div)}[op]
    with np.errstate(all="ignore"):
        got = to_host(fn[0](to_dev(x), to_dev(y), nc=nc))
        want = fn[1](x, y, nc=nc)
    assert_bits(got, want, f"{op} spread {dt.__name__} nc={nc}")


@pytest.mark.parametrize("dt", DTS)
@pytest.mark.parametrize("nc", [2, 3])
@pytest.mark.parametrize("op", ["mul", "div", "mul_slow"])
def test_div_mult_unordered_components(mcf, orc, dt, nc, op):
    """Div-MCN and Mult-MCN on component tuples whose magnitudes are out of order (each
    component drawn independently over 2^-20 .. 2^2): the kept-terms ScalingN steps
    then see terms out of magnitude order, which their order test sends to the general
    step.  Bit for bit; non-finite results by class."""
    n = 12_007
    g = np.random.default_rng(1300 + nc + 10 * ("mul" in op) + 20 * (dt == np.float32) + 40 * (op == "mul_slow"))
    def operand():
        return (g.normal(0.0, 1.0, (nc, n)) * np.exp2(g.integers(-20, 3, (nc, n)))).astype(dt)
    x, y = operand(), operand()
    fn = {"mul": (mcf.mc_mul, orc.mul), "div": (mcf.mc_div, orc.div),
          "mul_slow": (mcf.mc_mul_slow, orc.mul_slow)}[op]
    with np.errstate(all="ignore"):
        got = to_host(fn[0](to_dev(x), to_dev(y), nc=nc))
        want = fn[1](x, y, nc=nc)
    assert_bits(got, want, f"{op} unordered {dt.__name__} nc={nc}")
