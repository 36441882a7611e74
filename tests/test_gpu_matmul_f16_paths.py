"""GPU parity of the binary16 MC product on inputs that drive every branch of its
kept-terms step, bitwise against the CPU oracle.

The binary16 product computes only the terms Simple-Renorm keeps and proves per
lane that the dropped final carry is zero (zeros form a trailing run and the last
operation is exact, |result| < 2^-13); per tile it decides from the largest
magnitude of each component plane whether the products of low components are
exact, and whether A's components are in magnitude order.  These inputs make each of
those decisions go both ways:
  * per-row and per-column scales spread over 2^-14 .. 2^2, so some tiles have
    exact low products and others do not, and the last-term test fails for some
    lanes and passes for others;
  * components set to zero at random, including leading and middle components
    (not normalized MC values; the algorithms are defined for any component
    tuple), so zero terms appear before non-zero ones;
  * products straddling 2^-13 exactly;
  * pairs of reduction steps that cancel exactly, so accumulators return to zero;
  * zero leading components of A in some tiles only.
"""
import numpy as np
import pytest

from paper_2207_08867_amd import inputs
from test_gpu_elementwise import assert_bits, to_dev, to_host

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def mcf():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2207_08867_amd as m

    m.lib()
    return m


def spread(g, shape, nc, axis_scale):
    """float64 N(0,1) entries scaled by 2^s, s drawn per row (axis 0) or per column
    (axis 1) from -14 .. 2, split into nc binary16 components; then about a quarter
    of all components (any position) set to +0 or -0."""
    x = g.normal(0.0, 1.0, shape)
    s = g.integers(-14, 3, shape[axis_scale])
    x = x * np.exp2(s)[:, None] if axis_scale == 0 else x * np.exp2(s)[None, :]
    X = inputs.split(x, nc, np.float16)
    kill = g.random(X.shape) < 0.25
    X[kill] = np.where(g.random(kill.sum()) < 0.5, np.float16(0.0), np.float16(-0.0))
    return X


def straddle(g, shape, nc):
    """Entries of magnitude 2^-7 or 2^-6 times (1 + small), so that products of a
    leading and a low component land on either side of 2^-13."""
    x = np.exp2(g.integers(-7, -5, shape)) * (1 + g.integers(-3, 4, shape) * 2.0 ** -10)
    x = x * np.where(g.random(shape) < 0.5, -1.0, 1.0)
    x = x + g.normal(0.0, 2.0 ** -14, shape)
    return inputs.split(x, nc, np.float16)


def cancelling(g, M, N, K, nc):
    """A with equal adjacent column pairs and B with opposite adjacent row pairs: the
    terms of steps 2t and 2t+1 cancel exactly, so every accumulator is zero after each
    odd step (and the binary16 components are ordinary N(0, 1/K) splits)."""
    a = g.normal(0.0, 1 / np.sqrt(K), (M, K))
    b = g.normal(0.0, 1 / np.sqrt(K), (K, N))
    a[:, 1::2] = a[:, 0:K - 1:2][:, : a[:, 1::2].shape[1]]
    b[1::2, :] = -b[0:K - 1:2, :][: b[1::2, :].shape[0]]
    return inputs.split(a, nc, np.float16), inputs.split(b, nc, np.float16)


KINDS = [(True, True), (True, False), (False, True)]


@pytest.mark.parametrize("nc", [2, 3, 4])
@pytest.mark.parametrize("kinds", KINDS)
def test_spread_and_zero_components(mcf, orc, nc, kinds):
    a_mc, b_mc = kinds
    M, N, K = 70, 45, 300
    g = np.random.default_rng(700 + 10 * nc + 3 * a_mc + b_mc)
    A = spread(g, (M, K), nc, 0)
    B = spread(g, (K, N), nc, 1)
    A = A if a_mc else A[:1]
    B = B if b_mc else B[:1]
    got = to_host(mcf.mc_matmul(to_dev(A), to_dev(B), nc=nc, a_mc=a_mc, b_mc=b_mc))
    want = orc.matmul(A, B, nc=nc, a_mc=a_mc, b_mc=b_mc)
    assert_bits(got, want, f"spread nc={nc} {kinds}")


@pytest.mark.parametrize("nc", [2, 3])
@pytest.mark.parametrize("kinds", KINDS)
def test_straddle_exact_limit(mcf, orc, nc, kinds):
    a_mc, b_mc = kinds
    M, N, K = 48, 33, 200
    g = np.random.default_rng(800 + nc)
    A = straddle(g, (M, K), nc)
    B = straddle(g, (K, N), nc)
    A = A if a_mc else A[:1]
    B = B if b_mc else B[:1]
    got = to_host(mcf.mc_matmul(to_dev(A), to_dev(B), nc=nc, a_mc=a_mc, b_mc=b_mc))
    want = orc.matmul(A, B, nc=nc, a_mc=a_mc, b_mc=b_mc)
    assert_bits(got, want, f"straddle nc={nc} {kinds}")


@pytest.mark.parametrize("nc", [2, 3])
def test_exact_cancellation(mcf, orc, nc):
    M, N, K = 40, 36, 65
    g = np.random.default_rng(900 + nc)
    A, B = cancelling(g, M, N, K, nc)
    got = to_host(mcf.mc_matmul(to_dev(A), to_dev(B), nc=nc))
    assert_bits(got, orc.matmul(A, B, nc=nc), f"cancellation nc={nc}")


@pytest.mark.parametrize("bias", [False, True])
def test_linear_spread(mcf, orc, bias):
    """MC-Linear (plain x, MC weight stored [out][in]) on spread inputs with zeroed
    weight components."""
    T, I, O, nc = 50, 130, 37, 3
    g = np.random.default_rng(950 + bias)
    x = (g.normal(0.0, 1.0, (T, I)) * np.exp2(g.integers(-10, 5, T))[:, None]).astype(np.float16)
    W = spread(g, (O, I), nc, 0)
    b = spread(g, (1, O), nc, 1)[:, 0] if bias else None
    got = to_host(mcf.mc_linear_fwd(to_dev(x), to_dev(W), to_dev(b) if bias else None))
    want = orc.linear(x, W, b, nc=nc)
    assert_bits(got, want, f"linear spread bias={bias}")


def blocky(g, shape, nc, scale_rows, scale_cols, block=16):
    """N(0,1) entries scaled by 2^(r + c), r per block of 16 rows and c per block of
    16 columns (blocks aligned with the product's 16 x 16 tiles and 16-step reduction
    tiles), so that the per-tile magnitude test passes in some tiles of an output's
    reduction and fails in others."""
    x = g.normal(0.0, 1.0, shape)
    r = g.integers(scale_rows[0], scale_rows[1] + 1, (shape[0] + block - 1) // block)
    c = g.integers(scale_cols[0], scale_cols[1] + 1, (shape[1] + block - 1) // block)
    x = x * np.exp2(np.repeat(r, block)[: shape[0]])[:, None] * np.exp2(np.repeat(c, block)[: shape[1]])[None, :]
    return inputs.split(x, nc, np.float16)


@pytest.mark.parametrize("nc", [2, 3])
@pytest.mark.parametrize("kinds", KINDS)
def test_blocky_tiles(mcf, orc, nc, kinds):
    a_mc, b_mc = kinds
    M, N, K = 64, 48, 256
    g = np.random.default_rng(980 + nc)
    A = blocky(g, (M, K), nc, (-3, 1), (-3, 1))
    B = blocky(g, (K, N), nc, (-3, 1), (-3, 1))
    A = A if a_mc else A[:1]
    B = B if b_mc else B[:1]
    got = to_host(mcf.mc_matmul(to_dev(A), to_dev(B), nc=nc, a_mc=a_mc, b_mc=b_mc))
    want = orc.matmul(A, B, nc=nc, a_mc=a_mc, b_mc=b_mc)
    assert_bits(got, want, f"blocky nc={nc} {kinds}")


@pytest.mark.parametrize("nc", [2, 3])
def test_growing_low_accumulators(mcf, orc, nc):
    """Positive A ~ 1/2 and B ~ 2^-5 (MC x MC): every product of a low component is
    below 2^-13, so the tiles take the exact-low-products form, but the accumulators
    of B's low components grow past 2^-13 after a few dozen steps, where their
    tiny-sum form no longer applies and lanes fall back to the general step."""
    M, N, K = 40, 48, 256
    g = np.random.default_rng(990 + nc)
    A = inputs.split(0.5 + g.uniform(0.0, 0.25, (M, K)), nc, np.float16)
    B = inputs.split(2.0 ** -5 * (1.0 + g.uniform(0.0, 1.0, (K, N))), nc, np.float16)
    got = to_host(mcf.mc_matmul(to_dev(A), to_dev(B), nc=nc))
    assert_bits(got, orc.matmul(A, B, nc=nc), f"growing nc={nc}")


@pytest.mark.parametrize("nc", [2, 3])
def test_component_order_flag(mcf, orc, nc):
    """MC x MC with every low-component product below 2^-13 (N(0, 1/K) splits): per
    32-step tile the product skips the kept-terms test of B's low components when every
    value of A in the tile has its components in magnitude order.  Here some values of
    A in the k ranges 32..63 and 160..191 (and in a few rows only) get a zero leading
    component (a low component then exceeds the leading one), so those tiles run the
    test and its failing lanes take the general step, while the other tiles skip it."""
    M, N, K = 80, 48, 256
    g = np.random.default_rng(1150 + nc)
    A, B = inputs.matmul_normal(M, N, K, nc, np.float16, seed=1160 + nc)
    rows = g.choice(M, 12, replace=False)
    for k0 in (32, 160):
        ks = k0 + g.integers(0, 32, 12)
        A[0, rows, ks] = np.where(g.random(12) < 0.5, np.float16(0.0), np.float16(-0.0))
    assert (np.abs(A[1]) > np.abs(A[0])).any()
    got = to_host(mcf.mc_matmul(to_dev(A), to_dev(B), nc=nc))
    assert_bits(got, orc.matmul(A, B, nc=nc), f"order flag nc={nc}")


def unordered(g, shape, nc, nonfinite=0):
    """Components drawn independently, each N(0,1) times 2^s with s from -20 .. 2, so
    that a later component is larger than an earlier non-zero one about half the time
    (not normalized MC values; the algorithms take any component tuple).  ScalingN's
    kept terms are then out of magnitude order, the case its order test sends to the
    general step.  `nonfinite` entries get an infinite or NaN component."""
    X = (g.normal(0.0, 1.0, (nc,) + shape) * np.exp2(g.integers(-20, 3, (nc,) + shape))).astype(np.float16)
    if nonfinite:
        idx = tuple(g.integers(0, d, nonfinite) for d in (nc,) + shape)
        X[idx] = np.array([np.inf, -np.inf, np.nan], dtype=np.float16)[g.integers(0, 3, nonfinite)]
    return X


@pytest.mark.parametrize("nc", [2, 3])
@pytest.mark.parametrize("kinds", KINDS)
@pytest.mark.parametrize("nonfinite", [0, 5])
def test_unordered_components(mcf, orc, nc, kinds, nonfinite):
    a_mc, b_mc = kinds
    M, N, K = 52, 40, 150
    g = np.random.default_rng(1100 + 10 * nc + 3 * a_mc + b_mc + nonfinite)
    A = unordered(g, (M, K), nc, nonfinite)
    B = unordered(g, (K, N), nc, nonfinite)
    A = A if a_mc else A[:1]
    B = B if b_mc else B[:1]
    with np.errstate(all="ignore"):
        got = to_host(mcf.mc_matmul(to_dev(A), to_dev(B), nc=nc, a_mc=a_mc, b_mc=b_mc))
        want = orc.matmul(A, B, nc=nc, a_mc=a_mc, b_mc=b_mc)
    assert_bits(got, want, f"unordered nc={nc} {kinds} nonfinite={nonfinite}")


def test_linear_unordered(mcf, orc):
    T, I, O, nc = 40, 96, 33, 3
    g = np.random.default_rng(1200)
    x = (g.normal(0.0, 1.0, (T, I)) * np.exp2(g.integers(-12, 3, (T, I)))).astype(np.float16)
    W = unordered(g, (O, I), nc)
    b = unordered(g, (O,), nc)
    with np.errstate(all="ignore"):
        got = to_host(mcf.mc_linear_fwd(to_dev(x), to_dev(W), to_dev(b)))
        want = orc.linear(x, W, b, nc=nc)
    assert_bits(got, want, "linear unordered")
