"""GPU parity with binary64 components (the paper's MC float64), bitwise against the
CPU oracle: every elementwise operation and kind, the products (MM-MCN, MC-Linear,
K-split, batched, AddMM, pruned) and the linear-regression step, nc 1..4 (products
1..3), ragged sizes; Exp-MCN with the correctly rounded binary64 component
exponential."""
import os

import numpy as np
import pytest

from paper_2207_08867_amd import inputs
from test_gpu_elementwise import assert_bits, to_dev, to_host

pytestmark = pytest.mark.gpu
F64 = np.float64


@pytest.fixture(scope="module")
def mcf():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2207_08867_amd as m

    m.lib()
    return m


def ex(seed, shape, nc, scale=1.0):
    return inputs.expansion(np.random.default_rng(seed), shape, nc, F64, scale)


@pytest.mark.parametrize("nc", [1, 2, 3, 4])
def test_elementwise_f64(mcf, orc, nc):
    n = 10007
    x = ex(4000 + nc, n, nc)
    y = ex(4010 + nc, n, nc)
    y[0] = np.abs(y[0]) + 0.5
    v = np.random.default_rng(4020).normal(0, 1, n)
    tx, ty, tv = to_dev(x), to_dev(y), to_dev(v)
    cases = [
        ("add", mcf.mc_add(tx, ty, nc=nc), orc.add(x, y, nc=nc)),
        ("grow", mcf.mc_add(tx, tv, nc=nc, y_mc=False), orc.add(x, v, nc=nc, y_mc=False)),
        ("grow T,MC", mcf.mc_add(tv, tx, nc=nc, x_mc=False), orc.add(v, x, nc=nc, x_mc=False)),
        ("scaling", mcf.mc_mul(tx, tv, nc=nc, y_mc=False), orc.mul(x, v, nc=nc, y_mc=False)),
        ("mult", mcf.mc_mul(tx, ty, nc=nc), orc.mul(x, y, nc=nc)),
        ("div", mcf.mc_div(tx, ty, nc=nc), orc.div(x, y, nc=nc)),
        ("divn", mcf.mc_div(tv, ty, nc=nc, x_mc=False), orc.div(v, y, nc=nc, x_mc=False)),
        ("mult slow", mcf.mc_mul_slow(tx, ty, nc=nc), orc.mul_slow(x, y, nc=nc)),
        ("square", mcf.mc_square(tx, nc=nc), orc.square(x, nc=nc)),
        ("renorm", mcf.mc_renorm(tx), orc.renorm(x, nc=nc)),
        ("simple renorm", mcf.mc_renorm(tx, mode=1), orc.renorm(x, nc=nc, mode=1)),
    ]
    for name, got, want in cases:
        assert_bits(to_host(got), want, f"{name} f64 nc={nc}")


def _near_midpoints():
    path = os.path.join(os.path.dirname(__file__), "golden", "exp64_near_midpoints.txt")
    return np.array([float.fromhex(l) for l in open(path) if l.strip() and not l.startswith("#")])


def test_exp64_component_exponential(mcf, orc):
    """nc = 1 Exp-MCN is the correctly rounded binary64 e^x: 2^24 random arguments over
    the whole range (about 2^-15 of them take the 192-bit fixed-point stage), the range
    of subnormal results, tiny arguments, boundaries, special values, and the 311
    arguments whose e^x lies within 2^-72 of a rounding boundary (every one takes the
    fixed-point stage)."""
    g = np.random.default_rng(4100)
    xs = np.concatenate([g.uniform(-745.2, 709.8, 1 << 24), g.uniform(-746, -708, 1 << 16),
                         g.normal(0, 1, 1 << 14) * np.exp2(g.integers(-80, 0, 1 << 14)),
                         [0.0, -0.0, 709.782712893384, 709.7827128933841, -745.1332191019411,
                          -745.1332191019412, -708.3964185322641, 2.0 ** -53, -(2.0 ** -54), np.inf, -np.inf,
                          np.nan, 800.0, -800.0, 1e-300, -1e-300],
                         _near_midpoints()])
    got = to_host(mcf.mc_exp(to_dev(xs[None]), nc=1))[0]
    assert_bits(got, orc.fl_exp64(xs), "binary64 e^x")


def test_exp64_small_arguments(mcf, orc):
    """Arguments below 2^-27 in magnitude fill whole wavefronts (the short first stage
    runs only then): random ones of every scale, the near-boundary ones of the fixture
    (each of which must reach the fixed-point stage), as nc = 1 values and as the low
    component of nc = 2 values."""
    nm = _near_midpoints()
    small = nm[np.abs(nm) < 2.0 ** -27]
    assert small.size >= 40
    g = np.random.default_rng(4101)
    rnd = g.uniform(-1, 1, 1 << 16) * np.exp2(g.integers(-1074 + 60, -27, 1 << 16).astype(np.float64))
    xs = np.concatenate([np.tile(small, 64), rnd, [0.0, -0.0, 5e-324, -5e-324]])
    got = to_host(mcf.mc_exp(to_dev(xs[None]), nc=1))[0]
    assert_bits(got, orc.fl_exp64(xs), "binary64 e^x, small arguments")
    x2 = np.zeros((2, xs.size))
    x2[0] = g.uniform(-5, 5, xs.size)
    x2[1] = xs
    assert_bits(to_host(mcf.mc_exp(to_dev(x2), nc=2)), orc.exp(x2, nc=2), "Exp-MCN f64 small low components")


@pytest.mark.parametrize("nc", [2, 3, 4])
def test_exp_mcn_f64(mcf, orc, nc):
    """Exp-MCN over binary64 expansions (components from a draw of e^x-sized
    arguments), with the near-boundary arguments as leading and as lower components."""
    n = 20011
    g = np.random.default_rng(4200 + nc)
    x = np.zeros((nc, n))
    x[0] = g.uniform(-30, 30, n)
    for c in range(1, nc):
        x[c] = g.uniform(-1, 1, n) * np.exp2(-18 * c)
    nm = _near_midpoints()
    x[0, : nm.size] = nm
    x[1, nm.size: 2 * nm.size] = nm / 1024
    tx = to_dev(x)
    assert_bits(to_host(mcf.mc_exp(tx, nc=nc)), orc.exp(x, nc=nc), f"Exp-MCN f64 nc={nc}")
    mcf.mc_exp(tx, nc=nc, out=tx)  # in place
    assert_bits(to_host(tx), orc.exp(x, nc=nc), f"Exp-MCN f64 nc={nc} in place")


@pytest.mark.parametrize("nc", [1, 2, 3])
@pytest.mark.parametrize("kinds", [(True, True), (True, False), (False, True)])
def test_matmul_f64(mcf, orc, nc, kinds):
    a_mc, b_mc = kinds
    M, N, K = 70, 45, 37
    A = ex(4100 + nc, (M, K), nc, 1 / np.sqrt(K))
    B = ex(4110 + nc, (K, N), nc, 1 / np.sqrt(K))
    A, B = (A if a_mc else A[:1]), (B if b_mc else B[:1])
    got = to_host(mcf.mc_matmul(to_dev(A), to_dev(B), nc=nc, a_mc=a_mc, b_mc=b_mc))
    assert_bits(got, orc.matmul(A, B, nc=nc, a_mc=a_mc, b_mc=b_mc), f"matmul f64 nc={nc} {kinds}")
    if a_mc and b_mc:
        got = to_host(mcf.mc_matmul_pruned(to_dev(A), to_dev(B), nc=nc))
        assert_bits(got, orc.matmul_pruned(A, B, nc=nc), f"pruned f64 nc={nc}")


@pytest.mark.parametrize("nc", [2, 3])
def test_linear_splitk_batched_addmm_f64(mcf, orc, nc):
    g = np.random.default_rng(4200 + nc)
    X = g.normal(0, 1, (33, 50))
    W = ex(4201, (20, 50), nc, 0.1)
    b = ex(4202, 20, nc, 0.1)
    got = to_host(mcf.mc_linear_fwd(to_dev(X), to_dev(W), to_dev(b)))
    assert_bits(got, orc.linear(X, W, b, nc=nc), "linear f64")
    A = ex(4203, (1, 3000), nc)
    Bv = ex(4204, (3000, 1), nc)
    for S in (1, 7, 300):
        got = to_host(mcf.mc_matmul_splitk(to_dev(A), to_dev(Bv), nc=nc, slices=S))
        assert_bits(got, orc.matmul_splitk(A, Bv, nc=nc, slices=S), f"dot f64 S={S}")
    A3 = ex(4205, (3, 17, 9), nc)
    B3 = ex(4206, (3, 9, 11), nc)[:1]
    got = to_host(mcf.mc_matmul_batched(to_dev(A3), to_dev(B3), nc=nc, b_mc=False))
    assert_bits(got, orc.matmul_batched(A3, B3, nc=nc, b_mc=False), "bmm f64")
    Am = ex(4207, (12, 8), nc)
    Bm = ex(4208, (8, 10), nc)[:1]
    Y = ex(4209, 10, nc)
    got = to_host(mcf.mc_addmm(to_dev(Am), to_dev(Bm), to_dev(Y), nc=nc, alpha=0.1, beta=-3.7))
    assert_bits(got, orc.addmm(Am, Bm, Y, 0.1, -3.7, nc=nc), "addmm f64")


@pytest.mark.parametrize("nc", [1, 2, 3])
def test_linreg_f64(mcf, orc, nc):
    import torch

    n, d = 2000, 2
    X, y_neg, W, _ = inputs.linreg_inputs(n, d, nc, F64, seed=4300 + nc)
    W = ex(4301, d, nc, 0.5)
    Sg, Sl = mcf.mc_matmul_splitk_slices(1, d, n), mcf.mc_matmul_splitk_slices(1, 1, n)
    tX, ty, tW = to_dev(X), to_dev(y_neg), to_dev(W)
    loss = torch.empty(nc, dtype=torch.float64, device="cuda")
    for step in range(4):
        mcf.mc_linreg_gd_step(tX, ty, tW, 0.05, loss=loss)
        W, want = orc.linreg_gd_step(X, y_neg, W, 0.05, slices_g=Sg, slices_l=Sl)
        assert_bits(to_host(tW), W, f"W f64 step {step}")
        assert_bits(to_host(loss), want, f"loss f64 step {step}")
