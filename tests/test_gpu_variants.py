"""GPU parity of Mult-MCN-Slow and Square-MCN against the CPU oracle, bitwise."""
import numpy as np
import pytest

from paper_2207_08867_amd import inputs
from test_gpu_elementwise import assert_bits, to_dev, to_host

pytestmark = pytest.mark.gpu
DTS = [np.float16, np.float32]


@pytest.fixture(scope="module")
def mcf():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2207_08867_amd as m

    m.lib()
    return m


def spread_operand(g, n, nc, dt):
    """Magnitudes over 2^-20 .. 2^6, about a quarter of all components zeroed."""
    X = inputs.split(g.normal(0.0, 1.0, n) * np.exp2(g.integers(-20, 7, n)), nc, dt)
    kill = g.random(X.shape) < 0.25
    X[kill] = np.where(g.random(kill.sum()) < 0.5, dt(0.0), dt(-0.0))
    return X


@pytest.mark.parametrize("dt", DTS)
@pytest.mark.parametrize("nc", [1, 2, 3, 4])
def test_mul_slow_parity(mcf, orc, dt, nc):
    x, y = inputs.elementwise_inputs("mul", 40_003, nc, dt, seed=600 + nc)
    got = to_host(mcf.mc_mul_slow(to_dev(x), to_dev(y), nc=nc))
    assert_bits(got, orc.mul_slow(x, y, nc=nc), f"mul_slow {dt.__name__} nc={nc}")


@pytest.mark.parametrize("dt", DTS)
@pytest.mark.parametrize("nc", [2, 3, 4])
def test_mul_slow_spread(mcf, orc, dt, nc):
    g = np.random.default_rng(650 + nc)
    x, y = spread_operand(g, 20_011, nc, dt), spread_operand(g, 20_011, nc, dt)
    with np.errstate(all="ignore"):
        got = to_host(mcf.mc_mul_slow(to_dev(x), to_dev(y), nc=nc))
        want = orc.mul_slow(x, y, nc=nc)
    assert_bits(got, want, f"mul_slow spread {dt.__name__} nc={nc}")


@pytest.mark.parametrize("dt", DTS)
@pytest.mark.parametrize("nc", [1, 2, 3, 4])
def test_square_parity(mcf, orc, dt, nc):
    x, _ = inputs.elementwise_inputs("add", 40_003, nc, dt, seed=700 + nc)
    got = to_host(mcf.mc_square(to_dev(x), nc=nc))
    assert_bits(got, orc.square(x, nc=nc), f"square {dt.__name__} nc={nc}")
    g = np.random.default_rng(750 + nc)
    xs = spread_operand(g, 20_011, nc, dt)
    with np.errstate(all="ignore"):
        got = to_host(mcf.mc_square(to_dev(xs), nc=nc))
        want = orc.square(xs, nc=nc)
    assert_bits(got, want, f"square spread {dt.__name__} nc={nc}")


def test_in_place_and_full_size(mcf, orc):
    """In place (out == x), and the 2^26-element binary16 nc = 3 workload sampled."""
    x, y = inputs.elementwise_inputs("mul", 1000, 3, np.float32, seed=800)
    tx = to_dev(x)
    mcf.mc_square(tx, nc=3, out=tx)
    assert_bits(to_host(tx), orc.square(x, nc=3), "square in place")
    tx, ty = to_dev(x), to_dev(y)
    mcf.mc_mul_slow(tx, ty, nc=3, out=ty)
    assert_bits(to_host(ty), orc.mul_slow(x, y, nc=3), "mul_slow in place")
    n = 1 << 26
    s = inputs.elementwise_suite(n, 3, np.float16, seed=0)
    a, d = to_dev(s["a"]), to_dev(s["d"])
    gs = to_host(mcf.mc_square(a, nc=3))
    gm = to_host(mcf.mc_mul_slow(a, d, nc=3))
    g = np.random.default_rng(801)
    idx = np.unique(np.concatenate([g.integers(0, n, 1 << 15), np.arange(64), np.arange(n - 64, n)]))
    xa, xd = np.ascontiguousarray(s["a"][:, idx]), np.ascontiguousarray(s["d"][:, idx])
    assert_bits(gs[:, idx], orc.square(xa, nc=3), "square full size")
    assert_bits(gm[:, idx], orc.mul_slow(xa, xd, nc=3), "mul_slow full size")
