"""GPU parity of the pruned MC x MC product against the CPU oracle (bitwise), and its
error bound against the exact product."""
import numpy as np
import pytest

from paper_2207_08867_amd import inputs
from test_gpu_elementwise import assert_bits, to_dev, to_host

pytestmark = pytest.mark.gpu
U = {np.float16: 2.0 ** -11, np.float32: 2.0 ** -24}


@pytest.fixture(scope="module")
def mcf():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2207_08867_amd as m

    m.lib()
    return m


def bound_ok(orc, A, B, C, nc, K, dt, rows=None, cols=None):
    err, absab, _ = orc.matmul_exact_err(A, B, C, rows=rows, cols=cols)
    floor = nc * nc * K * 2.0 ** -25 if dt == np.float16 else 0.0
    return bool((np.abs(err) <= 4 * K * U[dt] ** min(nc, 3) * absab + floor).all())


@pytest.mark.parametrize("dt", [np.float16, np.float32])
@pytest.mark.parametrize("nc", [1, 2, 3, 4])
def test_pruned_small_ragged(mcf, orc, dt, nc):
    M, N, K = 70, 45, 37
    A, B = inputs.matmul_normal(M, N, K, nc, dt, seed=1700 + nc)
    got = to_host(mcf.mc_matmul_pruned(to_dev(A), to_dev(B), nc=nc))
    assert_bits(got, orc.matmul_pruned(A, B, nc=nc), f"pruned {dt.__name__} nc={nc}")
    assert bound_ok(orc, A, B, got, nc, K, dt)


@pytest.mark.parametrize("dt", [np.float16, np.float32])
@pytest.mark.parametrize("nc", [2, 3])
def test_pruned_spread_zeros(mcf, orc, dt, nc):
    """Spread magnitudes and zeroed components, so the per-lane and per-tile tests of
    every step go both ways."""
    g = np.random.default_rng(1750 + nc)
    def operand(shape, axis):
        x = g.normal(0.0, 1.0, shape) * (np.exp2(g.integers(-14, 3, shape[axis]))[:, None] if axis == 0
                                         else np.exp2(g.integers(-14, 3, shape[axis]))[None, :])
        X = inputs.split(x, nc, dt)
        kill = g.random(X.shape) < 0.25
        X[kill] = 0
        return X
    A, B = operand((64, 200), 0), operand((200, 48), 1)
    got = to_host(mcf.mc_matmul_pruned(to_dev(A), to_dev(B), nc=nc))
    assert_bits(got, orc.matmul_pruned(A, B, nc=nc), f"pruned spread {dt.__name__} nc={nc}")


def test_pruned_large_tile_path(mcf, orc):
    """2^25+ outputs take the two-outputs-per-lane binary32 tile: 6001 x 5603 x 37."""
    M, N, K, nc = 6001, 5603, 37, 3
    g = np.random.default_rng(1760)
    A = inputs.split(g.normal(0, 1 / np.sqrt(K), (M, K)), nc, np.float32)
    B = inputs.split(g.normal(0, 1 / np.sqrt(K), (K, N)), nc, np.float32)
    got = to_host(mcf.mc_matmul_pruned(to_dev(A), to_dev(B), nc=nc))
    rows = np.concatenate([g.integers(0, M, 2000), [0, 0, M - 1, M - 1]])
    cols = np.concatenate([g.integers(0, N, 2000), [0, N - 1, 0, N - 1]])
    assert_bits(got[:, rows, cols], orc.matmul_pruned(A, B, nc=nc, rows=rows, cols=cols), "pruned large")


def test_pruned_8192_f32_nc3_sampled(mcf, orc):
    """The 8192^3 binary32 nc = 3 workload: 128 sampled outputs bitwise against the
    oracle's pruned product and within 4 K u^3 of the exact product."""
    n, nc = 8192, 3
    A, B = inputs.matmul_normal(n, n, n, nc, np.float32, seed=0)
    got = to_host(mcf.mc_matmul_pruned(to_dev(A), to_dev(B), nc=nc))
    g = np.random.default_rng(1770)
    rows = np.concatenate([g.integers(0, n, 124), [0, 0, n - 1, n - 1]])
    cols = np.concatenate([g.integers(0, n, 124), [0, n - 1, 0, n - 1]])
    Cs = np.ascontiguousarray(got[:, rows, cols])
    assert_bits(Cs, orc.matmul_pruned(A, B, nc=nc, rows=rows, cols=cols), "pruned 8192^3")
    assert bound_ok(orc, A, B, Cs, nc, n, np.float32, rows=rows, cols=cols)


def test_pruned_1024_f16(mcf, orc):
    n = 1024
    for nc in (2, 3):
        A, B = inputs.matmul_normal(n, n, n, nc, np.float16, seed=0)
        got = to_host(mcf.mc_matmul_pruned(to_dev(A), to_dev(B), nc=nc))
        g = np.random.default_rng(1780 + nc)
        rows, cols = g.integers(0, n, 300), g.integers(0, n, 300)
        assert_bits(got[:, rows, cols], orc.matmul_pruned(A, B, nc=nc, rows=rows, cols=cols), f"pruned 1024 nc={nc}")
