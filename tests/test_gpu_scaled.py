"""GPU parity of binary16 with scaled low components (format MCF_F16S) against the
CPU oracle, bitwise: elementwise Add-MCN and ScalingN, the product in every operand
kind, MC-Linear; plus the stated product tolerance 4 K u^nc (|A||B|), as written, on
the 1024^3 workload at nc = 3 -- which plain binary16 components miss (the floor of
Section 2.4).  Inputs include exact cancellations and zeroed components so that the
general (compaction) path of every step runs beside the common one."""
import numpy as np
import pytest

from paper_2207_08867_amd import inputs
from test_gpu_elementwise import assert_bits, to_dev, to_host

pytestmark = pytest.mark.gpu

U16 = 2.0 ** -11


@pytest.fixture(scope="module")
def mcf():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2207_08867_amd as m

    m.lib()
    return m


def scaled_values(g, shape, nc, spread=8):
    """Scaled MC values with magnitudes 2^-spread .. 1, some exact zeros, some zeroed
    middle components and some values whose low components are zero."""
    x = g.uniform(-1, 1, shape) * np.exp2(g.integers(-spread, 1, shape))
    s = inputs.split_scaled(x, nc)
    flat = s.reshape(nc, -1)
    m = flat.shape[1]
    flat[:, g.integers(0, m, m // 50)] = 0
    if nc > 1:
        flat[1:, g.integers(0, m, m // 50)] = 0
        flat[nc // 2, g.integers(0, m, m // 50)] = 0
    return s


@pytest.mark.parametrize("nc", [1, 2, 3, 4])
@pytest.mark.parametrize("n", [4099, 8192])
def test_elementwise_parity(mcf, orc, nc, n):
    g = np.random.default_rng(100 + nc + n)
    x = scaled_values(g, n, nc)
    y = scaled_values(g, n, nc)
    y[:, : n // 16] = -x[:, : n // 16]  # exact cancellations
    v = (g.uniform(-1, 1, n) * np.exp2(g.integers(-6, 2, n))).astype(np.float16)
    v[g.integers(0, n, n // 40)] = 0
    tx, ty, tv = to_dev(x), to_dev(y), to_dev(v)
    assert_bits(to_host(mcf.mc_add(tx, ty, nc=nc, scaled=True)), orc.scaled_add(x, y, nc=nc), f"add nc={nc}")
    want = orc.scaled_mul(x, v[None], nc=nc)
    assert_bits(to_host(mcf.mc_mul(tx, tv, nc=nc, y_mc=False, scaled=True)), want, f"mul MC,T nc={nc}")
    assert_bits(to_host(mcf.mc_mul(tv, tx, nc=nc, x_mc=False, scaled=True)), want, f"mul T,MC nc={nc}")
    # in place
    t2 = to_dev(x)
    mcf.mc_add(t2, ty, nc=nc, out=t2, scaled=True)
    assert_bits(to_host(t2), orc.scaled_add(x, y, nc=nc), f"add in place nc={nc}")


@pytest.mark.parametrize("nc", [2, 3])
def test_scaling_overflow(mcf, orc, nc):
    """ScalingN whose leading product overflows although both factors are finite:
    bitwise against the algorithm (the NaN carry behind the infinite product)."""
    g = np.random.default_rng(120 + nc)
    n = 4099
    x = inputs.split_scaled(g.choice([-1.0, 1.0], n) * g.uniform(0.3, 1.0, n) * 65504.0, nc)
    v = (g.choice([-1.0, 1.0], n) * g.uniform(1.0, 4.0, n)).astype(np.float16)
    want = orc.scaled_mul(x, v[None], nc=nc)
    lead = want[0].astype(np.float64)
    assert np.isinf(lead).any() and np.isfinite(lead).any()
    tx, tv = to_dev(x), to_dev(v)
    assert_bits(to_host(mcf.mc_mul(tx, tv, nc=nc, y_mc=False, scaled=True)), want, f"scaled overflow nc={nc}")
    assert_bits(to_host(mcf.mc_mul(tv, tx, nc=nc, x_mc=False, scaled=True)), want, f"scaled overflow T,MC nc={nc}")


def test_elementwise_kinds_not_provided(mcf):
    import torch

    x = torch.zeros((3, 64), dtype=torch.float16, device="cuda")
    v = torch.zeros(64, dtype=torch.float16, device="cuda")
    with pytest.raises(ValueError, match="MCF_E_DTYPE"):
        mcf.mc_add(x, v, nc=3, y_mc=False, scaled=True)  # Grow-ExpN pairs levels
    with pytest.raises(ValueError, match="MCF_E_DTYPE"):
        mcf.mc_mul(x, x, nc=3, scaled=True)  # Mult-MCN
    with pytest.raises(TypeError):
        mcf.mc_add(x.float(), x.float(), nc=3, scaled=True)


@pytest.mark.parametrize("nc", [1, 2, 3, 4])
@pytest.mark.parametrize("kinds", [(True, True), (True, False), (False, True)])
def test_product_parity_ragged(mcf, orc, nc, kinds):
    a_mc, b_mc = kinds
    M, N, K = 70, 45, 37
    g = np.random.default_rng(200 + nc)
    A = scaled_values(g, (M, K), nc, spread=4)
    B = scaled_values(g, (K, N), nc, spread=4)
    A = A if a_mc else A[:1]
    B = B if b_mc else B[:1]
    got = to_host(mcf.mc_matmul(to_dev(A), to_dev(B), nc=nc, a_mc=a_mc, b_mc=b_mc, scaled=True))
    want = orc.scaled_matmul(A, B, nc=nc, a_mc=a_mc, b_mc=b_mc)
    assert_bits(got, want, f"scaled matmul nc={nc} {kinds}")


@pytest.mark.parametrize("shape", [(1, 1, 300), (1, 97, 64), (97, 1, 64), (33, 31, 1), (5, 7, 0), (17, 16, 33)])
def test_product_degenerate_shapes(mcf, orc, shape):
    M, N, K = shape
    A, B = inputs.matmul_normal_scaled(M, N, K, 3, seed=7)
    got = to_host(mcf.mc_matmul(to_dev(A), to_dev(B), nc=3, scaled=True))
    assert_bits(got, orc.scaled_matmul(A, B, nc=3), f"scaled matmul {shape}")


def _literal(orc, A, B, C, nc, K, rows, cols, bias=None):
    err, absab, _ = orc.matmul_exact_err(orc.unscale(A), orc.unscale(B), orc.unscale(C), rows=rows, cols=cols,
                                         bias=None if bias is None else orc.unscale(bias))
    return float(np.max(np.abs(err) / absab)) / (4 * K * U16 ** nc)


@pytest.mark.parametrize("nc", [2, 3])
def test_config_1024_literal_bound(mcf, orc, nc):
    """M = N = K = 1024, entries N(0, 1/K) split into scaled binary16 components:
    2048 sampled outputs bitwise against the oracle and within 4 K u^nc of the exact
    product as written (no floor)."""
    n = 1024
    A, B = inputs.matmul_normal_scaled(n, n, n, nc, seed=0)
    got = to_host(mcf.mc_matmul(to_dev(A), to_dev(B), nc=nc, scaled=True))
    g = np.random.default_rng(300 + nc)
    rows = np.concatenate([g.integers(0, n, 2044), [0, 0, n - 1, n - 1]])
    cols = np.concatenate([g.integers(0, n, 2044), [0, n - 1, 0, n - 1]])
    Cs = np.ascontiguousarray(got[:, rows, cols])
    assert_bits(Cs, orc.scaled_matmul(A, B, nc=nc, rows=rows, cols=cols), f"scaled 1024^3 nc={nc}")
    assert _literal(orc, A, B, Cs, nc, n, rows, cols) <= 1.0


@pytest.mark.parametrize("bias", [True, False])
def test_linear_small(mcf, orc, bias):
    x, W, b = next(inputs.linear_inputs_scaled(77, 53, 41, 3, seed=70))
    got = to_host(mcf.mc_linear_fwd(to_dev(x), to_dev(W), to_dev(b) if bias else None, scaled=True))
    assert_bits(got, orc.scaled_linear(x, W, b if bias else None, nc=3), f"scaled linear bias={bias}")


def test_linear_config_layer(mcf, orc):
    """Batch 4096, in 1024, out 1024, scaled binary16 nc = 3 (first layer): 2048
    sampled outputs bitwise and within 4 K u^3 (|x||W| + |b|) of the exact result."""
    T, I, O = 4096, 1024, 1024
    x, W, b = next(inputs.linear_inputs_scaled(T, I, O, 3, seed=0))
    got = to_host(mcf.mc_linear_fwd(to_dev(x), to_dev(W), to_dev(b), scaled=True))
    g = np.random.default_rng(310)
    rows = g.integers(0, T, 2048)
    cols = g.integers(0, O, 2048)
    Ys = np.ascontiguousarray(got[:, rows, cols])
    assert_bits(Ys, orc.scaled_linear(x, W, b, nc=3, rows=rows, cols=cols), "scaled linear layer")
    Wt = np.ascontiguousarray(W.transpose(0, 2, 1))
    assert _literal(orc, x[None], Wt, Ys, 3, I, rows, cols, bias=b) <= 1.0
