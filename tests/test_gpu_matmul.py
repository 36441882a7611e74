"""GPU parity of the MC matrix product and MC-Linear against the CPU oracle.

Each output is accumulated over k in MM-MCN order on the GPU as in the oracle, so
the comparison is bitwise.  The error against the exact product of the MC inputs
is checked as well: max_ij |C_ij - C*_ij| / (|A||B|)_ij <= 4 K u^nc as written
for the workloads (64^3 binary32 nc = 2, 1024^3 binary16 nc = 2, the MC-Linear
layers, 8192^3 binary32 nc = 3); elsewhere, and for 1024^3 binary16 nc = 3, with a
floor of nA nB K 2^-25 for Two-Prod errors that fall below the binary16 subnormal
grid.  Small cases span several 32x32 tiles with ragged edges; the
full-size workloads are checked on sampled outputs.
"""
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


def check_bound(orc, A, B, C, nc, K, dt, rows=None, cols=None, bias=None, literal=False):
    """Error against the exact product.  ScalingN and Add-MCN round their level-1
    carry, fl(e1 + e2), whose error is of order u^3 of the operands, so beyond
    nc = 3 the attainable accuracy stays at u^3: the bound uses u^min(nc, 3).
    literal=True checks the product's stated tolerance exactly as written,
    |C - C*| <= 4 K u^nc (|A||B|), with no binary16 floor."""
    err, absab, _ = orc.matmul_exact_err(A, B, C, rows=rows, cols=cols, bias=bias)
    u = U[dt]
    floor = A.shape[0] * B.shape[0] * K * 2.0 ** -25 if dt == np.float16 and not literal else 0.0
    lim = 4 * K * u ** (nc if literal else min(nc, 3)) * absab + floor
    ratio = np.abs(err) / np.where(lim > 0, lim, 1)
    assert (np.abs(err) <= lim).all(), f"bound exceeded: worst ratio {ratio.max():.3g}"
    return float(np.max(np.abs(err) / np.where(absab > 0, absab, 1)))


@pytest.mark.parametrize("dt", [np.float16, np.float32])
@pytest.mark.parametrize("nc", [1, 2, 3, 4])
@pytest.mark.parametrize("kinds", [(True, True), (True, False), (False, True)])
def test_small_ragged_parity(mcf, orc, dt, nc, kinds):
    a_mc, b_mc = kinds
    M, N, K = 70, 45, 37
    A, B = inputs.matmul_normal(M, N, K, nc, dt, seed=40 + nc)
    A = A if a_mc else A[:1]
    B = B if b_mc else B[:1]
    got = to_host(mcf.mc_matmul(to_dev(A), to_dev(B), nc=nc, a_mc=a_mc, b_mc=b_mc))
    want = orc.matmul(A, B, nc=nc, a_mc=a_mc, b_mc=b_mc)
    assert_bits(got, want, f"matmul {dt.__name__} nc={nc} {kinds}")
    check_bound(orc, A, B, got, nc, K, dt)


@pytest.mark.parametrize("shape", [(1, 1, 300), (1, 97, 64), (97, 1, 64), (33, 31, 1), (5, 7, 0), (129, 2, 3)])
def test_degenerate_shapes(mcf, orc, shape):
    M, N, K = shape
    nc, dt = 3, np.float32
    A, B = inputs.matmul_uniform(M, N, K, nc, dt, seed=50)
    got = to_host(mcf.mc_matmul(to_dev(A), to_dev(B), nc=nc))
    assert_bits(got, orc.matmul(A, B, nc=nc), f"matmul {shape}")


def test_config_64_fp32_nc2_exact(mcf, orc):
    """M = N = K = 64, binary32, nc = 2, A and B uniform in [-1, 1] (seed 0): every
    output bitwise and within 4 K u^2 of the exact product."""
    A, B = inputs.matmul_uniform(64, 64, 64, 2, np.float32, seed=0)
    got = to_host(mcf.mc_matmul(to_dev(A), to_dev(B), nc=2))
    assert_bits(got, orc.matmul(A, B, nc=2), "64^3")
    worst = check_bound(orc, A, B, got, 2, 64, np.float32, literal=True)
    assert worst < 2.0 ** -40


def config_1024_fp16(mcf, orc, nc, samples=2044):
    n = 1024
    A, B = inputs.matmul_normal(n, n, n, nc, np.float16, seed=0)
    got = to_host(mcf.mc_matmul(to_dev(A), to_dev(B), nc=nc))
    g = np.random.default_rng(60 + nc)
    rows = np.concatenate([g.integers(0, n, samples), [0, 0, n - 1, n - 1]])
    cols = np.concatenate([g.integers(0, n, samples), [0, n - 1, 0, n - 1]])
    want = orc.matmul(A, B, nc=nc, rows=rows, cols=cols)
    assert_bits(got[:, rows, cols], want, f"1024^3 nc={nc}")
    return A, B, np.ascontiguousarray(got[:, rows, cols]), rows, cols


def test_config_1024_fp16_nc2(mcf, orc):
    """M = N = K = 1024, binary16, nc = 2, entries N(0, 1/K): 2048 sampled outputs
    bitwise against the oracle and within the stated tolerance 4 K u^2 of the exact
    product as written (no floor)."""
    A, B, C, rows, cols = config_1024_fp16(mcf, orc, 2)
    worst = check_bound(orc, A, B, C, 2, 1024, np.float16, rows=rows, cols=cols, literal=True)
    assert worst < 4 * 1024 * 2.0 ** -22


def test_config_1024_fp16_nc3(mcf, orc):
    """The same at nc = 3.  binary16 components lose every Two-Prod error below the
    subnormal grid (2^-24), which the paper names as the limit of MC binary16 (Section
    2.4): the error is of the order of sqrt(K) eta (eta = 2^-25), about 11x the stated
    4 K u^3 on these inputs, and no smaller than at nc = 2.  Checked: bitwise parity,
    the bound with the binary16 floor nA nB K 2^-25, the rms errors of nc = 3 and
    nc = 2 within a factor 2 of each other (the paper's observation that more binary16
    components gain nothing), and that the literal tolerance is indeed missed here."""
    A, B, C, rows, cols = config_1024_fp16(mcf, orc, 3)
    worst3 = check_bound(orc, A, B, C, 3, 1024, np.float16, rows=rows, cols=cols)
    A2, B2, C2, rows2, cols2 = config_1024_fp16(mcf, orc, 2)
    check_bound(orc, A2, B2, C2, 2, 1024, np.float16, rows=rows2, cols=cols2)
    rms = []
    for a, b, c, r, q in ((A, B, C, rows, cols), (A2, B2, C2, rows2, cols2)):
        err, _, _ = orc.matmul_exact_err(a, b, c, rows=r, cols=q)
        rms.append(float(np.sqrt(np.mean(err * err))))
    assert 0.5 <= rms[0] / rms[1] <= 2.0, rms
    assert worst3 > 4 * 1024 * 2.0 ** -33  # the binary16 floor, not the component count, limits nc = 3


@pytest.mark.parametrize("kinds", [(True, True), (True, False), (False, True)])
def test_large_output_tile_path(mcf, orc, kinds):
    """Products with 2^25 or more outputs take the two-outputs-per-lane tile (the
    binary32 launch of the headline workload): 6001 x 5603 x 37, binary32, nc = 3,
    ragged in every dimension, checked on sampled outputs and the four corners."""
    a_mc, b_mc = kinds
    M, N, K, nc = 6001, 5603, 37, 3
    g = np.random.default_rng(45)
    A = inputs.split(g.normal(0, 1 / np.sqrt(K), (M, K)), nc if a_mc else 1, np.float32)
    B = inputs.split(g.normal(0, 1 / np.sqrt(K), (K, N)), nc if b_mc else 1, np.float32)
    got = to_host(mcf.mc_matmul(to_dev(A), to_dev(B), nc=nc, a_mc=a_mc, b_mc=b_mc))
    rows = np.concatenate([g.integers(0, M, 2000), [0, 0, M - 1, M - 1], np.full(16, M - 1)])
    cols = np.concatenate([g.integers(0, N, 2000), [0, N - 1, 0, N - 1], np.arange(N - 16, N)])
    want = orc.matmul(A, B, nc=nc, a_mc=a_mc, b_mc=b_mc, rows=rows, cols=cols)
    assert_bits(got[:, rows, cols], want, f"large tile {kinds}")


def test_config_8192_fp32_nc3_sampled(mcf, orc):
    """The 8192^3 binary32 nc = 3 MC x MC workload in the benchmark's launch
    configuration: 1024 sampled outputs bitwise against the oracle and within the
    stated tolerance 4 K u^3 of the exact product."""
    n, nc = 8192, 3
    A, B = inputs.matmul_normal(n, n, n, nc, np.float32, seed=0)
    got = to_host(mcf.mc_matmul(to_dev(A), to_dev(B), nc=nc))
    g = np.random.default_rng(46)
    rows = np.concatenate([g.integers(0, n, 1020), [0, 0, n - 1, n - 1]])
    cols = np.concatenate([g.integers(0, n, 1020), [0, n - 1, 0, n - 1]])
    want = orc.matmul(A, B, nc=nc, rows=rows, cols=cols)
    assert_bits(got[:, rows, cols], want, "8192^3")
    check_bound(orc, A, B, np.ascontiguousarray(got[:, rows, cols]), nc, n, np.float32, rows=rows, cols=cols,
                literal=True)


@pytest.mark.parametrize("bias", [True, False])
def test_linear_small(mcf, orc, bias):
    for dt in (np.float16, np.float32):
        x, W, b = next(inputs.linear_inputs(77, 53, 41, 3, dt, seed=70))
        got = to_host(mcf.mc_linear_fwd(to_dev(x), to_dev(W), to_dev(b) if bias else None))
        want = orc.linear(x, W, b if bias else None, nc=3)
        assert_bits(got, want, f"linear {dt.__name__} bias={bias}")


@pytest.fixture(scope="module")
def linear_layers():
    """Layers 0 and 99 of the MC-Linear workload (batch 4096, in 1024, out 1024,
    binary16 nc = 3, 100 layers drawn in order from seed 0)."""
    keep = {}
    for l, (x, W, b) in enumerate(inputs.linear_inputs(4096, 1024, 1024, 3, np.float16, layers=100, seed=0)):
        if l in (0, 99):
            keep[l] = (x, W, b)
    return keep


@pytest.mark.parametrize("layer", [0, 99])
def test_linear_config_layer(mcf, orc, linear_layers, layer):
    """Batch 4096, in 1024, out 1024, binary16 nc = 3: 4096 sampled outputs of the
    first and of the last layer bitwise against the oracle, and within the stated
    tolerance 4 K u^3 (|x||W| + |b|) of the exact result as written (no floor: with a
    plain x only about two of the three Two-Prods per step lose their error below the
    subnormal grid, and |x||W| is about 20 times larger than in the 1024^3 product)."""
    T, I, O = 4096, 1024, 1024
    x, W, b = linear_layers[layer]
    got = to_host(mcf.mc_linear_fwd(to_dev(x), to_dev(W), to_dev(b)))
    g = np.random.default_rng(71 + layer)
    rows = np.concatenate([g.integers(0, T, 4092), [0, 0, T - 1, T - 1]])
    cols = np.concatenate([g.integers(0, O, 4092), [0, O - 1, 0, O - 1]])
    want = orc.linear(x, W, b, nc=3, rows=rows, cols=cols)
    assert_bits(got[:, rows, cols], want, f"linear layer {layer}")
    Bm = np.ascontiguousarray(W.transpose(0, 2, 1))
    check_bound(orc, x[None], Bm, np.ascontiguousarray(got[:, rows, cols]), 3, I, np.float16, rows=rows, cols=cols,
                bias=b, literal=True)


def test_deterministic_and_errors(mcf):
    import torch

    A, B = inputs.matmul_normal(100, 90, 80, 3, np.float32, seed=80)
    tA, tB = to_dev(A), to_dev(B)
    c1 = to_host(mcf.mc_matmul(tA, tB, nc=3))
    c2 = to_host(mcf.mc_matmul(tA, tB, nc=3))
    assert_bits(c1, c2, "repeat")
    with pytest.raises(ValueError):  # wrong output shape
        mcf.mc_matmul(tA, tB, nc=3, out=torch.empty((3, 100, 91), dtype=torch.float32, device="cuda"))
    big = torch.empty((3, 100, 80), dtype=torch.float32, device="cuda")
    with pytest.raises(ValueError):  # output overlapping an input
        mcf.mc_matmul(big, tB[:, :80, :80].contiguous(), nc=3, out=big)
