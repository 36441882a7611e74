"""GPU parity of the exact binary16 MC product (int8 matrix cores) against the CPU
oracle, bitwise: the exact product split into nc components by successive rounding.

Covers ragged shapes across several 64 x 64 tiles, every operand kind and the
transposed (linear-layer) B, both digit-range instantiations (values needing at most
four 7-bit digit levels and values needing more), digit ranges that start above
level 0, reductions longer than one int32 accumulation chunk, non-finite inputs,
overflow, K = 0, workspace reuse, and the benchmark sizes at sampled outputs.
"""
import numpy as np
import pytest

from oracle import exact_product as xp
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


def operands(M, N, K, nc, seed, a_mc=True, b_mc=True, scale_a=1.0, scale_b=1.0):
    g = np.random.default_rng(seed)
    A = inputs.split(g.normal(0.0, scale_a / np.sqrt(max(K, 1)), (M, K)), nc, np.float16)
    B = inputs.split(g.normal(0.0, scale_b / np.sqrt(max(K, 1)), (K, N)), nc, np.float16)
    return (A if a_mc else A[:1]), (B if b_mc else B[:1])


def run(mcf, A, B, nc, a_mc=True, b_mc=True, b_trans=False, workspace=None):
    Bd = np.ascontiguousarray(np.swapaxes(B, 1, 2)) if b_trans else B
    return to_host(mcf.mc_matmul_exact(to_dev(A), to_dev(Bd), nc=nc, a_mc=a_mc, b_mc=b_mc, b_trans=b_trans,
                                       workspace=workspace))


KINDS = [(True, True), (True, False), (False, True)]


@pytest.mark.parametrize("nc", [1, 2, 3, 4])
@pytest.mark.parametrize("kinds", KINDS)
@pytest.mark.parametrize("b_trans", [False, True])
def test_exact_small_ragged(mcf, nc, kinds, b_trans):
    a_mc, b_mc = kinds
    M, N, K = 70, 45, 37
    A, B = operands(M, N, K, nc, 2000 + nc, a_mc, b_mc)
    got = run(mcf, A, B, nc, a_mc, b_mc, b_trans)
    assert_bits(got, xp.matmul_exact(A, B, nc=nc, a_mc=a_mc, b_mc=b_mc), f"exact nc={nc} {kinds} T={b_trans}")


@pytest.mark.parametrize("shape", [(1, 1, 1), (16, 16, 64), (64, 64, 64), (65, 63, 129), (3, 130, 65), (129, 2, 200)])
def test_exact_shapes(mcf, shape):
    M, N, K = shape
    A, B = operands(M, N, K, 3, 2100 + M)
    got = run(mcf, A, B, 3)
    assert_bits(got, xp.matmul_exact(A, B, nc=3), f"exact shape {shape}")


@pytest.mark.parametrize("scales", [(1e3, 1e3), (1e4, 1.0), (1e-3, 1e-2)])
def test_exact_digit_ranges(mcf, scales):
    """Large entries need five or more digit levels (the wide instantiation); small
    ones use only the low levels."""
    A, B = operands(40, 50, 96, 3, 2200, scale_a=scales[0] * np.sqrt(96), scale_b=scales[1] * np.sqrt(96))
    got = run(mcf, A, B, 3)
    assert_bits(got, xp.matmul_exact(A, B, nc=3), f"exact scales {scales}")


def test_exact_levels_above_zero(mcf):
    """Entries that are multiples of 2^-8 have zero low digits: the level range
    starts above 0 and the result is shifted accordingly."""
    g = np.random.default_rng(2300)
    A = np.zeros((2, 33, 70), np.float16)
    B = np.zeros((2, 70, 31), np.float16)
    A[0] = (g.integers(-2000, 2000, (33, 70)) * 2.0 ** -8).astype(np.float16)
    B[0] = (g.integers(-2000, 2000, (70, 31)) * 2.0 ** -6).astype(np.float16)
    got = run(mcf, A, B, 2)
    assert_bits(got, xp.matmul_exact(A, B, nc=2), "levels above zero")


def test_exact_overlapping_components(mcf):
    """Components that overlap (not a normalised expansion) and reach the top of the
    binary16 range: up to seven digit levels, results that overflow."""
    g = np.random.default_rng(2400)
    A = g.uniform(-60000, 60000, (4, 20, 30)).astype(np.float16)
    B = g.uniform(-1, 1, (4, 30, 25)).astype(np.float16)
    B[:, :, :5] *= np.float16(2.0 ** -14)
    got = run(mcf, A, B, 4)
    assert_bits(got, xp.matmul_exact(A, B, nc=4), "overlapping components")
    assert np.isinf(got[0]).any()


def test_exact_long_reduction(mcf):
    """K beyond one int32 accumulation chunk (65536): partial sums in the workspace."""
    M, N, K = 3, 5, 70000
    A, B = operands(M, N, K, 2, 2500)
    got = run(mcf, A, B, 2)
    assert_bits(got, xp.matmul_exact(A, B, nc=2), "K = 70000")


def test_exact_nonfinite_overflow_and_empty(mcf):
    A, B = operands(30, 20, 40, 2, 2600)
    A[1, 4, 7] = np.inf
    A[0, 9, 0] = -np.inf
    B[0, 3, 11] = np.nan
    got = run(mcf, A, B, 2)
    assert_bits(got, xp.matmul_exact(A, B, nc=2), "non-finite")
    nan = np.isnan(got[0])
    assert nan[4].all() and nan[9].all() and nan[:, 11].all() and nan.sum() == 2 * 20 + 30 - 2
    A2 = np.zeros((2, 3, 4), np.float16)
    A2[0] = 30000
    B2 = np.zeros((2, 4, 2), np.float16)
    B2[0] = -2
    got = run(mcf, A2, B2, 2)
    assert np.all(np.isneginf(got[0])) and not got[1].any()
    assert_bits(got, xp.matmul_exact(A2, B2, nc=2), "overflow")
    import torch

    Z = mcf.mc_matmul_exact(torch.zeros((3, 5, 0), dtype=torch.float16, device="cuda"),
                            torch.zeros((3, 0, 4), dtype=torch.float16, device="cuda"), nc=3)
    assert Z.shape == (3, 5, 4) and not to_host(Z).view(np.uint16).any()


def test_exact_workspace_reuse(mcf):
    """A workspace keeps nothing between calls: a larger call, then a smaller one
    with entries on other digit levels, through the same workspace."""
    import torch

    nc = 3
    ws = torch.empty(mcf.mc_matmul_exact_workspace(nc, 200, 150, 300), dtype=torch.uint8, device="cuda")
    A, B = operands(200, 150, 300, nc, 2700, scale_a=500.0)
    got = run(mcf, A, B, nc, workspace=ws)
    r = np.array([0, 199, 57, 100])
    c = np.array([0, 149, 3, 77])
    assert_bits(got[:, r, c], xp.matmul_exact(A, B, nc=nc, rows=r, cols=c), "first call")
    A2, B2 = operands(37, 29, 45, nc, 2701)
    A2[0, 5, 5] = np.nan
    got2 = run(mcf, A2, B2, nc, workspace=ws)
    assert_bits(got2, xp.matmul_exact(A2, B2, nc=nc), "second call")
    A3, B3 = operands(37, 29, 45, nc, 2702)
    got3 = run(mcf, A3, B3, nc, workspace=ws)
    assert_bits(got3, xp.matmul_exact(A3, B3, nc=nc), "third call (no stale non-finite flag)")


def sample_positions(M, N, n, seed):
    g = np.random.default_rng(seed)
    r = np.concatenate([[0, M - 1, 0, M - 1], g.integers(0, M, n)])
    c = np.concatenate([[0, N - 1, N - 1, 0], g.integers(0, N, n)])
    return r, c


@pytest.mark.parametrize("nc", [2, 3])
def test_exact_1024_cube_sampled(mcf, nc):
    """The 1024^3 binary16 MC x MC workload, checked at sampled outputs."""
    A, B = inputs.matmul_normal(1024, 1024, 1024, nc, np.float16, seed=2800 + nc)
    got = run(mcf, A, B, nc)
    r, c = sample_positions(1024, 1024, 60, 2810 + nc)
    assert_bits(got[:, r, c], xp.matmul_exact(A, B, nc=nc, rows=r, cols=c), f"1024^3 nc={nc}")


def test_exact_linear_layer_sampled(mcf):
    """The MC-Linear layer product x W^T (x plain 4096 x 1024, W MC 1024 x 1024,
    binary16, nc = 3), weight in its stored [out][in] layout, at sampled outputs."""
    nc = 3
    X, W, _ = next(inputs.linear_inputs(4096, 1024, 1024, nc, np.float16, seed=2900))
    got = to_host(mcf.mc_matmul_exact(to_dev(X), to_dev(W), nc=nc, a_mc=False, b_mc=True, b_trans=True))
    r, c = sample_positions(4096, 1024, 60, 2901)
    WT = np.ascontiguousarray(np.swapaxes(W, 1, 2))
    assert_bits(got[:, r, c], xp.matmul_exact(X.reshape(1, 4096, 1024), WT, nc=nc, a_mc=False, rows=r, cols=c),
                "linear 4096x1024x1024")


def test_exact_argument_errors(mcf):
    import torch

    A = torch.zeros((2, 8, 6), dtype=torch.float32, device="cuda")
    B = torch.zeros((2, 6, 5), dtype=torch.float32, device="cuda")
    with pytest.raises(ValueError):  # binary16 only
        mcf.mc_matmul_exact(A, B, nc=2)
    A = A.half()
    B = B.half()
    with pytest.raises(ValueError):  # workspace too small
        mcf.mc_matmul_exact(A, B, nc=2, workspace=torch.empty(16, dtype=torch.uint8, device="cuda"))


@pytest.mark.parametrize("nc", [1, 2, 3])
def test_exact_linear_with_bias(mcf, nc):
    """mc_linear_fwd_exact: y = x W^T + b, the bias added to the exact sum."""
    T, I, O = 70, 37, 45
    g = np.random.default_rng(3100 + nc)
    x = g.normal(0, 1, (T, I)).astype(np.float16)
    W = inputs.split(g.uniform(-1 / np.sqrt(I), 1 / np.sqrt(I), (O, I)), nc, np.float16)
    b = inputs.split(g.uniform(-1 / np.sqrt(I), 1 / np.sqrt(I), O), nc, np.float16)
    WT = np.ascontiguousarray(np.swapaxes(W, 1, 2))
    got = to_host(mcf.mc_linear_fwd_exact(to_dev(x), to_dev(W), to_dev(b)))
    assert_bits(got, xp.matmul_exact(x[None], WT, nc=nc, a_mc=False, bias=b), f"linear exact nc={nc}")
    got = to_host(mcf.mc_linear_fwd_exact(to_dev(x), to_dev(W)))
    assert_bits(got, xp.matmul_exact(x[None], WT, nc=nc, a_mc=False), f"linear exact no bias nc={nc}")
    b[nc - 1, 7] = np.nan
    got = to_host(mcf.mc_linear_fwd_exact(to_dev(x), to_dev(W), to_dev(b)))
    assert np.isnan(got[:, :, 7]).all() and not np.isnan(np.delete(got, 7, axis=2)).any()


def test_exact_linear_layer_with_bias_sampled(mcf):
    """The MC-Linear layer y = x W^T + b at 4096 x 1024 x 1024, binary16 nc = 3."""
    nc = 3
    X, W, b = next(inputs.linear_inputs(4096, 1024, 1024, nc, np.float16, seed=3200))
    got = to_host(mcf.mc_linear_fwd_exact(to_dev(X), to_dev(W), to_dev(b)))
    r, c = sample_positions(4096, 1024, 60, 3201)
    WT = np.ascontiguousarray(np.swapaxes(W, 1, 2))
    assert_bits(got[:, r, c], xp.matmul_exact(X[None], WT, nc=nc, a_mc=False, bias=b, rows=r, cols=c),
                "linear 4096x1024x1024 with bias")
