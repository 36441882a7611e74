"""GPU parity of the K-split MC matrix product against the CPU oracle.

The K-split product is a fixed function of the slice count S (round-robin slices,
each summed in MM-MCN order, pairwise Add-MCN tree over the slice sums), so the GPU
result is compared bitwise with the oracle's evaluation of the same function, for
slice counts that keep the tree inside one workgroup (S <= 256) and that need the
second reduction kernel (S > 256), ragged in every dimension.  The error against
the exact product is checked with the MM-MCN bound as well.
"""
import numpy as np
import pytest

from paper_2207_08867_amd import inputs
from test_gpu_elementwise import assert_bits, to_dev, to_host
from test_gpu_matmul import check_bound

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def mcf():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2207_08867_amd as m

    m.lib()
    return m


@pytest.mark.parametrize("dt", [np.float16, np.float32])
@pytest.mark.parametrize("nc", [1, 2, 3, 4])
@pytest.mark.parametrize("kinds", [(True, True), (True, False), (False, True)])
def test_small_parity(mcf, orc, dt, nc, kinds):
    a_mc, b_mc = kinds
    M, N, K = 7, 5, 611
    A, B = inputs.matmul_normal(M, N, K, nc, dt, seed=90 + nc)
    A = A if a_mc else A[:1]
    B = B if b_mc else B[:1]
    tA, tB = to_dev(A), to_dev(B)
    for S in (1, 3, 16, 37, 256, 257, 600, 611, 5000):
        got = to_host(mcf.mc_matmul_splitk(tA, tB, nc=nc, a_mc=a_mc, b_mc=b_mc, slices=S))
        want = orc.matmul_splitk(A, B, nc=nc, a_mc=a_mc, b_mc=b_mc, slices=S)
        assert_bits(got, want, f"splitk {dt.__name__} nc={nc} {kinds} S={S}")
    check_bound(orc, A, B, got, nc, K, dt)


def test_one_slice_equals_mc_matmul(mcf):
    A, B = inputs.matmul_normal(70, 45, 37, 3, np.float32, seed=95)
    tA, tB = to_dev(A), to_dev(B)
    assert_bits(to_host(mcf.mc_matmul_splitk(tA, tB, nc=3, slices=1)), to_host(mcf.mc_matmul(tA, tB, nc=3)),
                "S = 1")


@pytest.mark.parametrize("dt,nc", [(np.float32, 2), (np.float32, 3), (np.float16, 3)])
def test_dot(mcf, orc, dt, nc):
    """Dot-MCN (M = N = 1), K = 200003, default slice count (3125: 13 workgroups)."""
    K = 200003
    A, B = inputs.matmul_normal(1, 1, K, nc, dt, seed=96)
    S = mcf.mc_matmul_splitk_slices(1, 1, K)
    assert S == K // 64
    got = to_host(mcf.mc_matmul_splitk(to_dev(A), to_dev(B[:1]), nc=nc, b_mc=False))
    want = orc.matmul_splitk(A, B[:1], nc=nc, b_mc=False, slices=S)
    assert_bits(got, want, f"dot {dt.__name__} nc={nc}")
    check_bound(orc, A, B[:1], got, nc, K, dt)


def test_dot_max_slices(mcf, orc):
    """65536 slices (256 workgroups of 256, a 256-lane second tree), K = 2^20 + 3."""
    K = (1 << 20) + 3
    A, B = inputs.matmul_normal(1, 1, K, 2, np.float32, seed=97)
    got = to_host(mcf.mc_matmul_splitk(to_dev(A), to_dev(B), nc=2, slices=65536))
    want = orc.matmul_splitk(A, B, nc=2, slices=65536)
    assert_bits(got, want, "dot 65536 slices")
    check_bound(orc, A, B, got, 2, K, np.float32)


@pytest.mark.parametrize("S", [70000, 1 << 18, 300000, 1 << 20])
def test_dot_many_groups(mcf, orc, S):
    """More than 256 slice groups: the second launch folds aligned blocks of 4 or 16
    group roots per lane before its lane tree.  S = 70000: 274 groups, blocks of 4,
    the last one partial; S = 2^18 (the default Dot slice count): 1024 groups, 256 full
    blocks of 4; S = 300000: 1172 groups, blocks of 16, the last of 4 roots; S = 2^20
    (the maximum): 4096 groups, 256 full blocks of 16.  K = 2^21 + 3, so the largest S
    has two or three steps per slice."""
    K = (1 << 21) + 3
    A, B = inputs.matmul_normal(1, 1, K, 2, np.float32, seed=98)
    got = to_host(mcf.mc_matmul_splitk(to_dev(A), to_dev(B), nc=2, slices=S))
    want = orc.matmul_splitk(A, B, nc=2, slices=S)
    assert_bits(got, want, f"dot {S} slices")
    check_bound(orc, A, B, got, 2, K, np.float32)


@pytest.mark.parametrize("dt", [np.float16, np.float32])
def test_small_outputs_many_groups(mcf, orc, dt):
    """Several outputs (3 x 2, MC x MC, nc = 3) with 70000 slices: 274 group roots per
    output, folded in blocks of 4 by a 128-lane group per output in the second
    launch."""
    M, N, K, nc = 3, 2, 150_001, 3
    A, B = inputs.matmul_normal(M, N, K, nc, dt, seed=99)
    got = to_host(mcf.mc_matmul_splitk(to_dev(A), to_dev(B), nc=nc, slices=70000))
    want = orc.matmul_splitk(A, B, nc=nc, slices=70000)
    assert_bits(got, want, f"small outputs {dt.__name__}")


@pytest.mark.parametrize("dt", [np.float16, np.float32])
def test_mv(mcf, orc, dt):
    """MV-MCN (N = 1), M = 1000, K = 4099, default slice count."""
    M, K, nc = 1000, 4099, 3
    A, B = inputs.matmul_normal(M, 1, K, nc, dt, seed=98)
    S = mcf.mc_matmul_splitk_slices(M, 1, K)
    got = to_host(mcf.mc_matmul_splitk(to_dev(A), to_dev(B[:1]), nc=nc, b_mc=False))
    want = orc.matmul_splitk(A, B[:1], nc=nc, b_mc=False, slices=S)
    assert_bits(got, want, f"mv {dt.__name__} S={S}")
    check_bound(orc, A, B[:1], got, nc, K, dt)


@pytest.mark.parametrize("slices", [0, 8])
def test_config_64_fp32_nc2(mcf, orc, slices):
    """The 64^3 binary32 nc = 2 workload (uniform [-1, 1], seed 0) through the K-split
    product, with its default slice count (1 at this size, where a slice keeps at least
    64 steps) and with 8 slices: bitwise against the oracle's K-split product, and
    within 2^-40 relative of the exact product."""
    A, B = inputs.matmul_uniform(64, 64, 64, 2, np.float32, seed=0)
    S = slices or mcf.mc_matmul_splitk_slices(64, 64, 64)
    got = to_host(mcf.mc_matmul_splitk(to_dev(A), to_dev(B), nc=2, slices=slices))
    assert_bits(got, orc.matmul_splitk(A, B, nc=2, slices=S), f"64^3 split S={S}")
    assert check_bound(orc, A, B, got, 2, 64, np.float32) < 2.0 ** -40


def test_workspace_reuse_and_degenerate(mcf, orc):
    import torch

    A, B = inputs.matmul_normal(3, 4, 3000, 3, np.float32, seed=99)
    tA, tB = to_dev(A), to_dev(B)
    nbytes = mcf.mc_matmul_splitk_workspace(1, 3, 3, 4, 3000, True, True, 1000)
    assert nbytes == 4 * 3 * 3 * 12 * 4
    ws = torch.full((nbytes,), 0xFF, dtype=torch.uint8, device="cuda")  # contents on entry do not matter
    want = orc.matmul_splitk(A, B, nc=3, slices=1000)
    for _ in range(2):
        assert_bits(to_host(mcf.mc_matmul_splitk(tA, tB, nc=3, slices=1000, workspace=ws)), want, "reuse")
    with pytest.raises(ValueError):
        mcf.mc_matmul_splitk(tA, tB, nc=3, slices=1000, workspace=ws[:-1])
    with pytest.raises(ValueError):  # above the maximum of 2^20 slices
        mcf.mc_matmul_splitk(tA, tB, nc=3, slices=(1 << 20) + 1)
    Z = to_host(mcf.mc_matmul_splitk(to_dev(np.zeros((3, 5, 0), np.float32)), to_dev(np.zeros((3, 0, 6), np.float32)),
                                     nc=3, slices=8))
    assert Z.shape == (3, 5, 6) and (Z == 0).all() and not np.signbit(Z).any()
    E = mcf.mc_matmul_splitk(to_dev(np.zeros((3, 0, 9), np.float32)), to_dev(np.zeros((3, 9, 6), np.float32)), nc=3)
    assert tuple(E.shape) == (3, 0, 6)


def test_bench_shapes(mcf, orc):
    """The K-split launch configurations the benchmark times (default slice counts):
    Dot of two binary32 nc = 2 MC vectors at the 2^18 slices of a 2^24 Dot (1024
    workgroups of 256 slices, then one launch that folds the 1024 group roots in
    blocks of 4 per lane and runs a 256-lane tree over them) with K = 2^22 + 5 (the
    same launch; the one-output oracle is sequential), bitwise and within the bound;
    MV of an 8192 x 8192 binary32 nc = 3 MC matrix by a plain vector (128 slices), in
    full on the GPU, on 48 sampled rows."""
    K = (1 << 22) + 5
    S = mcf.mc_matmul_splitk_slices(1, 1, 1 << 24)
    assert S == 1 << 18
    A, B = inputs.matmul_normal(1, 1, K, 2, np.float32, seed=0)
    got = to_host(mcf.mc_matmul_splitk(to_dev(A), to_dev(B), nc=2, slices=S))
    assert_bits(got, orc.matmul_splitk(A, B, nc=2, slices=S), "dot 2^24")
    check_bound(orc, A, B, got, 2, K, np.float32)
    n = 8192
    A, B = inputs.matmul_normal(n, 1, n, 3, np.float32, seed=0)
    got = to_host(mcf.mc_matmul_splitk(to_dev(A), to_dev(B[:1]), nc=3, b_mc=False))
    S = mcf.mc_matmul_splitk_slices(n, 1, n)
    g = np.random.default_rng(47)
    rows = np.concatenate([g.integers(0, n, 46), [0, n - 1]])
    cols = np.zeros_like(rows)
    want = orc.matmul_splitk(A, B[:1], nc=3, b_mc=False, slices=S, rows=rows, cols=cols)
    assert_bits(got[:, rows, cols], want, "mv 8192")
