"""GPU parity of the matrix products against the CPU oracle when products of the
operands overflow although every entry is finite: the infinite leading component and
the NaN components behind it come out as the algorithms leave them, bit for bit (NaNs
by class).  The overflowing term sits at the first, a middle or the last reduction
step, and K = 1 stores the single ScalingN term as the result (no Add-MCN after it).
Sequential MM-MCN for every operand kind, the pruned product, the K-split product and
MC-Linear, binary16 and binary32, nc = 2 and 3."""
import numpy as np
import pytest

from paper_2207_08867_amd import inputs
from test_gpu_elementwise import assert_bits, to_dev, to_host

pytestmark = pytest.mark.gpu

BIG = {np.float16: 300.0, np.float32: 1.9e19}  # BIG^2 overflows the format


@pytest.fixture(scope="module")
def mcf():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2207_08867_amd as m

    m.lib()
    return m


def operands(dt, nc, K, kpos, seed=5):
    """Entries in (-1, 1) except a large one at reduction step kpos in every other row
    of A and every third column of B, so those outputs have one overflowing term."""
    g = np.random.default_rng(seed)
    M, N = 64, 48
    a = g.uniform(-1, 1, (M, K))
    b = g.uniform(-1, 1, (K, N))
    a[::2, kpos] = BIG[dt] * np.sign(a[::2, kpos])
    b[kpos, ::3] = BIG[dt] * np.sign(b[kpos, ::3])
    return inputs.split(a, nc, dt), inputs.split(b, nc, dt)


def check(got, want, what):
    lead = want[0].astype(np.float64)
    assert np.isinf(lead).any(), what  # the case occurs
    assert_bits(got, want, what)


@pytest.mark.parametrize("dt", [np.float16, np.float32])
@pytest.mark.parametrize("nc", [2, 3])
@pytest.mark.parametrize("K,kpos", [(1, 0), (37, 0), (37, 18), (37, 36)])
def test_matmul_overflow(mcf, orc, dt, nc, K, kpos):
    A, B = operands(dt, nc, K, kpos)
    for a_mc, b_mc in ((True, True), (True, False), (False, True)):
        Aa = A if a_mc else A[:1]
        Bb = B if b_mc else B[:1]
        got = to_host(mcf.mc_matmul(to_dev(Aa), to_dev(Bb), nc=nc, a_mc=a_mc, b_mc=b_mc))
        check(got, orc.matmul(Aa, Bb, nc=nc, a_mc=a_mc, b_mc=b_mc), f"matmul {a_mc, b_mc} K={K} at {kpos}")


@pytest.mark.parametrize("dt", [np.float16, np.float32])
@pytest.mark.parametrize("nc", [2, 3])
@pytest.mark.parametrize("K,kpos", [(1, 0), (37, 36)])
def test_pruned_and_splitk_overflow(mcf, orc, dt, nc, K, kpos):
    A, B = operands(dt, nc, K, kpos)
    check(to_host(mcf.mc_matmul_pruned(to_dev(A), to_dev(B), nc=nc)), orc.matmul_pruned(A, B, nc=nc),
          f"pruned K={K}")
    for S in (1, 4):
        for a_mc, b_mc in ((True, True), (True, False)):
            Aa = A if a_mc else A[:1]
            Bb = B if b_mc else B[:1]
            got = to_host(mcf.mc_matmul_splitk(to_dev(Aa), to_dev(Bb), nc=nc, a_mc=a_mc, b_mc=b_mc, slices=S))
            check(got, orc.matmul_splitk(Aa, Bb, nc=nc, slices=S, a_mc=a_mc, b_mc=b_mc), f"splitk S={S} K={K}")


@pytest.mark.parametrize("dt", [np.float16, np.float32])
@pytest.mark.parametrize("K", [1, 37])
def test_linear_overflow(mcf, orc, dt, K):
    A, B = operands(dt, 3, K, K - 1)
    x = np.ascontiguousarray(A[0])                     # (batch, in) plain
    W = np.ascontiguousarray(B.transpose(0, 2, 1))     # (nc, out, in)
    b = inputs.split(np.linspace(-1, 1, W.shape[1]), 3, dt)
    for bias in (None, b):
        got = to_host(mcf.mc_linear_fwd(to_dev(x), to_dev(W), None if bias is None else to_dev(bias)))
        check(got, orc.linear(x, W, bias, nc=3), f"linear K={K} bias={bias is not None}")
