"""GPU parity of the batched / broadcast product (BMM-MCN, 4DMM-MCN), AddMM-MCN and
the Matmul-MCN rank dispatch, bitwise against the CPU oracle."""
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


def operand(g, shape, nc, dt, is_mc):
    x = inputs.split(g.normal(0.0, 1.0 / np.sqrt(shape[-1]), shape), nc, dt)
    return x if is_mc else x[:1]


KINDS = [(True, True), (True, False), (False, True)]
SHAPES = [((3, 20, 17), (3, 17, 9)),            # BMM
          ((2, 1, 19, 13), (1, 3, 13, 21)),     # 4-D, both broadcast
          ((4, 18, 11), (2, 4, 11, 7)),         # 3-D against 4-D (missing leading dim)
          ((1, 16, 40), (5, 40, 33)),           # batch of one broadcast to five
          ((2, 3, 33, 5), (2, 3, 5, 34))]       # 4-D, no broadcast


@pytest.mark.parametrize("dt", [np.float16, np.float32])
@pytest.mark.parametrize("nc", [1, 2, 3])
@pytest.mark.parametrize("kinds", KINDS)
@pytest.mark.parametrize("shapes", SHAPES)
def test_batched_parity(mcf, orc, dt, nc, kinds, shapes):
    a_mc, b_mc = kinds
    g = np.random.default_rng(1000 + nc)
    A = operand(g, shapes[0], nc, dt, a_mc)
    B = operand(g, shapes[1], nc, dt, b_mc)
    got = to_host(mcf.mc_matmul_batched(to_dev(A), to_dev(B), nc=nc, a_mc=a_mc, b_mc=b_mc))
    want = orc.matmul_batched(A, B, nc=nc, a_mc=a_mc, b_mc=b_mc)
    assert_bits(got, want, f"batched {shapes} {dt.__name__} nc={nc} {kinds}")


def test_batched_many_batches(mcf, orc):
    """More batches than one launch's grid holds (65535): 70001 tiny products."""
    g = np.random.default_rng(1100)
    A = operand(g, (70001, 2, 3), 2, np.float32, True)
    B = operand(g, (70001, 3, 2), 2, np.float32, False)
    got = to_host(mcf.mc_matmul_batched(to_dev(A), to_dev(B), nc=2, a_mc=True, b_mc=False))
    idx = np.concatenate([np.arange(40), np.arange(65500, 65600), np.arange(70001 - 40, 70001)])
    want = orc.matmul_batched(np.ascontiguousarray(A[:, idx]), np.ascontiguousarray(B[:, idx]), nc=2, b_mc=False)
    assert_bits(got[:, idx], want, "many batches")


def test_bmm_paper_size(mcf, orc):
    """The paper's BMM-MCN workload, (16 x 500 x 200) x (16 x 200 x 50), MC x plain,
    binary32, nc = 3, in full."""
    g = np.random.default_rng(1200)
    A = operand(g, (16, 500, 200), 3, np.float32, True)
    B = operand(g, (16, 200, 50), 3, np.float32, False)
    got = to_host(mcf.mc_bmm(to_dev(A), to_dev(B), nc=3, a_mc=True, b_mc=False))
    assert_bits(got, orc.matmul_batched(A, B, nc=3, a_mc=True, b_mc=False), "bmm 16x500x200x50")


@pytest.mark.parametrize("dt", [np.float16, np.float32])
@pytest.mark.parametrize("nc", [2, 3])
@pytest.mark.parametrize("y_full", [True, False])
@pytest.mark.parametrize("ab", [(1.0, 1.0), (0.5, -3.0), (-2.0, 0.25), (1.5, 0.0)])
def test_addmm_parity(mcf, orc, dt, nc, y_full, ab):
    alpha, beta = ab
    M, N, K = 37, 29, 45
    g = np.random.default_rng(1300 + nc)
    A = operand(g, (M, K), nc, dt, True)
    B = operand(g, (K, N), nc, dt, False)
    Y = inputs.split(g.normal(0.0, 0.5, (M, N) if y_full else (N,)), nc, dt)
    got = to_host(mcf.mc_addmm(to_dev(A), to_dev(B), to_dev(Y), nc=nc, alpha=alpha, beta=beta))
    assert_bits(got, orc.addmm(A, B, Y, alpha, beta, nc=nc), f"addmm {dt.__name__} nc={nc} {ab} full={y_full}")


def test_addmm_paper_size_and_kinds(mcf, orc):
    """The paper's AddMM-MCN workload (500 x 200) x (200 x 100) + bias of 100, binary32
    nc = 3, MC x plain as printed, and the same with both operands MC."""
    g = np.random.default_rng(1400)
    A = operand(g, (500, 200), 3, np.float32, True)
    Bm = operand(g, (200, 100), 3, np.float32, True)
    Y = inputs.split(g.normal(0.0, 0.5, (100,)), 3, np.float32)
    for b_mc in (False, True):
        B = Bm if b_mc else Bm[:1]
        got = to_host(mcf.mc_addmm(to_dev(A), to_dev(B), to_dev(Y), nc=3, alpha=0.5, beta=2.0, b_mc=b_mc))
        assert_bits(got, orc.addmm(A, B, Y, 0.5, 2.0, nc=3, b_mc=b_mc), f"addmm paper size b_mc={b_mc}")


def test_matmul_mcn_dispatch(mcf, orc):
    """Matmul-MCN picks Dot, MV, vector-matrix, MM, BMM or 4DMM by operand rank."""
    g = np.random.default_rng(1500)
    nc, dt = 2, np.float32
    x1 = operand(g, (50,), nc, dt, True)
    y1 = operand(g, (50,), nc, dt, False)
    x2 = operand(g, (7, 50), nc, dt, True)
    y2 = operand(g, (50, 9), nc, dt, False)
    x3 = operand(g, (3, 7, 50), nc, dt, True)
    y3 = operand(g, (3, 50, 9), nc, dt, False)
    x4 = operand(g, (2, 1, 7, 50), nc, dt, True)
    y4 = operand(g, (1, 3, 50, 9), nc, dt, False)
    cases = [
        (x1, y1, orc.matmul(x1[:, None, :], y1[:, :, None], nc=nc, b_mc=False)[:, 0, 0]),
        (x2, y1, orc.matmul(x2, y1[:, :, None], nc=nc, b_mc=False)[:, :, 0]),
        (x1, y2, orc.matmul(x1[:, None, :], y2, nc=nc, b_mc=False)[:, 0, :]),
        (x2, y2, orc.matmul(x2, y2, nc=nc, b_mc=False)),
        (x3, y3, orc.matmul_batched(x3, y3, nc=nc, b_mc=False)),
        (x4, y4, orc.matmul_batched(x4, y4, nc=nc, b_mc=False)),
        (x3, y1, orc.matmul_batched(x3, y1[:, None, :, None], nc=nc, b_mc=False)[..., 0]),
    ]
    for i, (x, y, want) in enumerate(cases):
        got = to_host(mcf.matmul_mcn(to_dev(x), to_dev(y), nc=nc, x_mc=True, y_mc=False))
        assert_bits(got, want, f"dispatch case {i}")


def test_argument_errors(mcf):
    import torch

    g = np.random.default_rng(1600)
    A = to_dev(operand(g, (8, 6), 2, np.float16, True))
    B = to_dev(operand(g, (6, 5), 2, np.float16, False))
    Y = to_dev(inputs.split(g.normal(size=(5,)), 2, np.float16))
    with pytest.raises(ValueError):  # 0.1 is not a binary16 value
        mcf.mc_addmm(A, B, Y, nc=2, alpha=0.1)
    with pytest.raises(ValueError):  # bias of the wrong shape
        mcf.mc_addmm(A, B, torch.zeros((2, 4), dtype=torch.float16, device="cuda"), nc=2)
    with pytest.raises(ValueError):  # incompatible batch dimensions
        mcf.mc_matmul_batched(to_dev(operand(g, (2, 8, 6), 2, np.float16, True)),
                              to_dev(operand(g, (3, 6, 5), 2, np.float16, False)), nc=2, b_mc=False)
    # a plane too small for the batch strides is rejected by the C ABI itself
    lib = mcf.lib()
    import ctypes

    st = lib.mc_matmul_batched(0, 2, 1, 2, 8, 5, 6, ctypes.c_void_p(A.data_ptr()), 1, 48, 0, 48,
                               ctypes.c_void_p(B.data_ptr()), 0, 30, 0, 0,
                               ctypes.c_void_p(torch.empty(160, dtype=torch.float16, device="cuda").data_ptr()),
                               None)
    assert st == -3
