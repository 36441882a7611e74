"""GPU parity of the linear-regression gradient-descent step (mc_linreg_gd_step)
against the oracle's composition, bitwise, step after step: the paper's shape (n =
10000 samples, d = 2 weights) and a ragged one, both component formats, nc 1..3."""
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


@pytest.mark.parametrize("dt", [np.float16, np.float32])
@pytest.mark.parametrize("nc", [1, 2, 3])
@pytest.mark.parametrize("shape", [(10000, 2), (1000, 3), (7, 1)])
def test_linreg_steps(mcf, orc, dt, nc, shape):
    import torch

    n, d = shape
    X, y_neg, W, _ = inputs.linreg_inputs(n, d, nc, dt, seed=3000 + n + nc)
    Sg, Sl = mcf.mc_matmul_splitk_slices(1, d, n), mcf.mc_matmul_splitk_slices(1, 1, n)
    tX, ty, tW = to_dev(X), to_dev(y_neg), to_dev(W)
    loss = torch.empty(nc, dtype=tW.dtype, device="cuda")
    for step in range(6):
        mcf.mc_linreg_gd_step(tX, ty, tW, 0.05, loss=loss)
        W, want_loss = orc.linreg_gd_step(X, y_neg, W, 0.05, slices_g=Sg, slices_l=Sl)
        assert_bits(to_host(tW), W, f"W after step {step} n={n} d={d} nc={nc} {dt.__name__}")
        assert_bits(to_host(loss), want_loss, f"loss at step {step}")


def test_linreg_argument_errors(mcf):
    import torch

    X = torch.zeros((100, 2), dtype=torch.float32, device="cuda")
    y = torch.zeros(100, dtype=torch.float32, device="cuda")
    W = torch.zeros((2, 2), dtype=torch.float32, device="cuda")
    with pytest.raises(ValueError):  # workspace too small
        mcf.mc_linreg_gd_step(X, y, W, 0.05, workspace=torch.empty(8, dtype=torch.uint8, device="cuda"))
    with pytest.raises(ValueError):  # W overlapping X
        mcf.mc_linreg_gd_step(X, y, X[:2], 0.05)


@pytest.mark.parametrize("dt,nc", [(np.float32, 2), (np.float16, 3)])
def test_linreg_graph_replay(mcf, dt, nc):
    """Steps captured in a HIP graph (the library's launches are capturable: no
    allocation, synchronisation or memset inside a step) replay to the same bits as
    eager steps: 8 steps captured, replayed three times with eager work and a
    synchronisation between replays, W and the loss checked after every replay."""
    import torch

    n, d, k = 10000, 2, 8
    X, y_neg, W0, _ = inputs.linreg_inputs(n, d, nc, dt, seed=4242)
    tX, ty = to_dev(X), to_dev(y_neg)
    code = 0 if dt == np.float16 else 1
    # eager reference: W and loss after k, 2k, 3k steps
    tWe = to_dev(W0)
    le = torch.empty(nc, dtype=tWe.dtype, device="cuda")
    wse = torch.empty(mcf.mc_linreg_workspace(code, nc, n, d), dtype=torch.uint8, device="cuda")
    want = []
    for _ in range(3):
        for _ in range(k):
            mcf.mc_linreg_gd_step(tX, ty, tWe, 0.05, loss=le, workspace=wse)
        want.append((to_host(tWe), to_host(le)))
    # graph: capture k steps on fresh weights, replay
    tWg = to_dev(W0)
    lg = torch.empty(nc, dtype=tWg.dtype, device="cuda")
    wsg = torch.empty_like(wse)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for _ in range(k):
            mcf.mc_linreg_gd_step(tX, ty, tWg, 0.05, loss=lg, workspace=wsg)
    assert_bits(to_host(tWg), W0, "capture alone must not run the steps")
    other = to_dev(np.ones((nc, 1000), dt))
    for r in range(3):
        g.replay()
        torch.cuda.synchronize()
        assert_bits(to_host(tWg), want[r][0], f"W after replay {r}")
        assert_bits(to_host(lg), want[r][1], f"loss after replay {r}")
        mcf.mc_add(other, other, nc=nc)  # eager work between replays
        torch.cuda.synchronize()
