"""GPU parity of the MC-Linear backward (mc_linear_bwd: dX = dY W, dW = dY^T x, db =
column sums of dY, in MM-MCN order) against the oracle's composition of MM-MCN
products, bitwise: every format, nc 1..3, MC and plain dY, ragged shapes, outputs
requested one at a time; the 4096 x 1024 x 1024 binary16 nc = 3 layer on sampled
outputs (db in full)."""
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


@pytest.mark.parametrize("dt", [np.float16, np.float32, np.float64])
@pytest.mark.parametrize("nc", [1, 2, 3])
@pytest.mark.parametrize("dy_mc", [True, False])
def test_small_parity(mcf, orc, dt, nc, dy_mc):
    T, I, O = 77, 53, 41
    x, W, b = next(inputs.linear_inputs(T, I, O, nc, dt, seed=600 + nc))
    g = np.random.default_rng(610 + nc)
    dY = inputs.split(g.normal(0, 0.5, (T, O)), nc, dt)
    if not dy_mc:
        dY = np.ascontiguousarray(dY[0])
    got = mcf.mc_linear_bwd(to_dev(x), to_dev(W), to_dev(dY), dy_mc=dy_mc)
    want = orc.linear_bwd(x, W, dY, nc=nc, dy_mc=dy_mc)
    for name, a, w in zip(("dX", "dW", "db"), got, want):
        assert_bits(to_host(a), w, f"{name} {dt.__name__} nc={nc} dy_mc={dy_mc}")
    # one output at a time, with a workspace reused from the full call
    for k, flags in enumerate(((True, False, False), (False, True, False), (False, False, True))):
        part = mcf.mc_linear_bwd(to_dev(x), to_dev(W), to_dev(dY), dy_mc=dy_mc, dx=flags[0], dw=flags[1],
                                 db=flags[2])
        assert all((p is None) == (not f) for p, f in zip(part, flags))
        assert_bits(to_host(part[k]), want[k], f"output {k} alone")


def test_degenerate(mcf, orc):
    import torch

    x, W, b = next(inputs.linear_inputs(5, 3, 4, 2, np.float32, seed=620))
    dY = inputs.split(np.random.default_rng(621).normal(0, 1, (5, 4)), 2, np.float32)
    dX, dW, db = mcf.mc_linear_bwd(to_dev(x[:0]), to_dev(W), to_dev(dY[:, :0]))  # batch = 0
    assert dX.shape == (2, 0, 3) and not to_host(dW).any() and not to_host(db).any()
    got = mcf.mc_linear_bwd(to_dev(x[:1]), to_dev(W), to_dev(np.ascontiguousarray(dY[:, :1])))
    for name, a, w in zip(("dX", "dW", "db"), got, orc.linear_bwd(x[:1], W, dY[:, :1], nc=2)):
        assert_bits(to_host(a), w, f"batch 1 {name}")
    with pytest.raises(ValueError):
        mcf.mc_linear_bwd(to_dev(x), to_dev(W), to_dev(dY[:1]))
    with pytest.raises(ValueError):
        ws = torch.empty(8, dtype=torch.uint8, device="cuda")
        mcf.mc_linear_bwd(to_dev(x), to_dev(W), to_dev(dY), workspace=ws)


def test_layer_shape_sampled(mcf, orc):
    """The 4096 x 1024 x 1024 binary16 nc = 3 MC-Linear layer with an MC dY: 1024 sampled
    outputs of dX and of dW bitwise, db in full."""
    T, I, O, nc = 4096, 1024, 1024, 3
    x, W, b = next(inputs.linear_inputs(T, I, O, nc, np.float16, seed=0))
    dY = inputs.split(np.random.default_rng(630).normal(0, 1 / 32, (T, O)), nc, np.float16)
    dX, dW, db = mcf.mc_linear_bwd(to_dev(x), to_dev(W), to_dev(dY))
    g = np.random.default_rng(631)
    r, c = g.integers(0, T, 1024), g.integers(0, I, 1024)
    assert_bits(np.ascontiguousarray(to_host(dX)[:, r, c]), orc.matmul(dY, W, nc=nc, rows=r, cols=c), "dX")
    Yt = np.ascontiguousarray(np.transpose(dY, (0, 2, 1)))
    r, c = g.integers(0, O, 1024), g.integers(0, I, 1024)
    assert_bits(np.ascontiguousarray(to_host(dW)[:, r, c]), orc.matmul(Yt, x[None], nc=nc, b_mc=False, rows=r,
                                                                        cols=c), "dW")
    ones = np.ones((1, T, 1), dtype=np.float16)
    assert_bits(to_host(db), orc.matmul(Yt, ones, nc=nc, b_mc=False)[:, :, 0], "db")
