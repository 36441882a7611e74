"""Pins for the oracle's MC-Linear backward (dX = dY W, dW = dY^T x, db = column sums of
dY, each accumulated in MM-MCN order): nc = 1 is the plain sequential float
computation (numpy, one rounding per operation); a plain dY equals an MC dY with zero
low components; the results are within the MM-MCN bound of the exact gradients."""
import numpy as np
import pytest

from paper_2207_08867_amd import inputs

U = {np.float16: 2.0 ** -11, np.float32: 2.0 ** -24}


def _seq(A, B):
    dt = A.dtype.type
    acc = np.outer(A[:, 0], B[0, :]).astype(dt)
    with np.errstate(all="ignore"):
        for k in range(1, A.shape[1]):
            acc = (acc + np.outer(A[:, k], B[k, :]).astype(dt)).astype(dt)
    return acc


@pytest.mark.parametrize("dt", [np.float16, np.float32])
def test_nc1_is_sequential_float(orc, dt):
    g = np.random.default_rng(50)
    T, I, O = 23, 17, 11
    x = g.uniform(-1, 1, (T, I)).astype(dt)
    W = g.uniform(-1, 1, (1, O, I)).astype(dt)
    dY = g.uniform(-1, 1, (1, T, O)).astype(dt)
    dX, dW, db = orc.linear_bwd(x, W, dY, nc=1)
    assert np.array_equal(dX[0], _seq(dY[0], W[0]))
    assert np.array_equal(dW[0], _seq(np.ascontiguousarray(dY[0].T), x))
    acc = dY[0, 0].copy()
    for t in range(1, T):
        acc = (acc + dY[0, t]).astype(dt)
    assert np.array_equal(db[0], acc)


def test_plain_dy(orc):
    """With a plain dY, dW and db equal those of the MC dY with zero low components, and
    dX is the plain x MC product (MM-MCN of ScalingN(W, dY) terms)."""
    g = np.random.default_rng(51)
    x, W, b = next(inputs.linear_inputs(19, 13, 7, 3, np.float32, seed=52))
    dY = g.normal(0, 1, (19, 7)).astype(np.float32)
    dYmc = np.zeros((3, 19, 7), dtype=np.float32)
    dYmc[0] = dY
    dX, dW, db = orc.linear_bwd(x, W, dY, nc=3, dy_mc=False)
    _, dW2, db2 = orc.linear_bwd(x, W, dYmc, nc=3)
    assert np.array_equal(dW.view(np.uint32), dW2.view(np.uint32))
    assert np.array_equal(db.view(np.uint32), db2.view(np.uint32))
    assert np.array_equal(dX.view(np.uint32), orc.matmul(dY[None], W, nc=3, a_mc=False).view(np.uint32))


@pytest.mark.parametrize("nc", [2, 3])
def test_exact_bounds(orc, nc):
    """|dW - dY^T x| <= 4 T u^nc (|dY|^T |x|), |db - sum_t dY| <= 4 T u^nc sum_t |dY|, and
    |dX - dY W| <= 4 O u^nc (|dY| |W|) exactly (binary32, u^nc above the binary32 floor)."""
    T, I, O = 64, 24, 20
    x, W, b = next(inputs.linear_inputs(T, I, O, nc, np.float32, seed=53))
    dY = inputs.split(np.random.default_rng(54).normal(0, 1, (T, O)), nc, np.float32)
    dX, dW, db = orc.linear_bwd(x, W, dY, nc=nc)
    u = U[np.float32] ** nc
    err, absab, _ = orc.matmul_exact_err(dY, W, dX)
    assert np.all(np.abs(err) <= 4 * O * u * absab)
    Yt = np.ascontiguousarray(np.transpose(dY, (0, 2, 1)))
    err, absab, _ = orc.matmul_exact_err(Yt, x[None], dW)
    assert np.all(np.abs(err) <= 4 * T * u * absab)
    err, absab, _ = orc.matmul_exact_err(Yt, np.ones((1, T, 1), np.float32), db[:, :, None])
    assert np.all(np.abs(err) <= 4 * T * u * absab)
