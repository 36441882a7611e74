"""The library's binary16 division over every pair of binary16 encodings: mc_div at
nc = 1 (Div-MCN of one-component values: the correctly rounded quotient, a zero
quotient as +0) on all 2^32 pairs (a, b), bitwise against the oracle, NaNs by class.
The pairs are taken in four quarters of the dividends, each in chunks of 1024
dividends x all 65536 divisors (2^26 pairs per launch)."""
import numpy as np
import pytest

from test_gpu_elementwise import assert_bits, to_dev, to_host

pytestmark = pytest.mark.gpu

ALL = np.arange(65536, dtype=np.uint32).astype(np.uint16)
CHUNK = 1024


@pytest.fixture(scope="module")
def mcf():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2207_08867_amd as m

    m.lib()
    return m


@pytest.mark.parametrize("quarter", [0, 1, 2, 3])
def test_div_all_pairs(mcf, orc, quarter):
    import torch

    b = np.tile(ALL, CHUNK).view(np.float16)[None]
    tb = to_dev(b)
    out = torch.empty((1, b.shape[1]), dtype=torch.float16, device="cuda")
    for start in range(quarter * 16384, (quarter + 1) * 16384, CHUNK):
        a = np.repeat(ALL[start:start + CHUNK], 65536).view(np.float16)[None]
        mcf.mc_div(to_dev(a), tb, nc=1, out=out)
        assert_bits(to_host(out), orc.div(a, b, nc=1), f"division, dividends {start}..{start + CHUNK - 1}")
