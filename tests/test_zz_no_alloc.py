"""GPU check of the allocation-free K-split product (mc_matmul_splitk_noalloc).

Called through the C ABI: its output must equal, bit for bit, mc_matmul_splitk's
with a caller workspace on the same operands and slice count.  Three calls in a row
share the library's static scratch: the first fills most of it (7.4 MB of tree
roots), the next two are smaller, so stale roots from an earlier call are present
while they run; every call is also checked against the oracle's K-split product.
"""
import ctypes

import numpy as np
import pytest

from paper_2207_08867_amd import inputs
from test_gpu_elementwise import assert_bits, to_dev, to_host

pytestmark = pytest.mark.gpu

CODES = {np.float16: 0, np.float32: 1, np.float64: 2}


@pytest.fixture(scope="module")
def mcf():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2207_08867_amd as m

    m.lib()
    return m


def noalloc(mcf, A, B, nc, a_mc, b_mc, S):
    import torch

    tA, tB = to_dev(A), to_dev(B)
    M, K, N = A.shape[1], A.shape[2], B.shape[2]
    out = torch.empty((nc, M, N), dtype=tA.dtype, device=tA.device)
    stream = ctypes.c_void_p(torch.cuda.current_stream(tA.device).cuda_stream)
    st = mcf.lib().mc_matmul_splitk_noalloc(CODES[A.dtype.type], nc, M, N, K, ctypes.c_void_p(tA.data_ptr()),
                                            int(a_mc), ctypes.c_void_p(tB.data_ptr()), int(b_mc), S,
                                            ctypes.c_void_p(out.data_ptr()), stream)
    assert st == 0, mcf.mc_status_str(st)
    return to_host(out), tA, tB


CASES = [
    # (format, nc, M, N, K, a_mc, b_mc, slices): scratch bytes 7 372 800, 16 384, 720
    (np.float32, 3, 32, 64, 30000, True, True, 25600),
    (np.float32, 2, 1, 1, (1 << 20) + 3, True, True, 1 << 18),
    (np.float16, 3, 3, 2, 100003, True, False, 5000),
]


def test_noalloc_matches_workspace_call(mcf, orc):
    for dt, nc, M, N, K, a_mc, b_mc, S in CASES:
        what = f"noalloc {dt.__name__} nc={nc} {M}x{N}x{K} S={S}"
        print(what, flush=True)
        need = mcf.mc_matmul_splitk_workspace(CODES[dt], nc, M, N, K, a_mc, b_mc, S)
        assert 0 < need <= 8 << 20, (what, need)
        A, B = inputs.matmul_normal(M, N, K, nc, dt, seed=M + N + nc)
        A = A if a_mc else A[:1]
        B = B if b_mc else B[:1]
        got, tA, tB = noalloc(mcf, A, B, nc, a_mc, b_mc, S)
        ref = to_host(mcf.mc_matmul_splitk(tA, tB, nc=nc, a_mc=a_mc, b_mc=b_mc, slices=S))
        assert_bits(got, ref, what + " vs mc_matmul_splitk")
        want = orc.matmul_splitk(A, B, nc=nc, a_mc=a_mc, b_mc=b_mc, slices=S)
        assert_bits(got, want, what + " vs oracle")


def test_noalloc_scratch_limit(mcf):
    """Beyond the static scratch the call is refused with MCF_E_SCRATCH."""
    import torch

    # 256 group roots of 3 x 4096 binary32 components: 12.6 MB
    assert mcf.mc_matmul_splitk_workspace(1, 3, 4, 1024, 1 << 16, True, False, 1 << 16) == 256 * 3 * 4096 * 4
    A = torch.zeros((3, 4, 1 << 16), dtype=torch.float32, device="cuda")
    B = torch.zeros((1, 1 << 16, 1024), dtype=torch.float32, device="cuda")
    with pytest.raises(ValueError, match="MCF_E_SCRATCH"):
        mcf.mc_matmul_splitk_noalloc(A, B, nc=3, a_mc=True, b_mc=False, slices=1 << 16)
