"""The C ABI library loads without a GPU, exports every entry point that
include/mcf.h declares, and rejects invalid arguments before any HIP call."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mcf.h")

MCF_OK, MCF_E_NULL, MCF_E_NC, MCF_E_SHAPE, MCF_E_DTYPE, MCF_E_ALIAS, MCF_E_HIP, MCF_E_ARG = 0, -1, -2, -3, -4, -5, -6, -7
MCF_E_SCRATCH = -8


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(mc_\w+)\s*\(", text, flags=re.M)))


@pytest.fixture(scope="module")
def L():
    import paper_2207_08867_amd as m

    return m.lib()


def test_exports_every_declared_symbol(L):
    names = declared_functions()
    assert {"mc_add", "mc_mul", "mc_div", "mc_exp", "mc_renorm", "mc_matmul", "mc_linear_fwd",
            "mc_status_str"} <= set(names)
    for name in names:
        assert hasattr(L, name), name


def test_status_strings(L):
    for code in range(-8, 1):
        s = L.mc_status_str(code).decode()
        assert s.startswith("MCF_")
    assert L.mc_status_str(-99).decode() == "unknown status"


P = ctypes.c_void_p


def test_validation_elementwise(L):
    x = P(0x10000)
    y = P(0x20000)
    o = P(0x30000)
    for f in (L.mc_add, L.mc_mul, L.mc_div):
        assert f(0, 0, 10, x, 1, y, 1, o, None) == MCF_E_NC
        assert f(0, 5, 10, x, 1, y, 1, o, None) == MCF_E_NC
        assert f(4, 3, 10, x, 1, y, 1, o, None) == MCF_E_DTYPE  # 4: no such format
        assert f(0, 3, -1, x, 1, y, 1, o, None) == MCF_E_SHAPE
        assert f(0, 3, 10, x, 0, y, 0, o, None) == MCF_E_ARG
        assert f(0, 3, 10, x, 2, y, 1, o, None) == MCF_E_ARG
        assert f(0, 3, 0, None, 1, None, 1, None, None) == MCF_OK  # empty: no launch
        assert f(0, 3, 10, None, 1, y, 1, o, None) == MCF_E_NULL
        # out overlapping x partially (shifted by one element)
        assert f(1, 3, 10, P(0x10000), 1, y, 1, P(0x10004), None) == MCF_E_ALIAS
        # out overlapping a plain y that is shorter than out
        assert f(1, 3, 10, x, 1, P(0x30000), 0, o, None) == MCF_E_ALIAS
    assert L.mc_exp(4, 3, 10, x, o, None) == MCF_E_DTYPE
    assert L.mc_exp(2, 3, 10, x, P(0x10008), None) == MCF_E_ALIAS
    assert L.mc_exp(1, 3, 10, x, P(0x10004), None) == MCF_E_ALIAS
    assert L.mc_exp(0, 3, 0, None, None, None) == MCF_OK
    assert L.mc_renorm(0, 3, 4, 10, x, o, 0, None) == MCF_E_NC
    assert L.mc_renorm(0, 3, 0, 10, x, o, 0, None) == MCF_E_NC
    assert L.mc_renorm(0, 3, 2, 10, x, o, 2, None) == MCF_E_ARG
    assert L.mc_renorm(0, 3, 2, 10, x, x, 0, None) == MCF_E_ALIAS  # in place only when nc_out == nc_in


def test_validation_matrix(L):
    a, b, c = P(0x100000), P(0x200000), P(0x300000)
    assert L.mc_matmul(0, 3, 4, 4, 4, a, 0, b, 0, c, None) == MCF_E_ARG
    assert L.mc_matmul(0, 9, 4, 4, 4, a, 1, b, 1, c, None) == MCF_E_NC
    assert L.mc_matmul(0, 3, -4, 4, 4, a, 1, b, 1, c, None) == MCF_E_SHAPE
    assert L.mc_matmul(0, 3, 0, 4, 4, a, 1, b, 1, c, None) == MCF_OK
    assert L.mc_matmul(0, 3, 4, 4, 4, a, 1, b, 1, None, None) == MCF_E_NULL
    assert L.mc_matmul(0, 3, 4, 4, 4, a, 1, b, 1, P(0x100000 + 8), None) == MCF_E_ALIAS
    assert L.mc_linear_fwd(0, 3, 4, 4, 4, None, b, None, c, None) == MCF_E_NULL
    assert L.mc_linear_fwd(0, 3, 4, 4, 4, a, b, P(0x300000), c, None) == MCF_E_ALIAS
    assert L.mc_linear_fwd(0, 3, 0, 4, 4, None, None, None, None, None) == MCF_OK
    # operand matrices beyond 2^50 elements are rejected before any byte count is formed
    assert L.mc_matmul(0, 3, 1 << 12, 4, 1 << 39, a, 1, b, 1, c, None) == MCF_E_SHAPE  # M K = 2^51
    assert L.mc_matmul(0, 3, 4, 1 << 30, 1 << 21, a, 1, b, 1, c, None) == MCF_E_SHAPE  # K N = 2^51
    assert L.mc_linear_fwd(0, 3, 4, 1 << 39, 1 << 12, a, b, None, c, None) == MCF_E_SHAPE  # in out = 2^51


def test_validation_splitk(L):
    a, b, c, w = P(0x100000), P(0x200000), P(0x300000), P(0x400000)
    f = L.mc_matmul_splitk
    f.restype = ctypes.c_int
    f.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int64, ctypes.c_int64, ctypes.c_int64, P, ctypes.c_int, P,
                  ctypes.c_int, ctypes.c_int64, P, ctypes.c_int64, P, P]
    ws = L.mc_matmul_splitk_workspace
    ws.restype = ctypes.c_int64
    ws.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int64, ctypes.c_int64, ctypes.c_int64, ctypes.c_int,
                   ctypes.c_int, ctypes.c_int64]
    sl = L.mc_matmul_splitk_slices
    sl.restype = ctypes.c_int64
    sl.argtypes = [ctypes.c_int64] * 3
    # default slice count: about 2^20 lanes, at most K / 64, at most 2^20, at least 1
    assert sl(64, 64, 64) == 1
    assert sl(4096, 1, 4096) == 64
    assert sl(8192, 1, 8192) == 128
    assert sl(1, 1, 1 << 24) == 1 << 18
    assert sl(1, 1, 1 << 30) == 1 << 20
    assert sl(1, 1, 6400) == 100
    assert sl(1, 1, 100) == 1
    assert sl(1024, 1024, 1024) == 1
    assert sl(1, 1, 3) == 1
    assert sl(-1, 1, 3) == MCF_E_SHAPE
    # workspace: none while the slices fit one workgroup (<= 256), else G x planes
    assert ws(1, 3, 4, 4, 4096, 1, 0, 256) == 0
    assert ws(1, 3, 4, 4, 4096, 1, 0, 257) == 2 * 1 * 3 * 16 * 4
    assert ws(0, 2, 4, 4, 4096, 1, 1, 1024) == 4 * 2 * 2 * 16 * 2
    assert ws(1, 3, 4, 4, 4096, 1, 0, (1 << 20) + 1) == MCF_E_ARG
    # G = 274 group roots, and no further level in the workspace
    assert ws(1, 3, 4, 4, 1 << 20, 1, 0, 70000) == 274 * 1 * 3 * 16 * 4
    assert ws(1, 3, 4, 4, 100, 1, 0, 1000) == 0  # capped at K = 100 slices
    assert f(1, 3, 4, 4, 4096, a, 0, b, 0, 16, None, 0, c, None) == MCF_E_ARG
    assert f(1, 7, 4, 4, 4096, a, 1, b, 0, 16, None, 0, c, None) == MCF_E_NC
    assert f(1, 3, 4, 4, -1, a, 1, b, 0, 16, None, 0, c, None) == MCF_E_SHAPE
    assert f(1, 3, 1 << 16, 1 << 16, 4, a, 1, b, 0, 16, None, 0, c, None) == MCF_E_SHAPE  # M N > 2^31
    assert f(1, 3, 1, 1 << 14, 1 << 37, a, 1, b, 0, 16, None, 0, c, None) == MCF_E_SHAPE  # K N = 2^51
    assert f(1, 3, 0, 4, 4096, None, 1, None, 0, 16, None, 0, None, None) == MCF_OK
    assert f(1, 3, 4, 4, 4096, a, 1, b, 0, 1024, None, 0, c, None) == MCF_E_NULL  # workspace needed
    need = ws(1, 3, 4, 4, 4096, 1, 0, 1024)
    assert f(1, 3, 4, 4, 4096, a, 1, b, 0, 1024, w, need - 1, c, None) == MCF_E_ARG
    assert f(1, 3, 4, 4, 4096, a, 1, b, 0, 1024, P(0x300000 + 4), need, c, None) == MCF_E_ALIAS
    assert f(1, 3, 4, 4, 4096, a, 1, b, 0, 1024, a, need, c, None) == MCF_E_ALIAS
    assert f(1, 3, 4, 4, 4096, a, 1, b, 0, 16, None, 0, P(0x100000 + 8), None) == MCF_E_ALIAS


def test_validation_splitk_noalloc(L):
    """The allocation-free K-split call validates like mc_matmul_splitk and refuses
    calls whose tree roots exceed its static 8 MiB scratch, before any HIP call."""
    a, b, c = P(0x100000), P(0x200000), P(0x300000)
    f = L.mc_matmul_splitk_noalloc
    f.restype = ctypes.c_int
    f.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int64, ctypes.c_int64, ctypes.c_int64, P, ctypes.c_int, P,
                  ctypes.c_int, ctypes.c_int64, P, P]
    ws = L.mc_matmul_splitk_workspace
    ws.restype = ctypes.c_int64
    ws.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int64, ctypes.c_int64, ctypes.c_int64, ctypes.c_int,
                   ctypes.c_int, ctypes.c_int64]
    assert f(1, 3, 4, 4, 4096, a, 0, b, 0, 16, c, None) == MCF_E_ARG
    assert f(1, 7, 4, 4, 4096, a, 1, b, 0, 16, c, None) == MCF_E_NC
    assert f(5, 3, 4, 4, 4096, a, 1, b, 0, 16, c, None) == MCF_E_DTYPE
    assert f(1, 3, 4, 4, -1, a, 1, b, 0, 16, c, None) == MCF_E_SHAPE
    assert f(1, 3, 4, 4, 4096, a, 1, b, 0, (1 << 20) + 1, c, None) == MCF_E_ARG
    assert f(1, 3, 0, 4, 4096, None, 1, None, 0, 16, None, None) == MCF_OK
    assert f(1, 3, 4, 4, 4096, None, 1, b, 0, 16, c, None) == MCF_E_NULL
    assert f(1, 3, 4, 4, 4096, a, 1, b, 0, 16, P(0x100000 + 8), None) == MCF_E_ALIAS
    # 4 x 4096 outputs at 2^20 slices: 4096 roots of 3 x 16384 binary32 components
    need = ws(1, 3, 4, 4096, 1 << 20, 1, 0, 1 << 20)
    assert need == 4096 * 3 * 16384 * 4 > 8 << 20
    far = [P(k << 40) for k in (1, 2, 3)]  # operands of several GiB must not overlap
    assert f(1, 3, 4, 4096, 1 << 20, far[0], 1, far[1], 0, 1 << 20, far[2], None) == MCF_E_SCRATCH
    # the largest roots the default slice count asks for fit with room to spare
    assert ws(2, 4, 1, 4095, 1 << 30, 1, 1, 0) == 2 * 16 * 4095 * 8 == 1048320 < 8 << 20
    assert L.mc_status_str(MCF_E_SCRATCH).decode().startswith("MCF_E_SCRATCH")


def test_scaled_format_rejections(L):
    """binary16 with scaled low components (dtype 3) is provided for Add-MCN (MC, MC),
    ScalingN, the product and MC-Linear only; every other call is MCF_E_DTYPE before
    any HIP call."""
    x, y, o = P(0x100000), P(0x200000), P(0x300000)
    for name in ("mc_add", "mc_mul", "mc_div"):
        f = getattr(L, name)
        f.restype = ctypes.c_int
        f.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int64, P, ctypes.c_int, P, ctypes.c_int, P, P]
    assert L.mc_add(3, 3, 10, x, 1, y, 0, o, None) == MCF_E_DTYPE  # Grow-ExpN
    assert L.mc_add(3, 3, 10, x, 0, y, 1, o, None) == MCF_E_DTYPE
    assert L.mc_mul(3, 3, 10, x, 1, y, 1, o, None) == MCF_E_DTYPE  # Mult-MCN
    assert L.mc_div(3, 3, 10, x, 1, y, 1, o, None) == MCF_E_DTYPE
    assert L.mc_add(3, 3, 10, x, 0, y, 0, o, None) == MCF_E_ARG
    assert L.mc_add(3, 5, 10, x, 1, y, 1, o, None) == MCF_E_NC
    assert L.mc_add(3, 3, 0, None, 1, None, 1, None, None) == MCF_OK
    assert L.mc_add(3, 3, 10, x, 1, P(0x100000 + 2), 1, x, None) == MCF_E_ALIAS
    assert L.mc_exp(3, 3, 10, x, o, None) == MCF_E_DTYPE
    assert L.mc_renorm(3, 3, 3, 10, x, o, 0, None) == MCF_E_DTYPE
    assert L.mc_square(3, 3, 10, x, o, None) == MCF_E_DTYPE
    assert L.mc_matmul_pruned(3, 3, 4, 4, 4, x, y, o, None) == MCF_E_DTYPE
    assert L.mc_matmul(4, 3, 4, 4, 4, x, 1, y, 1, o, None) == MCF_E_DTYPE
    assert L.mc_matmul(3, 3, 4, 4, 4, x, 1, y, 1, P(0x100000 + 8), None) == MCF_E_ALIAS


def test_linear_bwd_workspace(L):
    """The backward's workspace: dY^T in nc planes, then the larger of a column of ones
    (db alone) and x with a column of ones appended plus the [dW | db] product (both)."""
    f = L.mc_linear_bwd_workspace
    f.restype = ctypes.c_int64
    f.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int64, ctypes.c_int64, ctypes.c_int64]
    a = lambda n: (n + 255) // 256 * 256
    # binary16 nc = 3, batch 4096, in 1024, out 1024 (the benchmark's layer)
    assert f(0, 3, 4096, 1024, 1024) == a(3 * 1024 * 4096 * 2) + a(4096 * 1025 * 2) + a(3 * 1024 * 1025 * 2)
    # binary32 nc = 2, batch 10, in 0: [x | 1] is the column of ones itself
    assert f(1, 2, 10, 0, 5) == a(2 * 5 * 10 * 4) + a(10 * 4) + a(2 * 5 * 4)
    assert f(0, 3, -1, 4, 4) == MCF_E_SHAPE
    assert f(7, 3, 4, 4, 4) == MCF_E_DTYPE
