"""MI355X (gfx950) multi-component floating-point (MCF) arithmetic.

Python binding of the C ABI in include/mcf.h (libmcf.so, built in-tree by
``paper_2207_08867_amd.build``).  This module only marshals arguments: it checks
shapes, dtypes and devices of torch tensors, passes their device pointers and the
current HIP stream, and turns status codes into exceptions.  Every arithmetic step
runs in the library's HIP kernels; there is no fallback.

Tensor conventions (component-major):
  * an MC tensor with nc components and logical shape S is a torch tensor of shape
    (nc, *S); a plain tensor has shape S or (1, *S);
  * component dtype torch.float16, torch.float32 or torch.float64; all tensors contiguous and on
    the same GPU.
"""
from __future__ import annotations

import ctypes
import os

__all__ = [
    "mc_add", "mc_mul", "mc_div", "mc_exp", "mc_renorm", "mc_matmul", "mc_matmul_splitk",
    "mc_matmul_splitk_slices", "mc_matmul_splitk_workspace", "mc_matmul_splitk_noalloc", "mc_linear_fwd", "mc_status_str",
    "mc_matmul_batched", "mc_bmm", "mc_addmm", "matmul_mcn", "mc_mul_slow", "mc_square", "mc_matmul_pruned",
    "mc_matmul_exact", "mc_matmul_exact_workspace", "mc_linreg_workspace", "mc_linreg_gd_step",
    "mc_linear_fwd_exact", "mc_linear_bwd", "mc_linear_bwd_workspace", "lib", "LIB_PATH", "MCFError",
]

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libmcf.so")
_lib = None

MCF_F16, MCF_F32, MCF_F64, MCF_F16S = 0, 1, 2, 3


class MCFError(RuntimeError):
    pass


def lib() -> ctypes.CDLL:
    """Load libmcf.so; raises if it has not been built (there is no fallback)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise MCFError(f"{LIB_PATH} is missing: build it with `python -m paper_2207_08867_amd.build` "
                           "(or __graft_entry__.build())")
        L = ctypes.CDLL(LIB_PATH)
        vp, i64, ci = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int
        for name in ("mc_add", "mc_mul", "mc_div"):
            f = getattr(L, name)
            f.restype = ci
            f.argtypes = [ci, ci, i64, vp, ci, vp, ci, vp, vp]
        L.mc_mul_slow.restype = ci
        L.mc_mul_slow.argtypes = [ci, ci, i64, vp, vp, vp, vp]
        L.mc_square.restype = ci
        L.mc_square.argtypes = [ci, ci, i64, vp, vp, vp]
        L.mc_exp.restype = ci
        L.mc_exp.argtypes = [ci, ci, i64, vp, vp, vp]
        L.mc_renorm.restype = ci
        L.mc_renorm.argtypes = [ci, ci, ci, i64, vp, vp, ci, vp]
        L.mc_matmul.restype = ci
        L.mc_matmul.argtypes = [ci, ci, i64, i64, i64, vp, ci, vp, ci, vp, vp]
        L.mc_matmul_splitk.restype = ci
        L.mc_matmul_splitk.argtypes = [ci, ci, i64, i64, i64, vp, ci, vp, ci, i64, vp, i64, vp, vp]
        L.mc_matmul_splitk_noalloc.restype = ci
        L.mc_matmul_splitk_noalloc.argtypes = [ci, ci, i64, i64, i64, vp, ci, vp, ci, i64, vp, vp]
        L.mc_matmul_splitk_slices.restype = i64
        L.mc_matmul_splitk_slices.argtypes = [i64, i64, i64]
        L.mc_matmul_splitk_workspace.restype = i64
        L.mc_matmul_splitk_workspace.argtypes = [ci, ci, i64, i64, i64, ci, ci, i64]
        L.mc_matmul_pruned.restype = ci
        L.mc_matmul_pruned.argtypes = [ci, ci, i64, i64, i64, vp, vp, vp, vp]
        L.mc_matmul_batched.restype = ci
        L.mc_matmul_batched.argtypes = [ci, ci, i64, i64, i64, i64, i64, vp, ci, i64, i64, i64, vp, ci, i64, i64,
                                        i64, vp, vp]
        L.mc_addmm.restype = ci
        L.mc_addmm.argtypes = [ci, ci, i64, i64, i64, vp, ci, vp, ci, vp, i64, ctypes.c_double, ctypes.c_double,
                               vp, vp]
        L.mc_matmul_exact.restype = ci
        L.mc_matmul_exact.argtypes = [ci, ci, i64, i64, i64, vp, ci, vp, ci, ci, vp, i64, vp, vp]
        L.mc_linear_fwd_exact.restype = ci
        L.mc_linear_fwd_exact.argtypes = [ci, ci, i64, i64, i64, vp, vp, vp, vp, i64, vp, vp]
        L.mc_matmul_exact_workspace.restype = i64
        L.mc_matmul_exact_workspace.argtypes = [ci, ci, i64, i64, i64]
        L.mc_linreg_workspace.restype = i64
        L.mc_linreg_workspace.argtypes = [ci, ci, i64, i64]
        L.mc_linreg_gd_step.restype = ci
        L.mc_linreg_gd_step.argtypes = [ci, ci, i64, i64, vp, vp, vp, ctypes.c_double, vp, i64, vp, vp]
        L.mc_linear_bwd.restype = ci
        L.mc_linear_bwd.argtypes = [ci, ci, i64, i64, i64, vp, vp, vp, ci, vp, vp, vp, vp, i64, vp]
        L.mc_linear_bwd_workspace.restype = i64
        L.mc_linear_bwd_workspace.argtypes = [ci, ci, i64, i64, i64]
        L.mc_linear_fwd.restype = ci
        L.mc_linear_fwd.argtypes = [ci, ci, i64, i64, i64, vp, vp, vp, vp, vp]
        L.mc_status_str.restype = ctypes.c_char_p
        L.mc_status_str.argtypes = [ci]
        _lib = L
    return _lib


def mc_status_str(status: int) -> str:
    return lib().mc_status_str(int(status)).decode()


def _check(status: int, what: str):
    if status != 0:
        msg = f"{what}: {mc_status_str(status)}"
        if status in (-1, -2, -3, -4, -5, -7, -8):
            raise ValueError(msg)
        raise MCFError(msg)


def _torch():
    import torch

    return torch


def _code(t, scaled: bool) -> int:
    """Format code of a tensor; scaled=True: binary16 with scaled low components
    (component c stands for 2^(-11 c) times its stored value), float16 tensors only."""
    if scaled:
        if t.dtype != _torch().float16:
            raise TypeError("scaled components need float16 tensors")
        return MCF_F16S
    return _dtype_code(t)


def _dtype_code(t) -> int:
    torch = _torch()
    if t.dtype == torch.float16:
        return MCF_F16
    if t.dtype == torch.float32:
        return MCF_F32
    if t.dtype == torch.float64:
        return MCF_F64
    raise TypeError(f"component dtype must be float16, float32 or float64, got {t.dtype}")


def _dev(t, name):
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _stream(t) -> ctypes.c_void_p:
    torch = _torch()
    return ctypes.c_void_p(torch.cuda.current_stream(t.device).cuda_stream)


def _logical_shape(t, nc, is_mc, name):
    if is_mc:
        if t.dim() < 1 or t.shape[0] != nc:
            raise ValueError(f"{name}: MC operand must have shape (nc={nc}, ...), got {tuple(t.shape)}")
        return tuple(t.shape[1:])
    return tuple(t.shape)


def _binary(fn_name, x, y, nc, x_mc, y_mc, out, scaled=False):
    torch = _torch()
    if x.dtype != y.dtype or x.device != y.device:
        raise ValueError("operands must share dtype and device")
    sx = _logical_shape(x, nc, x_mc, "x")
    sy = _logical_shape(y, nc, y_mc, "y")
    # a plain operand given as (1, *S) is accepted as S
    if not x_mc and len(sx) == len(sy) + 1 and sx[0] == 1:
        sx = sx[1:]
    if not y_mc and len(sy) == len(sx) + 1 and sy[0] == 1:
        sy = sy[1:]
    if sx != sy:
        raise ValueError(f"shape mismatch: {sx} vs {sy}")
    n = 1
    for d in sx:
        n *= d
    if out is None:
        out = torch.empty((nc,) + sx, dtype=x.dtype, device=x.device)
    elif out.shape != (nc,) + sx or out.dtype != x.dtype:
        raise ValueError("out has the wrong shape or dtype")
    st = getattr(lib(), fn_name)(_code(x, scaled), nc, n, _dev(x, "x"), int(bool(x_mc)), _dev(y, "y"),
                                 int(bool(y_mc)), _dev(out, "out"), _stream(x))
    _check(st, fn_name)
    return out


def mc_add(x, y, *, nc: int, x_mc: bool = True, y_mc: bool = True, out=None, scaled: bool = False):
    """Add-MCN for (MC, MC); Grow-ExpN for (MC, T) and (T, MC).  scaled=True: float16
    components with scaled low components (MC, MC only)."""
    return _binary("mc_add", x, y, nc, x_mc, y_mc, out, scaled)


def mc_mul(x, y, *, nc: int, x_mc: bool = True, y_mc: bool = True, out=None, scaled: bool = False):
    """Mult-MCN (fast) for (MC, MC); ScalingN for (MC, T) and (T, MC).  scaled=True:
    float16 components with scaled low components ((MC, T) and (T, MC) only)."""
    return _binary("mc_mul", x, y, nc, x_mc, y_mc, out, scaled)


def mc_div(x, y, *, nc: int, x_mc: bool = True, y_mc: bool = True, out=None):
    """Div-MCN for (MC, MC); DivN for (T, MC); zero-padded divisor for (MC, T)."""
    return _binary("mc_div", x, y, nc, x_mc, y_mc, out)


def mc_mul_slow(x, y, *, nc: int, out=None):
    """Mult-MCN-Slow of two MC operands of the same shape (nc, ...)."""
    torch = _torch()
    if x.dtype != y.dtype or x.device != y.device or x.shape != y.shape or x.shape[0] != nc:
        raise ValueError("x and y must be MC operands (nc, ...) of one shape, dtype and device")
    n = x.numel() // nc
    if out is None:
        out = torch.empty_like(x)
    elif out.shape != x.shape or out.dtype != x.dtype:
        raise ValueError("out has the wrong shape or dtype")
    st = lib().mc_mul_slow(_dtype_code(x), nc, n, _dev(x, "x"), _dev(y, "y"), _dev(out, "out"), _stream(x))
    _check(st, "mc_mul_slow")
    return out


def mc_square(x, *, nc: int, out=None):
    """Square-MCN of an MC operand (nc, ...)."""
    torch = _torch()
    _logical_shape(x, nc, True, "x")
    n = x.numel() // nc
    if out is None:
        out = torch.empty_like(x)
    elif out.shape != x.shape or out.dtype != x.dtype:
        raise ValueError("out has the wrong shape or dtype")
    _check(lib().mc_square(_dtype_code(x), nc, n, _dev(x, "x"), _dev(out, "out"), _stream(x)), "mc_square")
    return out


def mc_exp(x, *, nc: int, out=None):
    """Exp-MCN (every component format; the component exponential is correctly rounded)."""
    torch = _torch()
    s = _logical_shape(x, nc, True, "x")
    n = x.numel() // nc
    if out is None:
        out = torch.empty_like(x)
    elif out.shape != x.shape or out.dtype != x.dtype:
        raise ValueError("out has the wrong shape or dtype")
    del s
    _check(lib().mc_exp(_dtype_code(x), nc, n, _dev(x, "x"), _dev(out, "out"), _stream(x)), "mc_exp")
    return out


def mc_renorm(x, *, nc_out: int | None = None, mode: int = 0, out=None):
    """mode 0: Renormalize; mode 1: Simple-Renorm.  x: (nc_in, ...)."""
    torch = _torch()
    nc_in = x.shape[0]
    nc_out = nc_in if nc_out is None else nc_out
    n = x.numel() // nc_in if nc_in else 0
    if out is None:
        out = torch.empty((nc_out,) + tuple(x.shape[1:]), dtype=x.dtype, device=x.device)
    elif out.shape != (nc_out,) + tuple(x.shape[1:]) or out.dtype != x.dtype:
        raise ValueError("out has the wrong shape or dtype")
    st = lib().mc_renorm(_dtype_code(x), nc_in, nc_out, n, _dev(x, "x"), _dev(out, "out"), int(mode), _stream(x))
    _check(st, "mc_renorm")
    return out


def _mm_operands(A, B, nc, a_mc, b_mc, out):
    torch = _torch()
    if A.dtype != B.dtype or A.device != B.device:
        raise ValueError("operands must share dtype and device")
    A3 = A if A.dim() == 3 else A.reshape((1,) + tuple(A.shape))
    B3 = B if B.dim() == 3 else B.reshape((1,) + tuple(B.shape))
    if A3.shape[0] != (nc if a_mc else 1) or B3.shape[0] != (nc if b_mc else 1):
        raise ValueError("operand plane count does not match nc / kind")
    M, K = A3.shape[1:]
    K2, N = B3.shape[1:]
    if K != K2:
        raise ValueError(f"inner dimensions differ: {K} vs {K2}")
    if out is None:
        out = torch.empty((nc, M, N), dtype=A.dtype, device=A.device)
    elif out.shape != (nc, M, N) or out.dtype != A.dtype:
        raise ValueError("out has the wrong shape or dtype")
    return A3, B3, M, N, K, out


def mc_matmul(A, B, *, nc: int, a_mc: bool = True, b_mc: bool = True, out=None, scaled: bool = False):
    """C = A B in MM-MCN order.  A: (nc|1, M, K), B: (nc|1, K, N) -> (nc, M, N).
    scaled=True: float16 components with scaled low components."""
    A3, B3, M, N, K, out = _mm_operands(A, B, nc, a_mc, b_mc, out)
    st = lib().mc_matmul(_code(A, scaled), nc, M, N, K, _dev(A3, "A"), int(bool(a_mc)), _dev(B3, "B"),
                         int(bool(b_mc)), _dev(out, "out"), _stream(A))
    _check(st, "mc_matmul")
    return out


def mc_matmul_pruned(A, B, *, nc: int, out=None):
    """Pruned MC x MC product: component b of B multiplies the first nc - b components
    of A (the products A^(a) B^(b) with a + b >= nc, of order u^nc, are left out),
    parts combined by Add-MCN.  Same error bound as mc_matmul, about half the work at
    nc = 3; not mc_matmul's bits.  A: (nc, M, K), B: (nc, K, N) -> (nc, M, N)."""
    A3, B3, M, N, K, out = _mm_operands(A, B, nc, True, True, out)
    st = lib().mc_matmul_pruned(_dtype_code(A), nc, M, N, K, _dev(A3, "A"), _dev(B3, "B"), _dev(out, "out"),
                                _stream(A))
    _check(st, "mc_matmul_pruned")
    return out


def mc_matmul_splitk_slices(M: int, N: int, K: int) -> int:
    """Default slice count of the K-split product for this shape."""
    s = lib().mc_matmul_splitk_slices(M, N, K)
    _check(int(s) if s < 0 else 0, "mc_matmul_splitk_slices")
    return int(s)


def mc_matmul_splitk_workspace(dtype_code: int, nc: int, M: int, N: int, K: int, a_mc: bool, b_mc: bool,
                               slices: int) -> int:
    """Workspace bytes the K-split product needs."""
    w = lib().mc_matmul_splitk_workspace(dtype_code, nc, M, N, K, int(bool(a_mc)), int(bool(b_mc)), slices)
    _check(int(w) if w < 0 else 0, "mc_matmul_splitk_workspace")
    return int(w)


def mc_matmul_splitk(A, B, *, nc: int, a_mc: bool = True, b_mc: bool = True, slices: int = 0, out=None,
                     workspace=None):
    """C = A B with the reduction dealt round-robin to `slices` slices (0: the default
    for the shape), each summed in MM-MCN order, the slice sums combined by a
    pairwise Add-MCN tree.  Shapes as for mc_matmul.  `workspace`: an optional
    device byte tensor; one is allocated here when needed and not given."""
    torch = _torch()
    A3, B3, M, N, K, out = _mm_operands(A, B, nc, a_mc, b_mc, out)
    code = _dtype_code(A)
    wb = mc_matmul_splitk_workspace(code, nc, M, N, K, a_mc, b_mc, slices)
    if wb > 0 and workspace is None:
        workspace = torch.empty(wb, dtype=torch.uint8, device=A.device)
    wp = _dev(workspace, "workspace") if workspace is not None else None
    wn = workspace.numel() * workspace.element_size() if workspace is not None else 0
    st = lib().mc_matmul_splitk(code, nc, M, N, K, _dev(A3, "A"), int(bool(a_mc)), _dev(B3, "B"), int(bool(b_mc)),
                                int(slices), wp, wn, _dev(out, "out"), _stream(A))
    _check(st, "mc_matmul_splitk")
    return out


def mc_matmul_splitk_noalloc(A, B, *, nc: int, a_mc: bool = True, b_mc: bool = True, slices: int = 0, out=None):
    """mc_matmul_splitk without a workspace: the library's static per-device scratch
    (8 MiB) holds the partial tree roots, so nothing is allocated when `out` is
    given.  Raises ValueError (MCF_E_SCRATCH) when the call needs more scratch."""
    A3, B3, M, N, K, out = _mm_operands(A, B, nc, a_mc, b_mc, out)
    st = lib().mc_matmul_splitk_noalloc(_dtype_code(A), nc, M, N, K, _dev(A3, "A"), int(bool(a_mc)), _dev(B3, "B"),
                                        int(bool(b_mc)), int(slices), _dev(out, "out"), _stream(A))
    _check(st, "mc_matmul_splitk_noalloc")
    return out


def mc_matmul_exact_workspace(nc: int, M: int, N: int, K: int) -> int:
    """Workspace bytes the exact binary16 product needs."""
    w = lib().mc_matmul_exact_workspace(MCF_F16, nc, M, N, K)
    _check(int(w) if w < 0 else 0, "mc_matmul_exact_workspace")
    return int(w)


def mc_matmul_exact(A, B, *, nc: int, a_mc: bool = True, b_mc: bool = True, b_trans: bool = False, out=None,
                    workspace=None):
    """The exact product of binary16 MC matrices split into nc components by
    successive rounding (int8 matrix cores).  A: (nc|1, M, K); B: (nc|1, K, N), or
    (nc|1, N, K) with b_trans -> (nc, M, N).  `workspace`: an optional device byte
    tensor; one is allocated here when not given."""
    torch = _torch()
    if b_trans:
        Bv = B if B.dim() == 3 else B.reshape((1,) + tuple(B.shape))
        A3, _, M, N, K, out = _mm_operands(A, Bv.transpose(1, 2), nc, a_mc, b_mc, out)
        B3 = Bv
    else:
        A3, B3, M, N, K, out = _mm_operands(A, B, nc, a_mc, b_mc, out)
    wb = mc_matmul_exact_workspace(nc, M, N, K)
    if workspace is None:
        workspace = torch.empty(max(wb, 1), dtype=torch.uint8, device=A.device)
    wn = workspace.numel() * workspace.element_size()
    st = lib().mc_matmul_exact(_dtype_code(A), nc, M, N, K, _dev(A3, "A"), int(bool(a_mc)), _dev(B3, "B"),
                               int(bool(b_mc)), int(bool(b_trans)), _dev(workspace, "workspace"), wn,
                               _dev(out, "out"), _stream(A))
    _check(st, "mc_matmul_exact")
    return out


def mc_linreg_workspace(dtype_code: int, nc: int, n: int, d: int) -> int:
    """Workspace bytes of one linear-regression gradient-descent step."""
    w = lib().mc_linreg_workspace(dtype_code, nc, n, d)
    _check(int(w) if w < 0 else 0, "mc_linreg_workspace")
    return int(w)


def mc_linreg_gd_step(X, y_neg, W, lr: float, *, loss=None, workspace=None):
    """One gradient-descent step of MC-Linear regression with the mean-squared error
    (see include/mcf.h).  X: (n, d) plain; y_neg: (n,) the negated targets; W: (nc, d)
    MC, updated in place; loss: optional (nc,) MC output, the loss before the update.
    `workspace`: an optional device byte tensor; one is allocated here when not given."""
    torch = _torch()
    if X.dim() != 2 or W.dim() != 2 or y_neg.dim() != 1:
        raise ValueError("X must be (n, d), W (nc, d), y_neg (n,)")
    n, d = X.shape
    nc = W.shape[0]
    if W.shape[1] != d or y_neg.shape[0] != n or X.dtype != W.dtype or y_neg.dtype != W.dtype:
        raise ValueError("shape or dtype mismatch")
    if loss is not None and (tuple(loss.shape) != (nc,) or loss.dtype != W.dtype):
        raise ValueError("loss must be (nc,) of W's dtype")
    code = _dtype_code(W)
    if workspace is None:
        workspace = torch.empty(mc_linreg_workspace(code, nc, n, d), dtype=torch.uint8, device=W.device)
    st = lib().mc_linreg_gd_step(code, nc, n, d, _dev(X, "X"), _dev(y_neg, "y_neg"), _dev(W, "W"), float(lr),
                                 _dev(workspace, "workspace"), workspace.numel() * workspace.element_size(),
                                 None if loss is None else _dev(loss, "loss"), _stream(W))
    _check(st, "mc_linreg_gd_step")
    return W


def mc_linear_fwd_exact(x, W, b=None, *, out=None, workspace=None):
    """Exact MC-Linear forward y = x W^T + b for binary16 components (int8 matrix
    cores): the exact value of every output split into nc components by successive
    rounding.  x: (batch, in) plain, W: (nc, out, in), b: (nc, out) or None ->
    y: (nc, batch, out)."""
    torch = _torch()
    nc, O, I = W.shape
    if x.dim() != 2 or x.shape[1] != I:
        raise ValueError("x must be (batch, in)")
    if x.dtype != W.dtype or (b is not None and (b.dtype != W.dtype or tuple(b.shape) != (nc, O))):
        raise ValueError("dtype or bias shape mismatch")
    T = x.shape[0]
    if out is None:
        out = torch.empty((nc, T, O), dtype=W.dtype, device=W.device)
    elif tuple(out.shape) != (nc, T, O) or out.dtype != W.dtype:
        raise ValueError("out has the wrong shape or dtype")
    if workspace is None:
        workspace = torch.empty(max(mc_matmul_exact_workspace(nc, T, O, I), 1), dtype=torch.uint8, device=W.device)
    st = lib().mc_linear_fwd_exact(_dtype_code(W), nc, T, I, O, _dev(x, "x"), _dev(W, "W"),
                                   None if b is None else _dev(b, "b"), _dev(workspace, "workspace"),
                                   workspace.numel() * workspace.element_size(), _dev(out, "out"), _stream(W))
    _check(st, "mc_linear_fwd_exact")
    return out


def mc_linear_fwd(x, W, b=None, *, out=None, scaled: bool = False):
    """MC-Linear forward y = x W^T + b.  x: (batch, in) plain, W: (nc, out, in),
    b: (nc, out) or None -> y: (nc, batch, out).  scaled=True: float16 W, b and y with
    scaled low components (x is a plain float16 tensor)."""
    torch = _torch()
    nc, O, I = W.shape
    if x.dim() != 2 or x.shape[1] != I:
        raise ValueError("x must be (batch, in)")
    if x.dtype != W.dtype or (b is not None and (b.dtype != W.dtype or tuple(b.shape) != (nc, O))):
        raise ValueError("dtype or bias shape mismatch")
    T = x.shape[0]
    if out is None:
        out = torch.empty((nc, T, O), dtype=W.dtype, device=W.device)
    elif out.shape != (nc, T, O) or out.dtype != W.dtype:
        raise ValueError("out has the wrong shape or dtype")
    bp = _dev(b, "b") if b is not None else None
    st = lib().mc_linear_fwd(_code(W, scaled), nc, T, I, O, _dev(x, "x"), _dev(W, "W"), bp, _dev(out, "out"),
                             _stream(W))
    _check(st, "mc_linear_fwd")
    return out


def mc_linear_bwd_workspace(dtype_code: int, nc: int, batch: int, in_: int, out: int) -> int:
    w = lib().mc_linear_bwd_workspace(dtype_code, nc, batch, in_, out)
    _check(int(w) if w < 0 else 0, "mc_linear_bwd_workspace")
    return int(w)


def mc_linear_bwd(x, W, dY, *, dy_mc: bool = True, dx: bool = True, dw: bool = True, db: bool = True,
                  workspace=None):
    """MC-Linear backward: dX = dY W, dW = dY^T x, db = column sums of dY (MM-MCN order).
    x: (batch, in) plain, W: (nc, out, in), dY: (nc, batch, out) or plain (batch, out).
    Returns (dX (nc, batch, in), dW (nc, out, in), db (nc, out)), None for the outputs
    not requested.  `workspace`: optional device byte tensor (allocated here if needed)."""
    torch = _torch()
    nc, O, I = W.shape
    if x.dim() != 2 or x.shape[1] != I:
        raise ValueError("x must be (batch, in)")
    T = x.shape[0]
    if tuple(dY.shape) != ((nc, T, O) if dy_mc else (T, O)):
        raise ValueError(f"dY must be {(nc, T, O) if dy_mc else (T, O)}, got {tuple(dY.shape)}")
    if x.dtype != W.dtype or dY.dtype != W.dtype:
        raise ValueError("dtype mismatch")
    code = _dtype_code(W)
    outs = [torch.empty((nc, T, I), dtype=W.dtype, device=W.device) if dx else None,
            torch.empty((nc, O, I), dtype=W.dtype, device=W.device) if dw else None,
            torch.empty((nc, O), dtype=W.dtype, device=W.device) if db else None]
    if (dw or db) and workspace is None:
        workspace = torch.empty(max(mc_linear_bwd_workspace(code, nc, T, I, O), 1), dtype=torch.uint8,
                                device=W.device)
    wp = _dev(workspace, "workspace") if workspace is not None else None
    wn = workspace.numel() * workspace.element_size() if workspace is not None else 0
    ptr = [(_dev(o, "out") if o is not None else None) for o in outs]
    st = lib().mc_linear_bwd(code, nc, T, I, O, _dev(x, "x"), _dev(W, "W"), _dev(dY, "dY"), int(bool(dy_mc)),
                             ptr[0], ptr[1], ptr[2], wp, wn, _stream(W))
    _check(st, "mc_linear_bwd")
    return tuple(outs)


def _batch_strides(t, name, batch, rows, cols):
    """(plane, s1, s2) of operand t = (planes, *b, rows, cols), len(b) <= 2, broadcast to
    the two batch dimensions `batch` (size-1 or missing dimensions get stride 0)."""
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    b = tuple(t.shape[1:-2])
    t5 = t.reshape((t.shape[0],) + (1,) * (2 - len(b)) + b + (rows, cols)).expand(
        (t.shape[0],) + tuple(batch) + (rows, cols))
    plane = t.stride(0) if t.shape[0] > 1 else t.numel()
    return plane, t5.stride(1) if batch[0] > 1 else 0, t5.stride(2) if batch[1] > 1 else 0


def mc_matmul_batched(A, B, *, nc: int, a_mc: bool = True, b_mc: bool = True, out=None):
    """Batched / broadcast product (BMM-MCN, 4DMM-MCN): A (nc|1, *ba, M, K) times
    B (nc|1, *bb, K, N), up to two batch dimensions each, broadcast as torch.matmul
    broadcasts them -> (nc, *batch, M, N).  Each matrix product is taken as
    mc_matmul takes it."""
    torch = _torch()
    if A.dtype != B.dtype or A.device != B.device:
        raise ValueError("operands must share dtype and device")
    if A.dim() < 3 or B.dim() < 3 or A.dim() > 5 or B.dim() > 5:
        raise ValueError("operands must be (planes, [b1,] [b2,] rows, cols)")
    if A.shape[0] != (nc if a_mc else 1) or B.shape[0] != (nc if b_mc else 1):
        raise ValueError("operand plane count does not match nc / kind")
    M, K = A.shape[-2:]
    K2, N = B.shape[-2:]
    if K != K2:
        raise ValueError(f"inner dimensions differ: {K} vs {K2}")
    try:
        batch = tuple(torch.broadcast_shapes(tuple(A.shape[1:-2]), tuple(B.shape[1:-2])))
    except RuntimeError as e:
        raise ValueError(f"batch dimensions do not broadcast: {e}") from None
    b2 = (1,) * (2 - len(batch)) + batch
    if out is None:
        out = torch.empty((nc,) + batch + (M, N), dtype=A.dtype, device=A.device)
    elif tuple(out.shape) != (nc,) + batch + (M, N) or out.dtype != A.dtype:
        raise ValueError("out has the wrong shape or dtype")
    ap, as1, as2 = _batch_strides(A, "A", b2, M, K)
    bp, bs1, bs2 = _batch_strides(B, "B", b2, K, N)
    st = lib().mc_matmul_batched(_dtype_code(A), nc, b2[0], b2[1], M, N, K, _dev(A, "A"), int(bool(a_mc)), ap, as1,
                                 as2, _dev(B, "B"), int(bool(b_mc)), bp, bs1, bs2, _dev(out, "out"), _stream(A))
    _check(st, "mc_matmul_batched")
    return out


def mc_bmm(A, B, *, nc: int, a_mc: bool = True, b_mc: bool = True, out=None):
    """BMM-MCN: A (nc|1, b, M, K), B (nc|1, b, K, N) -> (nc, b, M, N)."""
    if A.dim() != 4 or B.dim() != 4:
        raise ValueError("BMM operands are (planes, batch, rows, cols)")
    return mc_matmul_batched(A, B, nc=nc, a_mc=a_mc, b_mc=b_mc, out=out)


def mc_addmm(A, B, Y, *, nc: int, alpha: float = 1.0, beta: float = 1.0, a_mc: bool = True, b_mc: bool = False,
             out=None):
    """AddMM-MCN: Add-MCN(ScalingN(A B, alpha), ScalingN(Y, beta)).  A (nc|1, M, K),
    B (nc|1, K, N), Y (nc, M, N) or (nc, N) (added to every row); alpha and beta must
    be values of the component format.  The paper's AddMM multiplies an MC matrix by a
    plain one (the defaults a_mc=True, b_mc=False)."""
    A3, B3, M, N, K, out = _mm_operands(A, B, nc, a_mc, b_mc, out)
    if Y.dtype != A.dtype or Y.device != A.device:
        raise ValueError("Y must share dtype and device with A")
    if tuple(Y.shape) == (nc, M, N):
        y_rows = M
    elif tuple(Y.shape) == (nc, N):
        y_rows = 1
    else:
        raise ValueError(f"Y must be (nc, M, N) or (nc, N), got {tuple(Y.shape)}")
    st = lib().mc_addmm(_dtype_code(A), nc, M, N, K, _dev(A3, "A"), int(bool(a_mc)), _dev(B3, "B"),
                        int(bool(b_mc)), _dev(Y, "Y"), y_rows, float(alpha), float(beta), _dev(out, "out"),
                        _stream(A))
    _check(st, "mc_addmm")
    return out


def matmul_mcn(x, y, *, nc: int, x_mc: bool = True, y_mc: bool = False):
    """Matmul-MCN: dispatch on the logical ranks of x and y (the planes dimension
    excluded) as torch.matmul does -- Dot-MCN (1, 1), MV-MCN (2, 1), vector-matrix
    (1, 2), MM-MCN (2, 2), batched (BMM-MCN / 4DMM-MCN) otherwise, with a 1-D operand
    taken as a column (resp. row) that is dropped from the result."""
    rx = x.dim() - 1
    ry = y.dim() - 1
    if rx < 1 or ry < 1:
        raise ValueError("operands need at least one logical dimension")
    xv = x.unsqueeze(-2) if rx == 1 else x  # (.., 1, K)
    yv = y.unsqueeze(-1) if ry == 1 else y  # (.., K, 1)
    if xv.dim() == 3 and yv.dim() == 3:
        out = mc_matmul(xv, yv, nc=nc, a_mc=x_mc, b_mc=y_mc)
    else:
        out = mc_matmul_batched(xv.contiguous(), yv.contiguous(), nc=nc, a_mc=x_mc, b_mc=y_mc)
    if rx == 1:
        out = out.squeeze(-2)
    if ry == 1:
        out = out.squeeze(-1)
    return out
