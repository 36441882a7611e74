"""CPU oracle for multi-component floating point (MCF) arithmetic.

TEST INFRASTRUCTURE ONLY: imported by tests/, by the smoke check and by the
CPU-baseline leg of bench.py.  The product library never imports, links or calls it,
and it shares no code with the HIP implementation.

The arithmetic lives in ``mcf_oracle.c`` (plain C, one rounding per printed step,
see its header for the number model).  This module only marshals numpy arrays.

Array conventions (component-major, "planar"):
  * an MC array with nc components and logical shape S is an ndarray of shape
    ``(nc, *S)``; a plain tensor has shape ``(1, *S)`` or ``S``;
  * dtype is ``np.float16`` or ``np.float32`` (the component format).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

F16, F32, F64 = 0, 1, 2
_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_SRC = os.path.join(_HERE, "mcf_oracle.c")

OP_ADD, OP_MUL, OP_DIV, OP_EXP, OP_RENORM, OP_SIMPLE_RENORM, OP_SCALING_EXPAND, OP_MUL_SLOW, OP_SQUARE = range(9)

_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (no contraction, no fast-math, OpenMP)."""
    if force or not os.path.exists(_LIB_PATH):
        cmd = ["gcc", "-O2", "-std=gnu11", "-ffp-contract=off", "-fno-fast-math", "-fopenmp",
               "-fPIC", "-shared", "-Wall", "-o", _LIB_PATH + ".tmp", _SRC, "-lquadmath", "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(_LIB_PATH + ".tmp", _LIB_PATH)
    return _LIB_PATH


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
            build()
        L = ctypes.CDLL(_LIB_PATH)
        vp, i64, ci, dbl = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_double
        L.mcf_oracle_check_env.restype = ci
        L.mcf_oracle_max_threads.restype = ci
        for name in ("mcf_oracle_round", "mcf_oracle_fl_exp"):
            getattr(L, name).restype = dbl
            getattr(L, name).argtypes = [ci, dbl]
        for name in ("mcf_oracle_fl_add", "mcf_oracle_fl_sub", "mcf_oracle_fl_mul", "mcf_oracle_fl_div"):
            getattr(L, name).restype = dbl
            getattr(L, name).argtypes = [ci, dbl, dbl]
        L.mcf_oracle_fl_fma.restype = dbl
        L.mcf_oracle_fl_fma.argtypes = [ci, dbl, dbl, dbl]
        L.mcf_oracle_f16_decode.restype = dbl
        L.mcf_oracle_f16_decode.argtypes = [ctypes.c_uint16]
        L.mcf_oracle_f16_encode.restype = ctypes.c_uint16
        L.mcf_oracle_f16_encode.argtypes = [dbl]
        L.mcf_oracle_binop_array.restype = None
        L.mcf_oracle_binop_array.argtypes = [ci, ci, i64, vp, vp, vp]
        L.mcf_oracle_exp32_near_ties.restype = i64
        L.mcf_oracle_exp32_near_ties.argtypes = [dbl, vp, i64]
        L.mcf_oracle_eft_array.restype = None
        L.mcf_oracle_eft_array.argtypes = [ci, ci, i64, vp, vp, vp, vp]
        L.mcf_oracle_elementwise.restype = ci
        L.mcf_oracle_elementwise.argtypes = [ci, ci, ci, ci, i64, vp, ci, vp, ci, vp]
        L.mcf_oracle_matmul.restype = ci
        L.mcf_oracle_matmul.argtypes = [ci, ci, i64, i64, i64, vp, ci, vp, ci, vp, vp, i64, vp]
        L.mcf_oracle_matmul_pruned.restype = ci
        L.mcf_oracle_matmul_pruned.argtypes = [ci, ci, i64, i64, i64, vp, vp, vp, vp, i64, vp]
        L.mcf_oracle_matmul_splitk.restype = ci
        L.mcf_oracle_matmul_splitk.argtypes = [ci, ci, i64, i64, i64, vp, ci, vp, ci, i64, vp, vp, i64, vp]
        L.mcf_oracle_linear.restype = ci
        L.mcf_oracle_linear.argtypes = [ci, ci, i64, i64, i64, vp, vp, vp, vp, vp, i64, vp]
        L.mcf_oracle_matmul_exact_err.restype = ci
        L.mcf_oracle_matmul_exact_err.argtypes = [ci, ci, i64, i64, i64, vp, ci, vp, ci, vp, ci,
                                                  vp, vp, i64, vp, vp, vp, vp]
        L.mcf_oracle_scaled_elementwise.restype = ci
        L.mcf_oracle_scaled_elementwise.argtypes = [ci, ci, i64, vp, ci, vp, ci, vp]
        L.mcf_oracle_scaled_matmul.restype = ci
        L.mcf_oracle_scaled_matmul.argtypes = [ci, i64, i64, i64, vp, ci, vp, ci, vp, vp, i64, vp]
        L.mcf_oracle_scaled_linear.restype = ci
        L.mcf_oracle_scaled_linear.argtypes = [ci, i64, i64, i64, vp, vp, vp, vp, vp, i64, vp]
        L.mcf_oracle_exp64_first.restype = None
        L.mcf_oracle_exp64_first.argtypes = [i64, vp, vp, vp]
        L.mcf_oracle_exp_mcn_given.restype = ci
        L.mcf_oracle_exp_mcn_given.argtypes = [ci, ci, i64, vp, vp]
        L.mcf_oracle_exp64_near_midpoints.restype = i64
        L.mcf_oracle_exp64_near_midpoints.argtypes = [dbl, dbl, ctypes.c_uint64, i64, dbl, vp, i64]
        L.mcf_oracle_exact_diff.restype = None
        L.mcf_oracle_exact_diff.argtypes = [ci, i64, vp, ci, vp, ci, vp]
        if L.mcf_oracle_check_env() != 0:
            raise RuntimeError("oracle: SSE flush-to-zero or denormals-are-zero is set")
        _lib = L
    return _lib


def fmt_of(dtype) -> int:
    dt = np.dtype(dtype)
    if dt == np.float16:
        return F16
    if dt == np.float32:
        return F32
    if dt == np.float64:
        return F64
    raise TypeError(f"component dtype must be float16, float32 or float64, got {dt}")


def _ptr(a: np.ndarray | None):
    return None if a is None else ctypes.c_void_p(a.ctypes.data)


def _planar(a: np.ndarray, dtype) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=dtype)


def threads() -> int:
    return int(lib().mcf_oracle_max_threads())


# ---------------------------------------------------------------------------------
# scalar primitives on float64 arrays (values exactly representable in the format)
# ---------------------------------------------------------------------------------

def _binop(fmt: int, op: int, a, b=None) -> np.ndarray:
    a = np.ascontiguousarray(a, dtype=np.float64).ravel()
    b = a if b is None else np.ascontiguousarray(b, dtype=np.float64).ravel()
    out = np.empty_like(a)
    lib().mcf_oracle_binop_array(fmt, op, a.size, _ptr(a), _ptr(b), _ptr(out))
    return out


def fl_round(fmt, x):
    """fl(x): round float64 values to the component format (returned as float64)."""
    return _binop(fmt, 6, x)


def fl_add(fmt, a, b):
    return _binop(fmt, 0, a, b)


def fl_sub(fmt, a, b):
    return _binop(fmt, 1, a, b)


def fl_mul(fmt, a, b):
    return _binop(fmt, 2, a, b)


def fl_div(fmt, a, b):
    return _binop(fmt, 3, a, b)


def two_prod_err(fmt, a, b):
    """fma(a, b, -fl(a*b)) rounded once."""
    return _binop(fmt, 4, a, b)


def fl_exp(fmt, a):
    """Correctly rounded component exponential."""
    return _binop(fmt, 5, a)


def exp32_near_ties(rel_margin: float, max_out: int = 4096):
    """binary32 inputs x (as uint32 bit patterns) whose long double e^x lies within
    rel_margin (relative) of a binary32 rounding boundary; scans every input with
    2^-30 <= |x| <= 105.  Returns (count, patterns[:min(count, max_out)])."""
    out = np.zeros(max_out, dtype=np.uint32)
    n = int(lib().mcf_oracle_exp32_near_ties(float(rel_margin), _ptr(out), max_out))
    return n, out[:min(n, max_out)]


def two_sum(fmt, a, b):
    a = np.ascontiguousarray(a, dtype=np.float64).ravel()
    b = np.ascontiguousarray(b, dtype=np.float64).ravel()
    s, e = np.empty_like(a), np.empty_like(a)
    lib().mcf_oracle_eft_array(fmt, 0, a.size, _ptr(a), _ptr(b), _ptr(s), _ptr(e))
    return s, e


def two_prod(fmt, a, b):
    a = np.ascontiguousarray(a, dtype=np.float64).ravel()
    b = np.ascontiguousarray(b, dtype=np.float64).ravel()
    s, e = np.empty_like(a), np.empty_like(a)
    lib().mcf_oracle_eft_array(fmt, 1, a.size, _ptr(a), _ptr(b), _ptr(s), _ptr(e))
    return s, e


# ---------------------------------------------------------------------------------
# elementwise MC operations on planar arrays
# ---------------------------------------------------------------------------------

def _as_operand(a, nc, is_mc, dtype):
    a = _planar(a, dtype)
    planes = nc if is_mc else 1
    if a.shape[0] != planes:
        a = a.reshape((1,) + a.shape) if not is_mc else a
    if a.shape[0] != planes:
        raise ValueError(f"operand has {a.shape[0]} planes, expected {planes}")
    return a


def elementwise(op: int, x, y=None, *, nc: int, x_mc=True, y_mc=True, nc_out=None, dtype=None):
    dtype = np.dtype(dtype or np.asarray(x).dtype)
    fmt = fmt_of(dtype)
    x = _as_operand(x, nc, x_mc, dtype)
    shape = x.shape[1:]
    n = int(np.prod(shape)) if shape else 1
    if y is not None:
        y = _as_operand(y, nc, y_mc, dtype)
        if y.shape[1:] != shape:
            raise ValueError("shape mismatch")
    if op in (OP_RENORM, OP_SIMPLE_RENORM):
        planes_out = nc_out
    elif op == OP_SCALING_EXPAND:
        planes_out = nc + 1
    else:
        planes_out = nc
    out = np.empty((planes_out,) + shape, dtype=dtype)
    rc = lib().mcf_oracle_elementwise(fmt, op, nc, nc_out or nc, n, _ptr(x), int(bool(x_mc)), _ptr(y),
                                      int(bool(y_mc)), _ptr(out))
    if rc != 0:
        raise ValueError("oracle: bad arguments")
    return out


def add(x, y, *, nc, x_mc=True, y_mc=True):
    """Add-MCN (MC,MC) or Grow-ExpN (MC,T)/(T,MC)."""
    return elementwise(OP_ADD, x, y, nc=nc, x_mc=x_mc, y_mc=y_mc)


def mul(x, y, *, nc, x_mc=True, y_mc=True):
    """Mult-MCN (MC,MC) or ScalingN (MC,T)/(T,MC)."""
    return elementwise(OP_MUL, x, y, nc=nc, x_mc=x_mc, y_mc=y_mc)


def div(x, y, *, nc, x_mc=True, y_mc=True):
    """Div-MCN (MC,MC), DivN (T,MC), Div-MCN with a zero-padded divisor (MC,T)."""
    return elementwise(OP_DIV, x, y, nc=nc, x_mc=x_mc, y_mc=y_mc)


def exp(x, *, nc):
    """Exp-MCN (binary64 components: component exponentials from fl_exp64)."""
    if np.dtype(np.asarray(x).dtype) == np.float64:
        x = _planar(x, np.float64)
        n = x.shape[-1]
        E = np.ascontiguousarray(fl_exp64(x.reshape(nc, n)))
        out = np.empty((nc, n), dtype=np.float64)
        if lib().mcf_oracle_exp_mcn_given(F64, nc, n, _ptr(E), _ptr(out)) != 0:
            raise ValueError("oracle: bad arguments")
        return out
    return elementwise(OP_EXP, x, nc=nc)


def _exp64_decimal(x: float) -> float:
    """e^x correctly rounded to binary64 from an 80-digit decimal evaluation (decimal's
    exp is correctly rounded to the context precision; the conversion of its decimal
    string to a binary64 number is correctly rounded too).  Raises if the decimal
    value lies within 10^-70 (relative) of a binary64 rounding boundary, where the two
    roundings could disagree."""
    import decimal

    with decimal.localcontext() as ctx:
        ctx.prec = 80
        ctx.Emin, ctx.Emax = -999999, 999999
        v = decimal.Decimal(float(x)).exp()
        r = float(v)
        if r != 0.0 and np.isfinite(r):
            for nb in (np.nextafter(r, np.inf), np.nextafter(r, -np.inf)):
                if np.isfinite(nb):
                    mid = (decimal.Decimal(r) + decimal.Decimal(float(nb))) / 2
                    if abs(v - mid) <= abs(v) * decimal.Decimal("1e-70"):
                        raise ArithmeticError(f"exp({x!r}) too close to a rounding boundary")
    return r


def fl_exp64(x) -> np.ndarray:
    """Correctly rounded binary64 e^x, elementwise: binary128 evaluation with a 2^-100
    margin test (C), the undecided arguments by 80-digit decimal arithmetic."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    flat = x.reshape(-1)
    out = np.empty_like(flat)
    unsure = np.zeros(flat.size, dtype=np.int32)
    lib().mcf_oracle_exp64_first(flat.size, _ptr(flat), _ptr(out), _ptr(unsure))
    for i in np.nonzero(unsure)[0]:
        out[i] = _exp64_decimal(flat[i])
    return out.reshape(x.shape)


def exp64_near_midpoints(lo: float, hi: float, seed: int, tries: int, rel: float, max_out: int = 4096):
    """Random binary64 x in [lo, hi] whose e^x lies within rel (relative) of a binary64
    rounding boundary (test inputs that drive a correctly rounded exponential's slow
    path).  Returns the inputs found (at most max_out)."""
    out = np.zeros(max_out, dtype=np.float64)
    n = int(lib().mcf_oracle_exp64_near_midpoints(float(lo), float(hi), int(seed), int(tries), float(rel),
                                                  _ptr(out), max_out))
    return out[:min(n, max_out)]


def renorm(x, *, nc, nc_out=None, mode=0):
    """mode 0: Renormalize; mode 1: Simple-Renorm."""
    return elementwise(OP_RENORM if mode == 0 else OP_SIMPLE_RENORM, x, nc=nc, nc_out=nc_out or nc)


def mul_slow(x, y, *, nc):
    """Mult-MCN-Slow (MC,MC)."""
    return elementwise(OP_MUL_SLOW, x, y, nc=nc)


def square(x, *, nc):
    """Square-MCN (first step read as fl(x_0 x_0))."""
    return elementwise(OP_SQUARE, x, nc=nc)


def scaling_expand(x, v, *, nc):
    """ScalingN with expand: nc+1 output components."""
    return elementwise(OP_SCALING_EXPAND, x, v, nc=nc, x_mc=True, y_mc=False)


# ---------------------------------------------------------------------------------
# matrix products
# ---------------------------------------------------------------------------------

def _positions(M, N, rows, cols):
    if rows is None:
        return None, None, M * N
    rows = np.ascontiguousarray(rows, dtype=np.int64).ravel()
    cols = np.ascontiguousarray(cols, dtype=np.int64).ravel()
    if rows.shape != cols.shape:
        raise ValueError("rows/cols mismatch")
    if rows.size and (rows.min() < 0 or rows.max() >= M or cols.min() < 0 or cols.max() >= N):
        raise ValueError("position out of range")
    return rows, cols, rows.size


def matmul(A, B, *, nc, a_mc=True, b_mc=True, rows=None, cols=None):
    """C = A x B (MM-MCN order; MC x MC by linearity over B's components).

    A: (nc|1, M, K), B: (nc|1, K, N).  Returns (nc, M, N), or (nc, count) at the
    given positions.
    """
    dtype = np.dtype(A.dtype)
    fmt = fmt_of(dtype)
    A = _planar(A, dtype)
    B = _planar(B, dtype)
    if A.ndim == 2:
        A = A[None]
    if B.ndim == 2:
        B = B[None]
    M, K = A.shape[1:]
    K2, N = B.shape[1:]
    if K2 != K or A.shape[0] != (nc if a_mc else 1) or B.shape[0] != (nc if b_mc else 1):
        raise ValueError("matmul: shape mismatch")
    r, c, count = _positions(M, N, rows, cols)
    out = np.empty((nc, count), dtype=dtype)
    rc = lib().mcf_oracle_matmul(fmt, nc, M, N, K, _ptr(A), int(a_mc), _ptr(B), int(b_mc), _ptr(r), _ptr(c),
                                 count, _ptr(out))
    if rc != 0:
        raise ValueError("oracle: bad arguments")
    return out.reshape(nc, M, N) if rows is None else out


def matmul_pruned(A, B, *, nc, rows=None, cols=None):
    """Pruned MC x MC product: C = MM_nc(A, B^(0)) (+) MM_{nc-1}(A[:nc-1], B^(1)) (+) ...
    (+) MM_1(A[:1], B^(nc-1)), each part in MM-MCN order with the stated number of
    components, zero-padded to nc, combined left to right by Add-MCN.
    A: (nc, M, K), B: (nc, K, N).  Returns (nc, M, N), or (nc, count) at positions."""
    dtype = np.dtype(A.dtype)
    fmt = fmt_of(dtype)
    A = _planar(A, dtype)
    B = _planar(B, dtype)
    M, K = A.shape[1:]
    K2, N = B.shape[1:]
    if K2 != K or A.shape[0] != nc or B.shape[0] != nc:
        raise ValueError("matmul_pruned: shape mismatch")
    r, c, count = _positions(M, N, rows, cols)
    out = np.empty((nc, count), dtype=dtype)
    rc = lib().mcf_oracle_matmul_pruned(fmt, nc, M, N, K, _ptr(A), _ptr(B), _ptr(r), _ptr(c), count, _ptr(out))
    if rc != 0:
        raise ValueError("oracle: bad arguments")
    return out.reshape(nc, M, N) if rows is None else out


def matmul_splitk(A, B, *, nc, slices, a_mc=True, b_mc=True, rows=None, cols=None):
    """C = A x B with the reduction dealt round-robin to min(slices, K) slices, each
    summed in MM-MCN order, then combined by a pairwise Add-MCN tree (MC x MC: one
    such product per component of B, combined left to right).  slices = 1 is
    ``matmul``.  Shapes and return value as for ``matmul``."""
    dtype = np.dtype(A.dtype)
    fmt = fmt_of(dtype)
    A = _planar(A, dtype)
    B = _planar(B, dtype)
    if A.ndim == 2:
        A = A[None]
    if B.ndim == 2:
        B = B[None]
    M, K = A.shape[1:]
    K2, N = B.shape[1:]
    if K2 != K or A.shape[0] != (nc if a_mc else 1) or B.shape[0] != (nc if b_mc else 1) or slices < 1:
        raise ValueError("matmul_splitk: bad arguments")
    r, c, count = _positions(M, N, rows, cols)
    out = np.empty((nc, count), dtype=dtype)
    rc = lib().mcf_oracle_matmul_splitk(fmt, nc, M, N, K, _ptr(A), int(a_mc), _ptr(B), int(b_mc), int(slices),
                                        _ptr(r), _ptr(c), count, _ptr(out))
    if rc != 0:
        raise ValueError("oracle: bad arguments")
    return out.reshape(nc, M, N) if rows is None else out


def matmul_batched(A, B, *, nc, a_mc=True, b_mc=True):
    """BMM-MCN / 4DMM-MCN (Appendix A.2.2): A (nc|1, *ba, M, K) and B (nc|1, *bb, K, N)
    with batch dimensions broadcast as torch.matmul broadcasts them; every batch's
    matrices are multiplied by ``matmul``.  Returns (nc, *batch, M, N)."""
    dtype = np.dtype(A.dtype)
    A = _planar(A, dtype)
    B = _planar(B, dtype)
    M, K = A.shape[-2:]
    N = B.shape[-1]
    batch = np.broadcast_shapes(A.shape[1:-2], B.shape[1:-2])
    # missing batch dimensions go in front of the operand's own, after its planes
    # axis (numpy would align the planes axis with a batch axis)
    A = A.reshape((A.shape[0],) + (1,) * (len(batch) - (A.ndim - 3)) + A.shape[1:])
    B = B.reshape((B.shape[0],) + (1,) * (len(batch) - (B.ndim - 3)) + B.shape[1:])
    Ab = np.broadcast_to(A, (A.shape[0],) + batch + (M, K))
    Bb = np.broadcast_to(B, (B.shape[0],) + batch + (K, N))
    out = np.empty((nc,) + batch + (M, N), dtype=dtype)
    for idx in np.ndindex(*batch):
        sl = (slice(None),) + idx
        out[sl] = matmul(np.ascontiguousarray(Ab[sl]), np.ascontiguousarray(Bb[sl]), nc=nc, a_mc=a_mc, b_mc=b_mc)
    return out


def addmm(A, B, Y, alpha, beta, *, nc, a_mc=True, b_mc=False):
    """AddMM-MCN (Appendix A.2.2), step by step: h = ScalingN(MM-MCN(A, B), alpha);
    bias = ScalingN(Y, beta); return Add-MCN(h, bias).  Y: (nc, M, N) or (nc, N) (one
    row for all); alpha, beta: values of the component format."""
    dtype = np.dtype(A.dtype)
    P = matmul(A, B, nc=nc, a_mc=a_mc, b_mc=b_mc)
    M, N = P.shape[1:]
    Y = _planar(Y, dtype)
    if Y.ndim == 2:  # one row for all: (nc, N) -> (nc, 1, N) before broadcasting
        Y = Y[:, None, :]
    Y = np.broadcast_to(Y, (nc, M, N))
    a = np.full((M, N), alpha, dtype=dtype)
    b = np.full((M, N), beta, dtype=dtype)
    if a.flat[0] != alpha or b.flat[0] != beta:
        raise ValueError("addmm: alpha and beta must be values of the component format")
    h = mul(P, a[None], nc=nc, x_mc=True, y_mc=False)
    bias = mul(np.ascontiguousarray(Y), b[None], nc=nc, x_mc=True, y_mc=False)
    return add(h, bias, nc=nc)


def linear(X, W, bias=None, *, nc, rows=None, cols=None):
    """MC-Linear forward: X plain (T, I), W (nc, O, I), bias (nc, O) or None."""
    dtype = np.dtype(W.dtype)
    fmt = fmt_of(dtype)
    X = _planar(X, dtype)
    W = _planar(W, dtype)
    T, I = X.shape[-2:]
    O = W.shape[1]
    if W.shape != (nc, O, I):
        raise ValueError("linear: shape mismatch")
    if bias is not None:
        bias = _planar(bias, dtype)
        if bias.shape != (nc, O):
            raise ValueError("linear: bias shape mismatch")
    r, c, count = _positions(T, O, rows, cols)
    out = np.empty((nc, count), dtype=dtype)
    rc = lib().mcf_oracle_linear(fmt, nc, T, I, O, _ptr(X), _ptr(W), _ptr(bias), _ptr(r), _ptr(c), count,
                                 _ptr(out))
    if rc != 0:
        raise ValueError("oracle: bad arguments")
    return out.reshape(nc, T, O) if rows is None else out


def linear_bwd(x, W, dY, *, nc, dy_mc=True):
    """MC-Linear backward from the output gradient dY, as the oracle's MM-MCN products:
    dX = dY W; dW = dY^T x and db = dY^T 1 with dY^T carried in nc components (+0 low
    components when dY is plain).  x: (T, I) plain; W: (nc, O, I); dY: (nc, T, O) or
    plain (T, O).  Returns (dX (nc, T, I), dW (nc, O, I), db (nc, O))."""
    dtype = np.dtype(W.dtype)
    x = _planar(x, dtype)
    W = _planar(W, dtype)
    Y = _planar(dY, dtype)
    if not dy_mc:
        Y = Y.reshape((1,) + Y.shape[-2:])
    T, I = x.shape
    O = W.shape[1]
    dX = matmul(Y, W, nc=nc, a_mc=dy_mc, b_mc=True)
    Yt = np.zeros((nc, O, T), dtype=dtype)
    Yt[: Y.shape[0]] = np.transpose(Y, (0, 2, 1))
    dW = matmul(Yt, x[None], nc=nc, a_mc=True, b_mc=False)
    db = matmul(Yt, np.ones((1, T, 1), dtype=dtype), nc=nc, a_mc=True, b_mc=False)[:, :, 0]
    return dX, dW, np.ascontiguousarray(db)


def linreg_gd_step(X, y_neg, W, lr, *, slices_g, slices_l):
    """One gradient-descent step of MC-Linear regression with the mean-squared error
    (the precision experiment of Section 2.4), written as the composition of this
    module's pinned operations.  The paper does not print the optimizer step; it keeps
    the gradient of an MC value as the plain gradient of its leading component (Section
    2.1).  The reading taken here:
        yhat = MC-Linear(X, W)                      (linear, MM-MCN order)
        r    = Grow-ExpN(yhat, -y)                  (add, MC + plain)
        G    = r^T X,  RR = r . r                   (matmul_splitk, slices_g / slices_l)
        g    = ScalingN(G, fl(2/n)); grad = g_0     (mul, MC x plain; leading component)
        W'   = Grow-ExpN(W, fl(-lr * grad))         (fl_mul, then add)
        loss = ScalingN(RR, fl(1/n))                (the loss at W, before the update)
    fl(2/n), fl(1/n): the binary64 quotient rounded to the component format; fl(-lr):
    the binary64 value -lr rounded to it.

    X: (n, d) plain; y_neg: (n,) plain (-y); W: (nc, d) MC.  Returns (W', loss (nc,)).
    """
    dtype = np.dtype(W.dtype)
    fmt = fmt_of(dtype)
    X = _planar(X, dtype)
    y_neg = _planar(y_neg, dtype)
    W = _planar(W, dtype)
    nc, d = W.shape
    n = X.shape[0]
    yhat = linear(X, W.reshape(nc, 1, d), nc=nc)                  # (nc, n, 1)
    r = add(yhat.reshape(nc, n), y_neg.reshape(1, n), nc=nc, y_mc=False)  # (nc, n)
    G = matmul_splitk(r.reshape(nc, 1, n), X, nc=nc, slices=slices_g, b_mc=False).reshape(nc, d)
    RR = matmul_splitk(r.reshape(nc, 1, n), r.reshape(nc, n, 1), nc=nc, slices=slices_l).reshape(nc, 1)
    s2n = fl_round(fmt, np.array([2.0 / n]))[0]
    s1n = fl_round(fmt, np.array([1.0 / n]))[0]
    neg_lr = fl_round(fmt, np.array([-float(lr)]))[0]
    g = mul(G, np.full((1, d), s2n, dtype=dtype), nc=nc, y_mc=False)
    step = fl_mul(fmt, np.full(d, neg_lr), g[0].astype(np.float64)).astype(dtype).reshape(1, d)
    W_new = add(W, step, nc=nc, y_mc=False)
    loss = mul(RR, np.full((1, 1), s1n, dtype=dtype), nc=nc, y_mc=False).reshape(nc)
    return W_new, loss


def matmul_exact_err(A, B, C, *, bias=None, rows=None, cols=None):
    """Exact error of a computed product C (nc, M, N) -- or (nc, count) at positions --
    against the exact product of the MC inputs A (planes, M, K), B (planes, K, N),
    plus an optional bias (planes, N).

    Returns (err, absab, exact) as float64 arrays: err = sum(C) - exact (computed
    exactly, then rounded), absab = sum_k |A^_ik||B^_kj| (+|bias^_j|).
    """
    dtype = np.dtype(A.dtype)
    fmt = fmt_of(dtype)
    A = _planar(A, dtype)
    B = _planar(B, dtype)
    if A.ndim == 2:
        A = A[None]
    if B.ndim == 2:
        B = B[None]
    M, K = A.shape[1:]
    N = B.shape[2]
    nc = C.shape[0]
    r, c, count = _positions(M, N, rows, cols)
    Cf = _planar(C, dtype).reshape(nc, count)
    if bias is not None:
        bias = _planar(bias, dtype)
        if bias.ndim == 1:
            bias = bias[None]
    err = np.empty(count)
    absab = np.empty(count)
    exact = np.empty(count)
    lib().mcf_oracle_matmul_exact_err(fmt, nc, M, N, K, _ptr(A), A.shape[0], _ptr(B), B.shape[0], _ptr(bias),
                                      0 if bias is None else bias.shape[0], _ptr(r), _ptr(c), count, _ptr(Cf),
                                      _ptr(err), _ptr(absab), _ptr(exact))
    return err, absab, exact


def exact_diff(x, y=None):
    """Exact (x - y) per element, rounded to double; x, y planar with any plane count."""
    dtype = np.dtype(x.dtype)
    fmt = fmt_of(dtype)
    x = _planar(x, dtype)
    n = int(np.prod(x.shape[1:]))
    if y is not None:
        y = _planar(y, dtype)
    out = np.empty(n)
    lib().mcf_oracle_exact_diff(fmt, n, _ptr(x), x.shape[0], _ptr(y), 0 if y is None else y.shape[0], _ptr(out))
    return out.reshape(x.shape[1:])


# ---------------------------------------------------------------------------------
# binary16 with scaled low components (reading SC1): component c of a stored value is
# a binary16 number standing for 2^(-11 c) times itself
# ---------------------------------------------------------------------------------

SCALE_SHIFT = 11


def unscale(x) -> np.ndarray:
    """float64 values of the components of a scaled binary16 MC array (nc, ...):
    component c times 2^(-11 c) (exact)."""
    x = np.asarray(x, dtype=np.float16).astype(np.float64)
    sh = np.ldexp(1.0, -SCALE_SHIFT * np.arange(x.shape[0])).reshape((-1,) + (1,) * (x.ndim - 1))
    return x * sh


def scaled_add(x, y, *, nc):
    """Add-MCN of two scaled binary16 MC arrays (nc, n)."""
    return _scaled_ew(0, x, y, nc, True, True)


def scaled_mul(x, y, *, nc, x_mc=True, y_mc=False):
    """ScalingN of a scaled binary16 MC array by a plain binary16 one (either order)."""
    return _scaled_ew(1, x, y, nc, x_mc, y_mc)


def _scaled_ew(op, x, y, nc, x_mc, y_mc):
    x = _planar(x, np.float16)
    y = _planar(y, np.float16)
    n = x.shape[-1]
    x = x.reshape((nc if x_mc else 1), n)
    y = y.reshape((nc if y_mc else 1), n)
    out = np.empty((nc, n), dtype=np.float16)
    rc = lib().mcf_oracle_scaled_elementwise(op, nc, n, _ptr(x), int(x_mc), _ptr(y), int(y_mc), _ptr(out))
    if rc != 0:
        raise ValueError("oracle: bad arguments")
    return out


def scaled_matmul(A, B, *, nc, a_mc=True, b_mc=True, rows=None, cols=None):
    """C = A x B on scaled binary16 planes (MC x plain, plain x MC: MM-MCN; MC x MC:
    level-aligned parts of the linearity over B's components).  A: (nc|1, M, K),
    B: (nc|1, K, N); returns (nc, M, N) or (nc, count)."""
    A = _planar(A, np.float16)
    B = _planar(B, np.float16)
    if A.ndim == 2:
        A = A[None]
    if B.ndim == 2:
        B = B[None]
    M, K = A.shape[1:]
    K2, N = B.shape[1:]
    if K2 != K or A.shape[0] != (nc if a_mc else 1) or B.shape[0] != (nc if b_mc else 1):
        raise ValueError("scaled_matmul: shape mismatch")
    r, c, count = _positions(M, N, rows, cols)
    out = np.empty((nc, count), dtype=np.float16)
    rc = lib().mcf_oracle_scaled_matmul(nc, M, N, K, _ptr(A), int(a_mc), _ptr(B), int(b_mc), _ptr(r), _ptr(c),
                                        count, _ptr(out))
    if rc != 0:
        raise ValueError("oracle: bad arguments")
    return out.reshape(nc, M, N) if rows is None else out


def scaled_linear(X, W, bias=None, *, nc, rows=None, cols=None):
    """MC-Linear forward on scaled binary16 planes: X plain (T, I), W (nc, O, I),
    bias (nc, O) or None."""
    X = _planar(X, np.float16)
    W = _planar(W, np.float16)
    T, I = X.shape[-2:]
    O = W.shape[1]
    if W.shape != (nc, O, I):
        raise ValueError("scaled_linear: shape mismatch")
    if bias is not None:
        bias = _planar(bias, np.float16)
        if bias.shape != (nc, O):
            raise ValueError("scaled_linear: bias shape mismatch")
    r, c, count = _positions(T, O, rows, cols)
    out = np.empty((nc, count), dtype=np.float16)
    rc = lib().mcf_oracle_scaled_linear(nc, T, I, O, _ptr(X), _ptr(W), _ptr(bias), _ptr(r), _ptr(c), count,
                                        _ptr(out))
    if rc != 0:
        raise ValueError("oracle: bad arguments")
    return out.reshape(nc, T, O) if rows is None else out
