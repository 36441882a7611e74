"""Seeded synthetic inputs for multi-component (MC) arithmetic.

This module only draws random numbers and splits them into components; it holds
none of the MC algorithms.  Both the CPU oracle's tests and the GPU path take their
inputs from here.

An MC value with nc components is built from a float64 draw x by successive
rounding: c_0 = RN(x), c_1 = RN(x - c_0), c_2 = RN(x - c_0 - c_1), ... where RN
rounds to the component format (numpy's float64 -> float16/float32 conversion is
round-to-nearest-even with gradual underflow).  Each residual is exact in float64,
so the components are non-overlapping and decreasing, as an MCTensor requires
(Section 2, equation of the MCF expansion).

Arrays are component-major ("planar"): shape (nc, *shape).
"""
from __future__ import annotations

import numpy as np


def split(x: np.ndarray, nc: int, dtype) -> np.ndarray:
    """Split float64 values into nc components of `dtype` by successive rounding."""
    x = np.asarray(x, dtype=np.float64)
    dtype = np.dtype(dtype)
    out = np.empty((nc,) + x.shape, dtype=dtype)
    r = x.copy()
    with np.errstate(over="ignore"):
        for c in range(nc):
            out[c] = r.astype(dtype)
            r -= out[c].astype(np.float64)
    return out


SCALE_SHIFT = 11  # level c of a scaled binary16 value is stored times 2^(11 c)


def split_scaled(x: np.ndarray, nc: int) -> np.ndarray:
    """Split float64 values into nc binary16 components with scaled low components:
    c_0 = RN(x), and c_i = RN(2^(11 i) r_i) for the residual r_i = x - sum_{j<i}
    2^(-11 j) c_j, so component i stands for 2^(-11 i) c_i.  Each residual is exact in
    float64 (at most 44 bits are split off), so level i holds the next binary16
    precision of x instead of underflowing below 2^-24."""
    x = np.asarray(x, dtype=np.float64)
    out = np.empty((nc,) + x.shape, dtype=np.float16)
    r = x.copy()
    with np.errstate(over="ignore"):
        for c in range(nc):
            out[c] = np.ldexp(r, SCALE_SHIFT * c).astype(np.float16)
            r -= np.ldexp(out[c].astype(np.float64), -SCALE_SHIFT * c)
    return out


def expansion(g: np.random.Generator, shape, nc: int, dtype, scale: float = 1.0) -> np.ndarray:
    """MC values with every component in use (for formats where splitting a float64
    draw would leave the low components zero, such as binary64): c_0 ~ N(0, scale^2)
    rounded to `dtype`, each later component a uniform draw within a quarter ulp of the
    component before, rounded to `dtype`."""
    dtype = np.dtype(dtype)
    p = {np.dtype(np.float16): 11, np.dtype(np.float32): 24, np.dtype(np.float64): 53}[dtype]
    out = np.zeros((nc,) + tuple(np.atleast_1d(shape)), dtype=dtype)
    out[0] = g.normal(0.0, scale, out.shape[1:]).astype(dtype)
    for c in range(1, nc):
        prev = np.abs(out[c - 1].astype(np.float64))
        ulp = np.exp2(np.floor(np.log2(np.where(prev > 0, prev, 1.0))) - (p - 1))
        out[c] = np.where(prev > 0, g.uniform(-0.25, 0.25, out.shape[1:]) * ulp, 0.0).astype(dtype)
    return out


def rng(seed: int = 0) -> np.random.Generator:
    return np.random.default_rng(seed)


# ---------------------------------------------------------------------------------
# workload recipes (sizes are parameters so tests can scale them down)
# ---------------------------------------------------------------------------------

def matmul_uniform(M, N, K, nc, dtype, seed=0, lo=-1.0, hi=1.0):
    """A, B entries float64 ~ U[lo, hi], split into nc components (A drawn first)."""
    g = rng(seed)
    A = split(g.uniform(lo, hi, (M, K)), nc, dtype)
    B = split(g.uniform(lo, hi, (K, N)), nc, dtype)
    return A, B


def matmul_normal(M, N, K, nc, dtype, seed=0):
    """A, B entries float64 ~ N(0, 1/K), split into nc components (A drawn first)."""
    g = rng(seed)
    s = 1.0 / np.sqrt(K) if K > 0 else 1.0
    A = split(g.normal(0.0, s, (M, K)), nc, dtype)
    B = split(g.normal(0.0, s, (K, N)), nc, dtype)
    return A, B


def matmul_normal_scaled(M, N, K, nc, seed=0):
    """The same draws as matmul_normal, split into scaled binary16 components."""
    g = rng(seed)
    s = 1.0 / np.sqrt(K) if K > 0 else 1.0
    A = split_scaled(g.normal(0.0, s, (M, K)), nc)
    B = split_scaled(g.normal(0.0, s, (K, N)), nc)
    return A, B


def elementwise_inputs(op: str, n: int, nc: int, dtype, seed=0):
    """Operands for the elementwise workload on n elements.

    add: x, y ~ U[-1/2, 1/2];  mul, div: x ~ U[-1/2, 1/2], y ~ U[1/2, 3/2] (y is
    a divisor inside Mult-MCN and Div-MCN);  exp: x ~ U[-4, 4];  renorm: x ~
    U[-1/2, 1/2].  Returns (x, y) with y None for unary ops.
    """
    g = rng(seed)
    if op == "exp":
        return split(g.uniform(-4.0, 4.0, n), nc, dtype), None
    if op == "renorm":
        return split(g.uniform(-0.5, 0.5, n), nc, dtype), None
    x = split(g.uniform(-0.5, 0.5, n), nc, dtype)
    if op in ("mul", "div"):
        y = split(g.uniform(0.5, 1.5, n), nc, dtype)
    else:
        y = split(g.uniform(-0.5, 0.5, n), nc, dtype)
    return x, y


def linear_inputs(T, I, O, nc, dtype, layers=1, seed=0):
    """MC-Linear workload: x ~ N(0,1) rounded once (plain), then for each layer
    W ~ U(-1/sqrt(I), 1/sqrt(I)) of shape (O, I) and b ~ same of shape (O,), split
    into nc components.  Yields (x, W, b) per layer; x is shared."""
    g = rng(seed)
    x = g.normal(0.0, 1.0, (T, I)).astype(dtype)
    lim = 1.0 / np.sqrt(I)
    for _ in range(layers):
        W = split(g.uniform(-lim, lim, (O, I)), nc, dtype)
        b = split(g.uniform(-lim, lim, (O,)), nc, dtype)
        yield x, W, b


def linear_inputs_scaled(T, I, O, nc, layers=1, seed=0):
    """The MC-Linear workload's draws (as linear_inputs) with W and b split into
    scaled binary16 components; x stays a plain binary16 tensor."""
    g = rng(seed)
    x = g.normal(0.0, 1.0, (T, I)).astype(np.float16)
    lim = 1.0 / np.sqrt(I)
    for _ in range(layers):
        W = split_scaled(g.uniform(-lim, lim, (O, I)), nc)
        b = split_scaled(g.uniform(-lim, lim, (O,)), nc)
        yield x, W, b


def linreg_inputs(n, d, nc, dtype, seed=0):
    """The linear-regression precision experiment (Section 2.4): X (n, d) with entries
    ~ N(-0.5, 0.5^2) rounded once to `dtype`; target weights W* (d,) ~ N(-0.5, 0.5^2) in
    float64; targets y = X W*^T evaluated in float64 from the rounded X and rounded once;
    initial weights W0 ~ U(-1/sqrt(d), 1/sqrt(d)) (a linear layer's default
    initialisation) split into nc components.  Returns (X, y_neg = -y, W0 (nc, d), W*)."""
    g = rng(seed)
    X = g.normal(-0.5, 0.5, (n, d)).astype(dtype)
    w_star = g.normal(-0.5, 0.5, d)
    y = (X.astype(np.float64) @ w_star).astype(dtype)
    lim = 1.0 / np.sqrt(d)
    W0 = split(g.uniform(-lim, lim, d), nc, dtype)
    return X, (-y).astype(dtype), W0, w_star


def elementwise_suite(n: int, nc: int, dtype, seed=0):
    """The elementwise workload's operands drawn once: a ~ U[-1/2, 1/2] (first
    operand of every op and the Renormalize input), b ~ U[-1/2, 1/2] (second addend),
    d ~ U[1/2, 3/2] (divisor, and Mult-MCN's second factor), e ~ U[-4, 4] (exp
    input), each split into nc components."""
    g = rng(seed)
    return {
        "a": split(g.uniform(-0.5, 0.5, n), nc, dtype),
        "b": split(g.uniform(-0.5, 0.5, n), nc, dtype),
        "d": split(g.uniform(0.5, 1.5, n), nc, dtype),
        "e": split(g.uniform(-4.0, 4.0, n), nc, dtype),
    }
