"""Exact MC matrix product rounded into nc binary16 components -- CPU oracle.

TEST INFRASTRUCTURE ONLY: imported by tests/, the smoke check and bench.py's
CPU-baseline leg; the product library never uses it.  Plain Python integers, no
blocking or reordering: written to be checked by eye.

What is computed.  An MC number is the unevaluated sum of its components (Section
2.1), so an MC matrix product has one exact value per output,
    P_ij = sum_k (sum_c A^(c)_ik) (sum_c B^(c)_kj),
the quantity MM-MCN (Section 2.2, Appendix A.2.2) approximates with error at most
about 4 K u^nc sum_k |A_ik||B_kj| (Section 2.4).  This variant returns P_ij itself,
rounded into nc components by successive rounding:
    c_0 = RN(P),  c_1 = RN(P - c_0),  ...,  c_{nc-1} = RN(P - c_0 - ... - c_{nc-2}),
RN being IEEE-754 binary16 round-to-nearest-even with gradual underflow.  The
components are non-overlapping and their sum is within half an ulp of c_{nc-1}
(or 2^-25, the half subnormal quantum) of P, which is far inside the paper's bound.

Readings (the paper defines no such product; these are choices of this variant):
  * overflow: if |P| rounds beyond 65504 the result is (+-inf, 0, ..., 0);
  * non-finite inputs: an output whose row of A or column of B holds an infinite or
    NaN component is NaN in every component;
  * an exact zero gives +0 in every component;
  * with a bias row (the MC-Linear forward y = x W^T + b, Section 2.3), the bias is
    added to the exact sum before the split, and a non-finite bias component makes
    its column NaN.

Exactness.  Every binary16 value is an integer multiple of 2^-24, so each MC entry
is an integer X = sum_c x_c 2^24, and every product term is an integer in units of
2^-48.  The sums below are Python integers, hence exact at any size.
"""
from __future__ import annotations

import numpy as np

F16_MAX_UNITS48 = 65504 << 48          # largest finite binary16, in units of 2^-48
SUBNORMAL_QUANTUM_EXP = 24             # 2^-24 = 2^24 units of 2^-48


def f16_units24(x: np.ndarray) -> np.ndarray:
    """binary16 values -> Python ints x * 2^24 (object array); non-finite -> None."""
    x = np.asarray(x, dtype=np.float16)
    out = np.empty(x.shape, dtype=object)
    flat = x.ravel()
    res = out.ravel()
    for i, v in enumerate(flat.astype(np.float64)):
        if not np.isfinite(v):
            res[i] = None
        else:
            # v * 2^24 is an integer of at most 40 bits, exact in float64
            res[i] = int(v * 16777216.0)
    return out


def round_units48(v: int) -> tuple[int, int]:
    """RN(v * 2^-48) into binary16.  Returns (bits, value in units of 2^-48);
    value is None when the rounded magnitude overflows (bits is then +-inf)."""
    if v == 0:
        return 0, 0
    neg = v < 0
    a = -v if neg else v
    e = a.bit_length() - 1                  # 2^e <= a < 2^(e+1)
    qe = max(e - 10, SUBNORMAL_QUANTUM_EXP)  # 11 significant bits, floor at 2^-24
    q = 1 << qe
    n, r = divmod(a, q)
    if 2 * r > q or (2 * r == q and n % 2 == 1):
        n += 1
    mag = n * q
    sign = 0x8000 if neg else 0
    if mag > F16_MAX_UNITS48:
        return sign | 0x7C00, None
    # encode from the value: mag = m 2^(E-10) 2^48 with m in [2^10, 2^11) (normal)
    # or mag = m 2^24 with m < 2^10 (subnormal)
    if mag < (1 << 34):                     # below 2^-14: subnormal (or zero)
        bits = mag >> 24
    else:
        E = mag.bit_length() - 1 - 48       # unbiased exponent
        m = mag >> (E + 48 - 10)
        bits = ((E + 15) << 10) | (m - 1024)
    return sign | bits, (-mag if neg else mag)


def split_units48(v: int, nc: int) -> list[int]:
    """Successive rounding of v * 2^-48 into nc binary16 bit patterns."""
    out = []
    rem = v
    for _ in range(nc):
        bits, val = round_units48(rem)
        out.append(bits)
        if val is None:  # overflow: infinity, then zeros
            out += [0] * (nc - len(out))
            break
        rem -= val
    return out


def exact_sums(A, B, *, a_mc=True, b_mc=True):
    """P (M, N) as Python ints in units of 2^-48, and the non-finite masks.
    A: (planes, M, K), B: (planes, K, N) binary16."""
    A = np.asarray(A, dtype=np.float16)
    B = np.asarray(B, dtype=np.float16)
    if A.ndim == 2:
        A = A[None]
    if B.ndim == 2:
        B = B[None]
    Au = f16_units24(A)
    Bu = f16_units24(B)
    bad_a = np.array([[any(v is None for v in Au[:, i, k]) for k in range(A.shape[2])]
                      for i in range(A.shape[1])], dtype=bool).reshape(A.shape[1], A.shape[2])
    bad_b = np.array([[any(v is None for v in Bu[:, k, j]) for j in range(B.shape[2])]
                      for k in range(B.shape[1])], dtype=bool).reshape(B.shape[1], B.shape[2])
    Xa = np.zeros(A.shape[1:], dtype=object)
    Xb = np.zeros(B.shape[1:], dtype=object)
    for c in range(A.shape[0]):
        Xa = Xa + np.where(bad_a, 0, Au[c]).astype(object)
    for c in range(B.shape[0]):
        Xb = Xb + np.where(bad_b, 0, Bu[c]).astype(object)
    P = Xa.dot(Xb) if A.shape[2] > 0 else np.zeros((A.shape[1], B.shape[2]), dtype=object)
    row_bad = bad_a.any(axis=1) if A.shape[2] else np.zeros(A.shape[1], bool)
    col_bad = bad_b.any(axis=0) if B.shape[1] else np.zeros(B.shape[2], bool)
    return P, row_bad, col_bad


def matmul_exact(A, B, *, nc, a_mc=True, b_mc=True, rows=None, cols=None, bias=None) -> np.ndarray:
    """The exact product split into nc binary16 components.

    A: (nc|1, M, K), B: (nc|1, K, N), binary16; bias: optional (planes, N) binary16 MC
    row added exactly to every row of the product before the split (the MC-Linear
    forward y = x W^T + b).  Returns (nc, M, N) binary16, or (nc, count) at the given
    positions (rows, cols index arrays).  An output whose bias column holds a
    non-finite component is NaN in every component.
    """
    A = np.asarray(A, dtype=np.float16)
    B = np.asarray(B, dtype=np.float16)
    if A.ndim == 2:
        A = A[None]
    if B.ndim == 2:
        B = B[None]
    if A.shape[0] != (nc if a_mc else 1) or B.shape[0] != (nc if b_mc else 1) or A.shape[2] != B.shape[1]:
        raise ValueError("matmul_exact: shape mismatch")
    M, N = A.shape[1], B.shape[2]
    # the bias column sums, in units of 2^-48, and their non-finite flags
    bsum = [0] * N
    bbad = [False] * N
    if bias is not None:
        bu = f16_units24(np.asarray(bias, dtype=np.float16).reshape(-1, N))
        for j in range(N):
            bbad[j] = any(v is None for v in bu[:, j])
            bsum[j] = 0 if bbad[j] else sum(int(v) for v in bu[:, j]) << 24
    if rows is None:
        P, rb, cb = exact_sums(A, B)
        pos = [(i, j) for i in range(M) for j in range(N)]
        vals = [(P[i, j] + bsum[j], rb[i] or cb[j] or bbad[j]) for i, j in pos]
    else:
        rows = np.asarray(rows, dtype=np.int64).ravel()
        cols = np.asarray(cols, dtype=np.int64).ravel()
        vals = []
        for i, j in zip(rows, cols):
            P, rb, cb = exact_sums(A[:, i:i + 1, :], B[:, :, j:j + 1])
            vals.append((P[0, 0] + bsum[j], bool(rb[0] or cb[0] or bbad[j])))
    out = np.empty((nc, len(vals)), dtype=np.uint16)
    for t, (p, bad) in enumerate(vals):
        out[:, t] = [0x7E00] * nc if bad else split_units48(int(p), nc)
    out = out.view(np.float16)
    return out.reshape(nc, M, N) if rows is None else out
