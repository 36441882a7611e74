"""Exhaustive binary16 pins of the oracle's error-free transformations and division:
every one of the 2^32 pairs (a, b) of binary16 encodings, against closed forms that
numpy evaluates exactly in binary64 (the sum, difference and product of two binary16
numbers are exact in binary64, and rounding a binary64 quotient to binary16 is
innocuous double rounding, 53 >= 2*11 + 2):
  * Two-Sum:  s = RN16(a + b), e = (a + b) - s exactly -- except where the algorithm's
              intermediate fl(s - a) overflows although a + b does not (|s| in the
              top binade, e.g. a = 48, b = -65504), where its error is NaN;
  * Two-Prod: p = RN16(a b),   e = RN16(a b - p);
  * division: RN16(a / b) (Div-MCN at nc = 1 is this quotient up to the sign of a zero).
Pairs whose rounded result overflows are checked for the overflow (infinite s or p)
only.  About half an hour on eight cores: marked slow and run when MCF_EXHAUSTIVE=1
(the GPU tier checks the library's binary16 division over all pairs against the
oracle in tests/test_gpu_div_exhaustive.py)."""
import os

import numpy as np
import pytest

pytestmark = [pytest.mark.slow,
              pytest.mark.skipif(os.environ.get("MCF_EXHAUSTIVE") != "1",
                                 reason="exhaustive 2^32-pair pins: set MCF_EXHAUSTIVE=1 (about half an hour)")]

ALL = np.arange(65536, dtype=np.uint32).astype(np.uint16).view(np.float16)
FIN = ALL[np.isfinite(ALL)]
BLOCK = 512


def _blocks():
    for i in range(0, FIN.size, BLOCK):
        a = FIN[i:i + BLOCK]
        yield np.repeat(a, FIN.size).astype(np.float64), np.tile(FIN, a.size).astype(np.float64)


def test_two_sum_all_pairs(orc):
    L = orc.lib()
    for a, b in _blocks():
        s = np.empty_like(a)
        e = np.empty_like(a)
        L.mcf_oracle_eft_array(0, 0, a.size, orc._ptr(a), orc._ptr(b), orc._ptr(s), orc._ptr(e))
        with np.errstate(over="ignore", invalid="ignore"):
            ws = (a + b).astype(np.float16).astype(np.float64)
            # the algorithm's second step fl(s - a) overflows for a few pairs whose sum
            # is finite (|s| in the top binade, a of the opposite sign): the error is NaN
            ovf = np.isinf((ws - a).astype(np.float16))
        fin = np.isfinite(ws)
        assert np.array_equal(np.isinf(s), ~fin)
        assert np.array_equal(s[fin], ws[fin])
        ok = fin & ~ovf
        assert np.array_equal(e[ok], (a + b - ws)[ok])
        assert np.isnan(e[fin & ovf]).all()


def test_two_prod_all_pairs(orc):
    L = orc.lib()
    for a, b in _blocks():
        p = np.empty_like(a)
        e = np.empty_like(a)
        L.mcf_oracle_eft_array(0, 1, a.size, orc._ptr(a), orc._ptr(b), orc._ptr(p), orc._ptr(e))
        ab = a * b
        with np.errstate(over="ignore"):
            wp = ab.astype(np.float16).astype(np.float64)
        fin = np.isfinite(wp)
        assert np.array_equal(np.isinf(p), ~fin)
        assert np.array_equal(p[fin], wp[fin])
        we = (ab - wp)[fin].astype(np.float16).astype(np.float64)
        assert np.array_equal(e[fin], we)


def test_division_all_pairs(orc):
    L = orc.lib()
    for a, b in _blocks():
        q = np.empty_like(a)
        L.mcf_oracle_binop_array(0, 3, a.size, orc._ptr(a), orc._ptr(b), orc._ptr(q))
        with np.errstate(all="ignore"):
            w = (a / b).astype(np.float16).astype(np.float64)
        nan = np.isnan(w)
        assert np.array_equal(np.isnan(q), nan)
        assert np.array_equal(q[~nan], w[~nan])
        assert np.array_equal(np.signbit(q[~nan]), np.signbit(w[~nan]))
