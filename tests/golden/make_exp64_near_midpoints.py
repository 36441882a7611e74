"""Writes exp64_near_midpoints.txt: binary64 arguments x whose e^x lies within 2^-72
(relative) of a binary64 rounding boundary, found by the oracle's binary128 search over
seeded random arguments (whole range, the range of subnormal results, and |x| < 2^-27,
where e^x is 1 + x + x^2/2 + ... to far beyond binary64).  A
correctly rounded binary64 exponential that first evaluates e^x to a few bits beyond
2^-70 must take its slow path on every one of them.  Run from the repository root:
    python tests/golden/make_exp64_near_midpoints.py
"""
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402

REL = 2.0 ** -72
runs = [(-745.0, 709.7, 1, 1 << 26), (-745.13, -708.4, 2, 1 << 24), (-0.5, 0.5, 3, 1 << 24),
        (-2.0 ** -27, 2.0 ** -27, 4, 1 << 24)]
xs = []
for lo, hi, seed, tries in runs:
    xs.extend(float(v) for v in oracle.exp64_near_midpoints(lo, hi, seed, tries, REL, max_out=100000))
path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "exp64_near_midpoints.txt")
with open(path, "w") as f:
    f.write("# binary64 x (hex) with e^x within 2^-72 of a binary64 rounding boundary;\n")
    f.write("# written by make_exp64_near_midpoints.py (oracle binary128 search, seeded)\n")
    for v in sorted(set(xs)):
        f.write(float.hex(v) + "\n")
print(len(set(xs)), "arguments written to", path)
