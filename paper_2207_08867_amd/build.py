"""Build libmcf.so (the HIP kernels and the C ABI) for gfx950 with hipcc.

Flags that matter for the arithmetic:
  -ffp-contract=off   no multiply-add fusion except the explicit FMA of Two-Prod;
  no fast-math        IEEE rounding, gradual underflow, correctly rounded division;
  -fno-slp-vectorize  keep binary16 arithmetic scalar: gfx950 issues packed binary16
                      instructions at half the rate of scalar ones, so packing only adds
                      the cost of moving halves around;
  -packed-fp32-ops    the compiler may not pair binary32 operations into packed
                      instructions.
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libmcf.so")
SOURCES = ["abi.cpp", "elementwise.hip", "matmul.hip", "splitk.hip", "exact.hip", "linreg.hip", "scaled.hip",
           "exp64.hip", "linear_bwd.hip"]
# the VALU issue-rate probe behind the roofline figures (bench.py --issue-probe): a
# library of its own, not part of libmcf.so
PROBE_LIB = os.path.join(HERE, "libmcf_probe.so")
PROBE_SOURCES = ["issue_probe.hip"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

CFLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-ffp-contract=off",
    "-fno-gpu-flush-denormals-to-zero", "-fno-slp-vectorize",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
]


def build(verbose: bool = False) -> str:
    objdir = os.path.join(HERE, "_build")
    os.makedirs(objdir, exist_ok=True)
    procs = []
    objs = []
    for src in SOURCES + PROBE_SOURCES:
        obj = os.path.join(objdir, os.path.splitext(src)[0] + ".o")
        objs.append(obj)
        cmd = [HIPCC, *CFLAGS, "-c", os.path.join(CSRC, src), "-o", obj]
        if src.endswith(".cpp"):
            cmd[1:1] = ["-x", "hip"]
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append((src, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)))
    failed = []
    for src, p in procs:
        out, _ = p.communicate()
        if p.returncode != 0:
            failed.append((src, out))
        elif verbose and out.strip():
            print(out, flush=True)
    if failed:
        for src, out in failed:
            sys.stderr.write(f"--- {src} ---\n{out}\n")
        raise RuntimeError("hipcc failed for " + ", ".join(s for s, _ in failed))
    probe_objs = [o for o, src in zip(objs, SOURCES + PROBE_SOURCES) if src in PROBE_SOURCES]
    for target, parts in ((LIB, [o for o in objs if o not in probe_objs]), (PROBE_LIB, probe_objs)):
        tmp = target + ".tmp"
        cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *parts]
        subprocess.run(cmd, check=True)
        os.replace(tmp, target)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
