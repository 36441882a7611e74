#!/usr/bin/env python3
"""Throughput of the multi-component (MC) matrix product on one MI355X.

Headline workload: C = A B with binary32 components, nc = 3, M = N = K = 8192,
A and B drawn float64 ~ N(0, 1/K) (seed 0) and split into 3 components by
successive rounding, both operands MC.  One step is one full product; the metric is
MC-GFLOP/s = 2 M N K / time (one MC multiply-add counts as 2 flops), inputs resident
in HBM before the timed region.

Also reported on the same line (not part of `value`):
  * roofline of the product kernel: algorithmic VALU operations per launch over the
    launch duration measured with HIP events, against the VALU issue peak;
  * the maximum error against the exact product on sampled outputs;
  * the pruned MC x MC product (mc_matmul_pruned) on the headline operands;
  * the other workloads (64^3 binary32 nc=2; 1024^3 binary16 nc=2 and 3; the
    4096x1024x1024 binary16 nc=3 MC-Linear over 100 layers; the exact binary16
    product on the int8 matrix cores at 1024^3 and the MC-Linear layer shape; the
    paper's linear-regression gradient descent (time per step, final loss); binary64
    components (2^26-element Add-MCN, ScalingN, Div-MCN and a 1024^3 product); the
    2^26-element binary16
    nc=3 elementwise operations with their HBM bandwidth; the K-split Dot and MV; the
    paper's BMM-MCN and AddMM-MCN sizes);
  * cpu_baseline: the CPU oracle timed on a sample of the headline workload.

Usage: python bench.py [--gpus 1] [--steps 3] [--warmup 1] [--no-extra]
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

# VALU issue peak: 256 CUs x 128 binary32 lane-operations per clock x 2.4 GHz = 78.6e12
# lane-operations / s (the 157.3 TFLOP/s binary32 vector figure counts an FMA as two).
# A packed binary16 instruction carries two lanes of work but issues at half rate, so
# the element-operation peak is the same for binary16.
VALU_PEAK = 256 * 128 * 2.4e9
HBM_PEAK = 8.0e12  # bytes / s


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def algo_ops_per_mac(nc: int, mc_x_mc: bool) -> int:
    """Floating-point operations of the algorithm that determine the result, per
    multiply-add, on the common path where Simple-Renorm keeps the first nc terms and
    drops the final carry (whose computation is then not needed):
      ScalingN: component 0: mul + fma; components 1..nc-2: mul + fma + Two-Sum (6)
                + carry add; component nc-1: mul + add (the kept sum only);
      Add-MCN:  component 0: Two-Sum (6; the Two-Sum with the zero carry is an
                identity); components 1..nc-2: two Two-Sums + carry add (13);
                component nc-1: add + add.
    nc = 1: one mul, one add.  MC x MC repeats this for each component of B.
    Zero checks, selects, loads and loop control are overhead, not counted."""
    if nc == 1:
        per = 2
    else:
        per = (2 + 9 * (nc - 2) + 2) + (6 + 13 * (nc - 2) + 2)
    return per * (nc if mc_x_mc else 1)


def pruned_ops_per_mac(nc: int) -> int:
    """Essential operations per multiply-add of the pruned MC x MC product: component p
    of B drives an (nc - p)-component ScalingN + Add-MCN step (counted as in
    algo_ops_per_mac): 34 + 12 + 2 = 48 at nc = 3."""
    return sum(algo_ops_per_mac(nc - p, False) for p in range(nc))


def ew_fp_ops(op: str, nc: int) -> int:
    """Floating-point operations of the printed elementwise algorithm per element, for
    the VALU-bound ones: Two-Sum = 6, Two-Prod = 2 (mul + fma), a carry addition = 1,
    a component division = 1; negations and Simple-Renorm's compare/selects are not
    counted, nor the Two-Sums and divisions the kernel can prove unnecessary.
      ScalingN(nc):  2 nc + 7 (nc - 1);   Add-MCN(nc): 6 + 13 (nc - 1);
      Div-MCN:       (nc + 1) divisions + nc (ScalingN + Add-MCN);
      Renormalize:   (nc - 1) + nc Two-Sums;
      Mult-MCN:      2 Div-MCN + 2 Renormalize;
      Mult-MCN-Slow: 1 + nc (Div-MCN + Add-MCN + 1)."""
    scal = 2 * nc + 7 * (nc - 1)
    add = 6 + 13 * (nc - 1)
    div = (nc + 1) + nc * (scal + add)
    if op == "div":
        return div
    if op == "mult_slow":  # first digit, then nc times DivN + Add-MCN + next digit
        return 1 + nc * (div + add + 1)
    return 2 * div + 2 * 6 * (2 * nc - 1)


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "mm_kernel_f32_nc3_8192.traffic.txt")


def measured_traffic():
    """HBM bytes per launch of the headline kernel from its rocprofv3 counter record,
    or None when the record is missing or the kernel sources changed since."""
    import hashlib

    try:
        kv = {}
        for line in open(TRAFFIC_FILE):
            if "=" in line and not line.lstrip().startswith("#"):
                k, v = line.split("=", 1)
                kv[k.strip()] = v.strip()
        h = hashlib.sha256()
        for f in kv["sources"].split():
            h.update(open(os.path.join(ROOT, f), "rb").read())
        if h.hexdigest() != kv["source_sha256"]:
            return None
        return float(kv["fetch_bytes"]) + float(kv["write_bytes"])
    except (OSError, KeyError, ValueError):
        return None


COUNTER_FILE = os.path.join(ROOT, "profiles", "valu_counters.txt")


def valu_counts():
    """VALU instructions per launch (wave64 SQ_INSTS_VALU) from the committed rocprofv3
    counter table, for the groups whose kernel sources still hash to what was
    measured: {workload: count}."""
    import hashlib

    out = {}
    try:
        groups, cur = {}, None
        for line in open(COUNTER_FILE):
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            if line.startswith("[") and line.endswith("]"):
                cur = groups.setdefault(line[1:-1], {})
            elif "=" in line and cur is not None:
                k, v = line.split("=", 1)
                cur[k.strip()] = v.strip()
        for kv in groups.values():
            h = hashlib.sha256()
            for f in kv["sources"].split():
                h.update(open(os.path.join(ROOT, f), "rb").read())
            if h.hexdigest() != kv["source_sha256"]:
                continue
            out.update({k: float(v) for k, v in kv.items() if k not in ("sources", "source_sha256")})
    except (OSError, KeyError, ValueError):
        return {}
    return out


def issue_fields(key, seconds, work_units=None):
    """Measured VALU issue efficiency of one launch: the counted lane-instructions
    (64 per wave64 instruction) over the live launch time, against the VALU issue peak;
    plus lane-instructions per unit of work (per MAC or per element).  Empty when the
    counter table does not cover the current sources."""
    c = valu_counts().get(key)
    if c is None:
        return {}
    lanes = 64.0 * c
    out = {"issue_frac": round(lanes / seconds / VALU_PEAK, 3)}
    if work_units:
        out["valu_lane_instr_per_unit"] = round(lanes / work_units, 1)
    return out


class Timer:
    """HIP events on torch's current stream, the stream the library launches on."""

    def __init__(self, torch):
        self.torch = torch
        self.pairs = []

    def run(self, fn):
        s = self.torch.cuda.Event(enable_timing=True)
        e = self.torch.cuda.Event(enable_timing=True)
        s.record()
        fn()
        e.record()
        self.pairs.append((s, e))

    def ms(self):
        self.torch.cuda.synchronize()
        return [s.elapsed_time(e) for s, e in self.pairs]


def warm(torch, fn, seconds=0.2, min_calls=3):
    """Untimed calls of fn for at least `seconds` of wall time (and min_calls calls):
    the timed calls that follow then run at the clocks the workload holds once the GPU
    is busy, not during the ramp after the host-side work before it (input generation,
    error checks), which costs the first calls of a 1 ms product up to 10%."""
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    n = 0
    while n < min_calls or time.perf_counter() - t0 < seconds:
        fn()
        n += 1
        if n % 4 == 0:
            torch.cuda.synchronize()
    torch.cuda.synchronize()


def bench_matmul(torch, mcf, A, B, nc, steps, warmup, a_mc=True, b_mc=True, warm_s=0.0):
    """warmup untimed calls (warm_s > 0: untimed calls for warm_s seconds instead),
    then `steps` timed ones."""
    tA = torch.from_numpy(A).cuda()
    tB = torch.from_numpy(B).cuda()
    M, K = A.shape[1:]
    N = B.shape[2]
    C = torch.empty((nc, M, N), dtype=tA.dtype, device="cuda")
    if warm_s > 0:
        warm(torch, lambda: mcf.mc_matmul(tA, tB, nc=nc, a_mc=a_mc, b_mc=b_mc, out=C), warm_s, warmup)
    for _ in range(0 if warm_s > 0 else warmup):
        mcf.mc_matmul(tA, tB, nc=nc, a_mc=a_mc, b_mc=b_mc, out=C)
    torch.cuda.synchronize()
    tm = Timer(torch)
    t0 = time.perf_counter()
    for _ in range(steps):
        tm.run(lambda: mcf.mc_matmul(tA, tB, nc=nc, a_mc=a_mc, b_mc=b_mc, out=C))
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    return C, wall / steps * 1e3, float(np.mean(tm.ms()))


U_OF = {np.dtype(np.float16): 2.0 ** -11, np.dtype(np.float32): 2.0 ** -24, np.dtype(np.float64): 2.0 ** -53}
# half the smallest subnormal of the component format
ETA_OF = {np.dtype(np.float16): 2.0 ** -25, np.dtype(np.float32): 2.0 ** -150, np.dtype(np.float64): 2.0 ** -1075}


def exact_error(oracle, A, B, C, nc, K, dt, count=64, seed=5, bias=None):
    """Error of a computed product C against the exact product of the MC inputs (plus
    an optional bias row: the MC-Linear layer), on `count` sampled outputs:
      max_rel_err      max |C - C*| / (|A||B|) (with |bias| added to |A||B|);
      literal_ratio    max_rel_err / (4 K u^nc), the tolerance stated for the product:
                       <= 1 means it holds on every sampled output;
      amended_ratio    max |C - C*| / (4 K u^min(nc,3) |A||B| + nA nB K eta): the same
                       bound with the binary16 floor for Two-Prod errors below the
                       subnormal grid (eta = half the smallest subnormal; no floor in
                       binary32 / binary64) and u^3 beyond nc = 3;
      rms_err_over_sqrtK_eta  (binary16) the rms absolute error in units of sqrt(K) eta,
                       the size the floor predicts for errors lost below the grid."""
    M, N = C.shape[1:]
    g = np.random.default_rng(seed)
    rows = g.integers(0, M, count)
    cols = g.integers(0, N, count)
    Cs = np.ascontiguousarray(C[:, rows, cols])
    err, absab, _ = oracle.matmul_exact_err(A, B, Cs, bias=bias, rows=rows, cols=cols)
    rel = np.abs(err) / absab
    dtn = np.dtype(dt)
    u, eta = U_OF[dtn], ETA_OF[dtn]
    literal = 4 * K * u ** nc
    floor = A.shape[0] * B.shape[0] * K * eta if dtn == np.dtype(np.float16) else 0.0
    amended = 4 * K * u ** min(nc, 3) * absab + floor
    out = {"sampled_outputs": int(count), "max_rel_err": float(rel.max()), "bound_literal_4Ku^nc": literal,
           "literal_ratio": float(rel.max() / literal), "literal_holds": bool(rel.max() <= literal),
           "amended_ratio": float(np.max(np.abs(err) / amended)),
           "rms_rel_err": float(np.sqrt(np.mean(rel * rel)))}
    if dtn == np.dtype(np.float16):
        out["rms_err_over_sqrtK_eta"] = float(np.sqrt(np.mean(err * err)) / (np.sqrt(K) * eta))
    return out


def cpu_oracle_other(oracle, inputs):
    """The CPU oracle on bounded samples of the other workloads, for context beside the
    GPU lines: binary16 nc = 3 elementwise operations on 2^22 elements, 32 full rows of the
    1024^3 binary16 nc = 3 MC x MC product and of the 4096x1024x1024 MC-Linear layer, and
    the whole 64^3 binary32 nc = 2 product."""
    out = {"threads": oracle.threads(), "cpu_model": cpu_model()}
    n, nc = 1 << 22, 3
    s = inputs.elementwise_suite(n, nc, np.float16, seed=0)
    for name, fn, bpe in (("add_mcn", lambda: oracle.add(s["a"], s["b"], nc=nc), 18),
                          ("div_mcn", lambda: oracle.div(s["a"], s["d"], nc=nc), 18),
                          ("mult_mcn", lambda: oracle.mul(s["a"], s["d"], nc=nc), 18),
                          ("exp_mcn", lambda: oracle.exp(s["e"], nc=nc), 12)):
        t0 = time.perf_counter()
        fn()
        dt = time.perf_counter() - t0
        out[name] = {"Melem/s": round(n / dt / 1e6, 2), "GB/s": round(bpe * n / dt / 1e9, 3),
                     "sample": "2^22 elements, binary16 nc = 3", "seconds": round(dt, 3)}
    A, B = inputs.matmul_normal(1024, 1024, 1024, nc, np.float16, seed=0)
    rows = np.repeat(np.arange(32), 1024)
    cols = np.tile(np.arange(1024), 32)
    t0 = time.perf_counter()
    oracle.matmul(A, B, nc=nc, rows=rows, cols=cols)
    dt = time.perf_counter() - t0
    out["matmul_1024_f16_nc3"] = {"MC-GFLOP/s": round(2.0 * rows.size * 1024 / dt / 1e9, 5),
                                  "sample": "32 full rows (32768 outputs, K = 1024)", "seconds": round(dt, 3)}
    A, B = inputs.matmul_uniform(64, 64, 64, 2, np.float32, seed=0)
    t0 = time.perf_counter()
    oracle.matmul(A, B, nc=2)
    dt = time.perf_counter() - t0
    out["matmul_64_f32_nc2"] = {"MC-GFLOP/s": round(2.0 * 64 ** 3 / dt / 1e9, 5), "sample": "the full product",
                                "seconds": round(dt, 4)}
    x, W, b = next(inputs.linear_inputs(4096, 1024, 1024, nc, np.float16, layers=1, seed=0))
    rows = np.repeat(np.arange(32), 1024)
    cols = np.tile(np.arange(1024), 32)
    t0 = time.perf_counter()
    oracle.linear(x, W, b, nc=nc, rows=rows, cols=cols)
    dt = time.perf_counter() - t0
    out["linear_4096x1024x1024_f16_nc3"] = {"MC-GFLOP/s": round(2.0 * rows.size * 1024 / dt / 1e9, 5),
                                            "sample": "32 full rows of the first layer (32768 outputs, K = 1024)",
                                            "seconds": round(dt, 3)}
    return out


def cpu_baseline(oracle, A, B, nc, target_s=12.0):
    """The oracle on a bounded sample of output entries of the headline product."""
    M, K = A.shape[1:]
    N = B.shape[2]
    g = np.random.default_rng(9)
    probe = 16
    t0 = time.perf_counter()
    oracle.matmul(A, B, nc=nc, rows=g.integers(0, M, probe), cols=g.integers(0, N, probe))
    dt = time.perf_counter() - t0
    count = int(max(probe, min(16384, probe * target_s / max(dt, 1e-3))))
    threads = oracle.threads()
    count = max(threads, (count // threads) * threads)
    rows = g.integers(0, M, count)
    cols = g.integers(0, N, count)
    t0 = time.perf_counter()
    oracle.matmul(A, B, nc=nc, rows=rows, cols=cols)
    dt = time.perf_counter() - t0
    return {"value": 2.0 * K * count / dt / 1e9, "unit": "MC-GFLOP/s", "cores": threads, "kind": "oracle",
            "sample": f"{count} sampled outputs of the 8192^3 product (each a full K = {K} reduction), "
                      f"{dt:.1f} s", "seconds": dt, "cpu_model": cpu_model()}


def cpu_model():
    """The host CPU's model name (first 'model name' line of /proc/cpuinfo)."""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def bench_elementwise(torch, mcf, inputs, steps=10):
    n, nc, dt = 1 << 26, 3, np.float16
    s = inputs.elementwise_suite(n, nc, dt, seed=0)
    dev = {k: torch.from_numpy(v).cuda() for k, v in s.items()}
    out = torch.empty((nc, n), dtype=torch.float16, device="cuda")
    ops = {
        "add_mcn": (lambda: mcf.mc_add(dev["a"], dev["b"], nc=nc, out=out), 18),
        "grow_expn": (lambda: mcf.mc_add(dev["a"], dev["b"][0], nc=nc, y_mc=False, out=out), 14),
        "scaling_n": (lambda: mcf.mc_mul(dev["a"], dev["d"][0], nc=nc, y_mc=False, out=out), 14),
        "mult_mcn": (lambda: mcf.mc_mul(dev["a"], dev["d"], nc=nc, out=out), 18),
        "div_mcn": (lambda: mcf.mc_div(dev["a"], dev["d"], nc=nc, out=out), 18),
        "exp_mcn": (lambda: mcf.mc_exp(dev["e"], nc=nc, out=out), 12),
        "renormalize": (lambda: mcf.mc_renorm(dev["a"], mode=0, out=out), 12),
        # Square-MCN depends on the two leading components only: 4 bytes read, 6 written
        "square_mcn": (lambda: mcf.mc_square(dev["a"], nc=nc, out=out), 10),
        "mult_mcn_slow": (lambda: mcf.mc_mul_slow(dev["a"], dev["d"], nc=nc, out=out), 18),
    }
    # binary32 Exp-MCN (correctly rounded component exponential), same input recipe
    e32 = torch.from_numpy(inputs.split(np.random.default_rng(0).uniform(-4.0, 4.0, n), nc, np.float32)).cuda()
    out32 = torch.empty((nc, n), dtype=torch.float32, device="cuda")
    ops["exp_mcn_f32"] = (lambda: mcf.mc_exp(e32, nc=nc, out=out32), 24)
    res = {}
    for name, (fn, bpe) in ops.items():
        warm(torch, fn)
        tm = Timer(torch)
        for _ in range(steps):
            tm.run(fn)
        ms = float(np.median(tm.ms()))
        gbs = bpe * n / (ms * 1e-3) / 1e9
        res[name] = {"us": round(ms * 1e3, 1), "GB/s": round(gbs, 1), "hbm_frac": round(gbs * 1e9 / HBM_PEAK, 3),
                     "Gelem/s": round(n / (ms * 1e-3) / 1e9, 2)}
        if name in ("mult_mcn", "div_mcn", "mult_mcn_slow"):  # VALU-bound: their binding roofline
            nops = ew_fp_ops({"div_mcn": "div", "mult_mcn": "mult", "mult_mcn_slow": "mult_slow"}[name], nc)
            res[name]["printed_fp_ops_per_elem"] = nops
            res[name]["valu_frac_printed_ops"] = round(nops * n / (ms * 1e-3) / VALU_PEAK, 3)
        res[name].update(issue_fields(name, ms * 1e-3, n))
        log(f"  elementwise {name}: {ms * 1e3:.1f} us, {gbs:.0f} GB/s")
    return {"workload": "2^26 elements, binary16, nc = 3", "ops": res}


def bench_splitk(torch, mcf, inputs, steps=20):
    """K-split products on the shapes they are for, with their HBM bandwidth:
    Dot-MCN of two binary32 nc = 2 MC vectors of 2^24 entries, and MV-MCN of an
    8192 x 8192 binary32 nc = 3 MC matrix by a plain vector (default slice counts)."""
    res = {}
    cases = (("dot_2^24_f32_nc2", 1, 1, 1 << 24, 2, True, True),
             ("mv_8192x8192_f32_nc3", 8192, 1, 8192, 3, True, False))
    for name, M, N, K, nc, a_mc, b_mc in cases:
        A, B = inputs.matmul_normal(M, N, K, nc, np.float32, seed=0)
        tA = torch.from_numpy(A if a_mc else A[:1]).cuda()
        tB = torch.from_numpy(B if b_mc else B[:1]).cuda()
        del A, B
        out = torch.empty((nc, M, N), dtype=torch.float32, device="cuda")
        S = mcf.mc_matmul_splitk_slices(M, N, K)
        wb = mcf.mc_matmul_splitk_workspace(1, nc, M, N, K, a_mc, b_mc, S)
        ws = torch.empty(max(wb, 1), dtype=torch.uint8, device="cuda")
        fn = lambda: mcf.mc_matmul_splitk(tA, tB, nc=nc, a_mc=a_mc, b_mc=b_mc, out=out, workspace=ws)
        warm(torch, fn)
        tm = Timer(torch)
        for _ in range(steps):
            tm.run(fn)
        ms = float(np.median(tm.ms()))
        nbytes = (tA.numel() + tB.numel() + out.numel()) * 4
        gbs = nbytes / (ms * 1e-3) / 1e9
        res[name] = {"us": round(ms * 1e3, 1), "slices": S, "GB/s": round(gbs, 1),
                     "hbm_frac": round(gbs * 1e9 / HBM_PEAK, 3),
                     "MC-GFLOP/s": round(2 * M * N * K / (ms * 1e-3) / 1e9, 1)}
        log(f"  splitk {name}: {ms * 1e3:.1f} us, {gbs:.0f} GB/s (S = {S})")
        del tA, tB, out, ws
    return res


# The paper's CPU times (Ryzen 7 5800X, PyTorch 1.11; Appendix A.3, matrix operator
# table) for 1-, 2-, 3-component MC x plain products: context, not a target.
PAPER_CPU_S = {"bmm": (4.84, 8.03, 11.2), "addmm": (0.750, 1.12, 1.44)}


def bench_batched(torch, mcf, inputs, steps=20):
    """The paper's BMM-MCN (16 x 500 x 200) x (16 x 200 x 50) and AddMM-MCN
    100 + (500 x 200) x (200 x 100) workloads, MC x plain, binary32, nc = 1, 2, 3."""
    res = {}
    g = np.random.default_rng(0)
    for nc in (1, 2, 3):
        A = inputs.split(g.normal(0.0, 1 / np.sqrt(200), (16, 500, 200)), nc, np.float32)
        B = inputs.split(g.normal(0.0, 1 / np.sqrt(200), (16, 200, 50)), 1, np.float32)
        tA, tB = torch.from_numpy(A).cuda(), torch.from_numpy(B).cuda()
        out = torch.empty((nc, 16, 500, 50), dtype=torch.float32, device="cuda")
        cases = [("bmm", lambda: mcf.mc_bmm(tA, tB, nc=nc, b_mc=False, out=out), 16 * 500 * 200 * 50)]
        A2 = inputs.split(g.normal(0.0, 1 / np.sqrt(200), (500, 200)), nc, np.float32)
        B2 = inputs.split(g.normal(0.0, 1 / np.sqrt(200), (200, 100)), 1, np.float32)
        Y2 = inputs.split(g.normal(0.0, 1.0, (100,)), nc, np.float32)
        tA2, tB2, tY2 = (torch.from_numpy(v).cuda() for v in (A2, B2, Y2))
        out2 = torch.empty((nc, 500, 100), dtype=torch.float32, device="cuda")
        cases.append(("addmm", lambda: mcf.mc_addmm(tA2, tB2, tY2, nc=nc, alpha=1.0, beta=1.0, out=out2),
                      500 * 200 * 100))
        for name, fn, macs in cases:
            warm(torch, fn)
            tm = Timer(torch)
            for _ in range(steps):
                tm.run(fn)
            ms = float(np.median(tm.ms()))
            res[f"{name}_f32_nc{nc}"] = {
                "us": round(ms * 1e3, 1), "MC-GFLOP/s": round(2 * macs / (ms * 1e-3) / 1e9, 1),
                "valu_frac": round(algo_ops_per_mac(nc, False) * macs / (ms * 1e-3) / VALU_PEAK, 3),
                "paper_cpu_s": PAPER_CPU_S[name][nc - 1]}
            log(f"  {name} nc={nc}: {ms * 1e3:.1f} us")
    return {"workload": "BMM-MCN (16x500x200)x(16x200x50), AddMM-MCN 100+(500x200)x(200x100); MC x plain, "
                        "binary32", "ops": res}


def bench_linear(torch, mcf, oracle, inputs, layers=100):
    """MC-Linear y = x W^T + b over 100 independent layers (binary16 nc = 3), with the
    error against the exact layer output on 2048 sampled outputs of the first and of
    the last layer."""
    T, I, O, nc = 4096, 1024, 1024, 3
    gen = inputs.linear_inputs(T, I, O, nc, np.float16, layers=layers, seed=0)
    x = None
    Ws, bs, host = [], [], {}
    for l, (xx, W, b) in enumerate(gen):
        x = xx
        Ws.append(torch.from_numpy(W).cuda())
        bs.append(torch.from_numpy(b).cuda())
        if l in (0, layers - 1):
            host[l] = (np.ascontiguousarray(W.transpose(0, 2, 1)), b)
    tx = torch.from_numpy(x).cuda()
    y = torch.empty((nc, T, O), dtype=torch.float16, device="cuda")
    warm(torch, lambda: mcf.mc_linear_fwd(tx, Ws[0], bs[0], out=y))
    tm = Timer(torch)
    t0 = time.perf_counter()
    for W, b in zip(Ws, bs):
        tm.run(lambda: mcf.mc_linear_fwd(tx, W, b, out=y))
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    kms = float(np.mean(tm.ms()))
    macs = T * I * O
    errors = {}
    for l, (Wt, b) in host.items():
        mcf.mc_linear_fwd(tx, Ws[l], bs[l], out=y)
        errors[f"layer_{l}"] = exact_error(oracle, x[None], Wt, y.cpu().numpy(), nc, I, np.float16, count=2048,
                                           seed=11 + l, bias=b)
    # the backward of one layer (dX = dY W, dW = dY^T x, db), dY a plain gradient and an MC one
    bwd = {}
    g = np.random.default_rng(12)
    dYmc = torch.from_numpy(inputs.split(g.normal(0.0, 1 / 32, (T, O)), nc, np.float16)).cuda()
    ws = torch.empty(mcf.mc_linear_bwd_workspace(0, nc, T, I, O), dtype=torch.uint8, device="cuda")
    for kind, dY, mc in (("plain_dY", dYmc[0].contiguous(), False), ("mc_dY", dYmc, True)):
        run = lambda: mcf.mc_linear_bwd(tx, Ws[0], dY, dy_mc=mc, workspace=ws)
        warm(torch, run)
        tb = Timer(torch)
        for _ in range(3):
            tb.run(run)
        bwd[kind] = {"ms": round(float(np.median(tb.ms())), 3)}
    return {"workload": f"MC-Linear {T}x{I}x{O} binary16 nc=3, {layers} layers", "ms_per_layer": round(kms, 3),
            "backward_one_layer": bwd,
            "MC-GFLOP/s": round(2 * macs * layers / wall / 1e9, 1),
            "valu_frac_printed_ops": round(algo_ops_per_mac(nc, False) * macs / (kms * 1e-3) / VALU_PEAK, 3),
            **issue_fields("linear_4096x1024x1024_f16_nc3", kms * 1e-3, macs), "error": errors}


MFMA_I8_PEAK = 5.0e15  # dense int8 matrix-core operations / s


def digit_levels(X16):
    """Balanced base-256 digit levels in use by binary16 MC entries (planes first):
    (lowest, highest + 1) over the whole operand.  Measurement support only: the
    number of int8 digit-pair contractions the exact product performs."""
    X = np.zeros(X16.shape[1:], dtype=np.int64)
    for c in range(X16.shape[0]):
        X += np.round(X16[c].astype(np.float64) * 2.0 ** 24).astype(np.int64)
    D = (X + 0x808080808080) ^ 0x808080808080  # digit bytes (zero byte = zero digit)
    used = [bool(((D >> (8 * s)) & 0xFF).any()) for s in range(6)]
    lv = [s for s in range(6) if used[s]]
    return (lv[0], lv[-1] + 1) if lv else (0, 0)


def bench_exact(torch, mcf, oracle, inputs, steps=20):
    """The exact binary16 product (int8 matrix cores) on the 1024^3 MC x MC operands of
    the binary16 MM-MCN lines, and the exact MC-Linear forward x W^T + b on one layer of
    the MC-Linear workload."""
    out = {}
    cases = []
    for nc in (2, 3):
        A, B = inputs.matmul_normal(1024, 1024, 1024, nc, np.float16, seed=0)
        cases.append((f"matmul_exact_1024_f16_nc{nc}", A, B, nc, True, False))
    x, W, b = next(inputs.linear_inputs(4096, 1024, 1024, 3, np.float16, seed=0))
    cases.append(("linear_exact_4096x1024x1024_f16_nc3", x[None], W, 3, False, True))
    for name, A, B, nc, a_mc, b_trans in cases:
        tA, tB = torch.from_numpy(np.ascontiguousarray(A)).cuda(), torch.from_numpy(B).cuda()
        M, K = A.shape[1:]
        N = B.shape[1] if b_trans else B.shape[2]
        ws = torch.empty(mcf.mc_matmul_exact_workspace(nc, M, N, K), dtype=torch.uint8, device="cuda")
        C = torch.empty((nc, M, N), dtype=torch.float16, device="cuda")
        if b_trans:  # the MC-Linear layer y = x W^T + b (bias added to the exact sum)
            tb = torch.from_numpy(b).cuda()
            run = lambda: mcf.mc_linear_fwd_exact(tA[0], tB, tb, out=C, workspace=ws)
        else:
            run = lambda: mcf.mc_matmul_exact(tA, tB, nc=nc, out=C, workspace=ws)
        warm(torch, run)
        tm = Timer(torch)
        for _ in range(steps):
            tm.run(run)
        us = float(np.median(tm.ms())) * 1e3
        Bm = np.ascontiguousarray(np.swapaxes(B, 1, 2)) if b_trans else B
        la, lb = digit_levels(A), digit_levels(Bm)
        pairs = (la[1] - la[0]) * (lb[1] - lb[0])
        ops = 2.0 * M * N * K * pairs
        Ch = C.cpu().numpy()
        err = exact_error(oracle, A, Bm, Ch, nc, K, np.float16, bias=b if b_trans else None)
        out[name] = {"us": round(us, 1), "MC-GFLOP/s": round(2.0 * M * N * K / (us * 1e-6) / 1e9, 1),
                     "digit_pairs": pairs, "int8_ops": ops,
                     "mfma_int8_frac_whole_call": round(ops / (us * 1e-6) / MFMA_I8_PEAK, 4), "error": err}
        log(f"  {name}: {us:.1f} us ({pairs} digit pairs)")
        del tA, tB, ws, C
    return out


def bench_scaled(torch, mcf, oracle, inputs, steps=5):
    """binary16 with scaled low components (component c stands for 2^(-11 c) times its
    stored value): the 1024^3 MC x MC product at nc = 2 and 3 on the same draws as the
    binary16 lines, and one 4096x1024x1024 MC-Linear layer at nc = 3, each with its
    error against the exact result (the stated tolerance as written)."""
    out = {}
    for nc in (2, 3):
        A, B = inputs.matmul_normal_scaled(1024, 1024, 1024, nc, seed=0)
        tA, tB = torch.from_numpy(A).cuda(), torch.from_numpy(B).cuda()
        C = torch.empty((nc, 1024, 1024), dtype=torch.float16, device="cuda")
        run = lambda: mcf.mc_matmul(tA, tB, nc=nc, out=C, scaled=True)
        warm(torch, run)
        tm = Timer(torch)
        for _ in range(steps):
            tm.run(run)
        ms = float(np.median(tm.ms()))
        Ch = C.cpu().numpy()
        g = np.random.default_rng(5)
        rows, cols = g.integers(0, 1024, 1024), g.integers(0, 1024, 1024)
        err, absab, _ = oracle.matmul_exact_err(oracle.unscale(A), oracle.unscale(B),
                                                oracle.unscale(np.ascontiguousarray(Ch[:, rows, cols])),
                                                rows=rows, cols=cols)
        rel = np.abs(err) / absab
        lit = 4 * 1024 * 2.0 ** (-11 * nc)
        out[f"matmul_1024_f16s_nc{nc}"] = {
            "ms": round(ms, 3), "MC-GFLOP/s": round(2 * 1024 ** 3 / (ms * 1e-3) / 1e9, 1),
            "error": {"sampled_outputs": 1024, "max_rel_err": float(rel.max()), "bound_literal_4Ku^nc": lit,
                      "literal_ratio": float(rel.max() / lit), "literal_holds": bool(rel.max() <= lit),
                      "rms_rel_err": float(np.sqrt(np.mean(rel * rel)))}}
        log(f"  scaled 1024^3 nc={nc}: {ms:.2f} ms, literal ratio {rel.max() / lit:.3g}")
        del tA, tB, C
    x, W, b = next(inputs.linear_inputs_scaled(4096, 1024, 1024, 3, seed=0))
    tx, tW, tb = (torch.from_numpy(v).cuda() for v in (x, W, b))
    y = torch.empty((3, 4096, 1024), dtype=torch.float16, device="cuda")
    run = lambda: mcf.mc_linear_fwd(tx, tW, tb, out=y, scaled=True)
    warm(torch, run)
    tm = Timer(torch)
    for _ in range(steps):
        tm.run(run)
    ms = float(np.median(tm.ms()))
    yh = y.cpu().numpy()
    g = np.random.default_rng(6)
    rows, cols = g.integers(0, 4096, 1024), g.integers(0, 1024, 1024)
    Wt = np.ascontiguousarray(W.transpose(0, 2, 1))
    err, absab, _ = oracle.matmul_exact_err(x[None].astype(np.float64), oracle.unscale(Wt),
                                            oracle.unscale(np.ascontiguousarray(yh[:, rows, cols])),
                                            bias=oracle.unscale(b), rows=rows, cols=cols)
    rel = np.abs(err) / absab
    lit = 4 * 1024 * 2.0 ** -33
    out["linear_4096x1024x1024_f16s_nc3"] = {
        "ms": round(ms, 3), "MC-GFLOP/s": round(2 * 4096 * 1024 * 1024 / (ms * 1e-3) / 1e9, 1),
        "error": {"sampled_outputs": 1024, "max_rel_err": float(rel.max()), "literal_ratio": float(rel.max() / lit),
                  "literal_holds": bool(rel.max() <= lit)}}
    log(f"  scaled MC-Linear layer: {ms:.2f} ms, literal ratio {rel.max() / lit:.3g}")
    return out


def bench_f64(torch, mcf, oracle, inputs, steps=10):
    """binary64 components (the paper's MC float64): 2^26-element Add-MCN, ScalingN,
    Div-MCN and Exp-MCN at nc = 2 (HBM bandwidth; Div-MCN also against the binary64 VALU
    rate), and
    the 1024^3 MC x MC product at nc = 2 (VALU: binary64 adds and FMAs issue at half the
    binary32 rate)."""
    g = np.random.default_rng(0)
    n, nc = 1 << 26, 2
    a = torch.from_numpy(inputs.expansion(g, n, nc, np.float64)).cuda()
    b = torch.from_numpy(inputs.expansion(g, n, nc, np.float64)).cuda()
    d = torch.from_numpy(np.abs(inputs.expansion(g, n, nc, np.float64)) + np.array([[0.5], [0.0]])).cuda()
    v = b[0].contiguous()
    out = torch.empty((nc, n), dtype=torch.float64, device="cuda")
    ops = {"add_mcn": (lambda: mcf.mc_add(a, b, nc=nc, out=out), 48),
           "scaling_n": (lambda: mcf.mc_mul(a, v, nc=nc, y_mc=False, out=out), 40),
           "div_mcn": (lambda: mcf.mc_div(a, d, nc=nc, out=out), 48),
           "exp_mcn": (lambda: mcf.mc_exp(a, nc=nc, out=out), 32)}
    res = {}
    for name, (fn, bpe) in ops.items():
        warm(torch, fn)
        tm = Timer(torch)
        for _ in range(steps):
            tm.run(fn)
        ms = float(np.median(tm.ms()))
        gbs = bpe * n / (ms * 1e-3) / 1e9
        res[name] = {"us": round(ms * 1e3, 1), "GB/s": round(gbs, 1), "hbm_frac": round(gbs * 1e9 / HBM_PEAK, 3)}
        if name == "div_mcn":
            fops = ew_fp_ops("div", nc)
            res[name]["valu_frac_f64"] = round(fops * n / (ms * 1e-3) / (VALU_PEAK / 2), 3)
        log(f"  f64 {name}: {ms * 1e3:.1f} us, {gbs:.0f} GB/s")
    del a, b, d, v, out
    A = inputs.expansion(g, (1024, 1024), nc, np.float64, 1 / 32)
    B = inputs.expansion(g, (1024, 1024), nc, np.float64, 1 / 32)
    C, _, kms = bench_matmul(torch, mcf, A, B, nc, 10, 3, warm_s=0.2)
    macs = 1024 ** 3
    res["matmul_1024_nc2"] = {
        "ms": round(kms, 3), "MC-GFLOP/s": round(2 * macs / (kms * 1e-3) / 1e9, 1),
        "valu_frac_f64": round(algo_ops_per_mac(nc, True) * macs / (kms * 1e-3) / (VALU_PEAK / 2), 3),
        "error": exact_error(oracle, A, B, C.cpu().numpy(), nc, 1024, np.float64)}
    log(f"  f64 1024^3 nc=2: {kms:.2f} ms")
    return {"workload": "binary64 components: 2^26 elements nc = 2; 1024^3 MC x MC nc = 2", "ops": res}


def bench_linreg(torch, mcf, inputs, steps=3000):
    """The paper's linear-regression precision experiment (Section 2.4): X 10000 x 2
    ~ N(-0.5, 0.5^2), y = X W*^T, gradient descent with lr = 0.05 on an MC-Linear layer
    without bias (mc_linreg_gd_step, one call per step).  Reports the time per step and
    the mean-squared error before the first and after the last step, beside plain
    float64 gradient descent on the same data (context, like the paper's float64 row)."""
    n, d, lr = 10000, 2, 0.05
    out = {}
    for dt, nc in ((np.float16, 1), (np.float16, 2), (np.float16, 3), (np.float32, 1), (np.float32, 2)):
        X, y_neg, W0, _ = inputs.linreg_inputs(n, d, nc, dt, seed=0)
        tX, ty, tW = (torch.from_numpy(np.ascontiguousarray(a)).cuda() for a in (X, y_neg, W0))
        loss = torch.empty(nc, dtype=tW.dtype, device="cuda")
        ws = torch.empty(mcf.mc_linreg_workspace(0 if dt == np.float16 else 1, nc, n, d), dtype=torch.uint8,
                         device="cuda")
        mcf.mc_linreg_gd_step(tX, ty, tW, lr, loss=loss, workspace=ws)
        torch.cuda.synchronize()
        first = float(loss.double().sum())
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s.record()
        for _ in range(steps - 1):
            mcf.mc_linreg_gd_step(tX, ty, tW, lr, loss=loss, workspace=ws)
        e.record()
        torch.cuda.synchronize()
        us = s.elapsed_time(e) * 1e3 / (steps - 1)
        name = f"{'f16' if dt == np.float16 else 'f32'}_nc{nc}"
        # the same steps replayed from a HIP graph of 100 captured steps (the loop is
        # launch-bound: five kernels per step), checked bit for bit against the eager run
        tWg = torch.from_numpy(np.ascontiguousarray(W0)).cuda()
        lossg, wsg = torch.empty_like(loss), torch.empty_like(ws)
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            for _ in range(100):
                mcf.mc_linreg_gd_step(tX, ty, tWg, lr, loss=lossg, workspace=wsg)
        torch.cuda.synchronize()
        sg, eg = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        sg.record()
        for _ in range(steps // 100):
            graph.replay()
        eg.record()
        torch.cuda.synchronize()
        us_graph = sg.elapsed_time(eg) * 1e3 / (steps // 100 * 100)
        same = bool(torch.equal(tWg.view(torch.int16 if dt == np.float16 else torch.int32),
                                tW.view(torch.int16 if dt == np.float16 else torch.int32)))
        del graph
        # the same loss in float64 from the final weights (a binary16 MC loss underflows
        # to 0 below the smallest subnormal, 2^-24)
        w = tW.double().sum(dim=0).cpu().numpy()
        r64 = X.astype(np.float64) @ w + y_neg.astype(np.float64)
        out[name] = {"us_per_step": round(us, 2), "us_per_step_graph": round(us_graph, 2),
                     "graph_matches_eager": same, "loss_first": first, "loss_last": float(loss.double().sum()),
                     "loss_last_float64": float(np.mean(r64 * r64))}
        log(f"  linreg {name}: {us:.1f} us/step ({us_graph:.1f} from a graph, same bits: {same}), "
            f"loss {first:.3g} -> {out[name]['loss_last']:.3g} (float64 {out[name]['loss_last_float64']:.3g})")
    # float64 gradient descent on the binary32 data, for context
    X, y_neg, W0, _ = inputs.linreg_inputs(n, d, 1, np.float32, seed=0)
    X64, y64, w = X.astype(np.float64), -y_neg.astype(np.float64), W0[0].astype(np.float64)
    for _ in range(steps):
        r = X64 @ w - y64
        w = w - lr * (2.0 / n) * (X64.T @ r)
    r = X64 @ w - y64
    out["float64_reference_loss_last"] = float(np.mean(r * r))
    out["workload"] = (f"n = {n}, d = {d}, lr = {lr}, {steps} steps; one mc_linreg_gd_step call per step, "
                       f"eager and replayed from a HIP graph of 100 captured steps")
    return out


def issue_probe(blocks=2048, iters=20000):
    """VALU issue rates per instruction kind (the probe library: 8 independent chains
    per lane, 8 wavefronts per SIMD on every CU), printed as one JSON line: lane-
    instructions per second, per clock per CU at the clock the wavefronts measured,
    and relative to v_add_f32.  This is the evidence for the VALU peak of
    128 lane-operations per clock per CU used by the roofline."""
    import ctypes

    path = os.path.join(ROOT, "paper_2207_08867_amd", "libmcf_probe.so")
    if not os.path.exists(path):
        raise SystemExit(f"{path} is missing: build it with python -m paper_2207_08867_amd.build")
    L = ctypes.CDLL(path)
    L.mcf_probe_count.restype = ctypes.c_int
    L.mcf_probe_name.restype = ctypes.c_char_p
    L.mcf_probe_name.argtypes = [ctypes.c_int]
    L.mcf_probe_issue.restype = ctypes.c_int
    d = ctypes.c_double
    L.mcf_probe_issue.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.POINTER(d), ctypes.POINTER(d),
                                  ctypes.POINTER(d)]
    res = {}
    base = None
    for op in range(L.mcf_probe_count()):
        name = L.mcf_probe_name(op).decode()
        ms, li, ghz = d(), d(), d()
        st = L.mcf_probe_issue(op, blocks, iters, ctypes.byref(ms), ctypes.byref(li), ctypes.byref(ghz))
        if st != 0:
            raise SystemExit(f"issue probe {name}: HIP error {st}")
        rate = li.value / (ms.value * 1e-3)
        per_clk = rate / 256 / (ghz.value * 1e9)
        base = base or per_clk
        res[name] = {"ms": round(ms.value, 3), "T_lane_instr_per_s": round(rate / 1e12, 2),
                     "clock_GHz": round(ghz.value, 3), "per_clk_per_CU": round(per_clk, 1),
                     "vs_v_add_f32": round(per_clk / base, 3)}
        log(f"  {name:32s} {ms.value:8.2f} ms  {rate / 1e12:6.2f} T/s  {per_clk:6.1f} per clk per CU "
            f"at {ghz.value:.2f} GHz")
    print(json.dumps({"issue_probe": res, "blocks": blocks, "lanes_per_block": 256, "iters": iters,
                      "chains_per_lane": 8, "unroll": 16}), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--no-extra", action="store_true", help="only the headline workload")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--only", default="",
                    help="comma-separated groups of extra workloads to run (pruned, small, linear, exact, linreg, "
                         "scaled, f64, elementwise, splitk, batched, cpu_oracle); default: all")
    ap.add_argument("--copy-probe", action="store_true",
                    help="also run one 1 GiB device-to-device copy (reference for HBM byte counters)")
    ap.add_argument("--issue-probe", action="store_true",
                    help="only run the VALU issue-rate probe (libmcf_probe.so) and print its rates")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py: this library runs on one GPU only; the MC product shards by output blocks "
              "with no communication, so there is no multi-GPU path to measure", file=sys.stderr)
        sys.exit(2)

    if args.issue_probe:
        issue_probe()
        return

    import torch

    import oracle
    import paper_2207_08867_amd as mcf
    from paper_2207_08867_amd import inputs

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    mcf.lib()

    if args.copy_probe:
        src = torch.empty(1 << 28, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    M = N = K = 8192
    nc = 3
    log("generating 8192^3 binary32 nc=3 operands")
    A, B = inputs.matmul_normal(M, N, K, nc, np.float32, seed=0)
    log("headline product")
    C, ms_step, kms = bench_matmul(torch, mcf, A, B, nc, args.steps, args.warmup)
    value = 2.0 * M * N * K / (ms_step * 1e-3) / 1e9
    ops = algo_ops_per_mac(nc, True) * M * N * K
    achieved = ops / (kms * 1e-3) / 1e12
    log(f"  {ms_step:.1f} ms/step, kernel {kms:.1f} ms, {value:.1f} MC-GFLOP/s, {achieved:.2f} TOP/s")
    Ch = C.cpu().numpy()
    del C
    err = exact_error(oracle, A, B, Ch, nc, K, np.float32)
    log(f"  max rel err vs exact {err['max_rel_err']:.3g} (bound {err['bound_literal_4Ku^nc']:.3g})")

    line = {
        "metric": "MC-matmul MC-GFLOP/s (binary32, nc=3, MC x MC)",
        "value": round(value, 2),
        "unit": "MC-GFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": "MC matmul C = A B, M = N = K = 8192, binary32 components, nc = 3, A and B MC, "
                               "entries float64 ~ N(0, 1/K) seed 0 split by successive rounding",
                   "M": M, "N": N, "K": K, "nc": nc, "component": "binary32"},
        "roofline": {"bound": "alu", "achieved": round(achieved, 3), "peak": round(VALU_PEAK / 1e12, 2),
                     "unit": "TOP/s", "frac": round(achieved * 1e12 / VALU_PEAK, 4), "traffic": measured_traffic(),
                     "kernel": "mm_kernel (MC x MC, binary32, nc = 3)", "kernel_ms": round(kms, 3),
                     "ops_per_mac": algo_ops_per_mac(nc, True),
                     **issue_fields("matmul_8192_f32_nc3", kms * 1e-3, M * N * K)},
        "error": err,
    }
    groups = [g for g in args.only.split(",") if g]
    want = lambda name: not groups or name in groups
    if not args.no_extra:
        extra = {}
    if not args.no_extra and want("pruned"):
        log("pruned MC x MC product on the headline operands")
        tA, tB = torch.from_numpy(A).cuda(), torch.from_numpy(B).cuda()
        Cp = torch.empty((nc, M, N), dtype=torch.float32, device="cuda")
        mcf.mc_matmul_pruned(tA, tB, nc=nc, out=Cp)
        torch.cuda.synchronize()
        tm = Timer(torch)
        for _ in range(args.steps):
            tm.run(lambda: mcf.mc_matmul_pruned(tA, tB, nc=nc, out=Cp))
        pms = float(np.mean(tm.ms()))
        Cph = Cp.cpu().numpy()
        del tA, tB, Cp
        extra["matmul_pruned_8192_f32_nc3"] = {
            "ms": round(pms, 3), "MC-GFLOP/s": round(2.0 * M * N * K / (pms * 1e-3) / 1e9, 2),
            "ops_per_mac": pruned_ops_per_mac(nc),
            "valu_frac": round(pruned_ops_per_mac(nc) * M * N * K / (pms * 1e-3) / VALU_PEAK, 4),
            "error": exact_error(oracle, A, B, Cph, nc, K, np.float32)}
        log(f"  pruned: {pms:.1f} ms")
        del Cph
    if not args.no_extra and want("small"):
        A1, B1 = inputs.matmul_uniform(64, 64, 64, 2, np.float32, seed=0)
        C1, ms1, k1 = bench_matmul(torch, mcf, A1, B1, 2, 20, 3, warm_s=0.2)
        extra["matmul_64_f32_nc2"] = {"us": round(k1 * 1e3, 1),
                                      "error": exact_error(oracle, A1, B1, C1.cpu().numpy(), 2, 64, np.float32,
                                                           count=4096)}
        for nc3 in (2, 3):
            A3, B3 = inputs.matmul_normal(1024, 1024, 1024, nc3, np.float16, seed=0)
            C3, ms3, k3 = bench_matmul(torch, mcf, A3, B3, nc3, 10, 3, warm_s=0.2)
            macs = 1024 ** 3
            extra[f"matmul_1024_f16_nc{nc3}"] = {
                "ms": round(k3, 3), "MC-GFLOP/s": round(2 * macs / (k3 * 1e-3) / 1e9, 1),
                "valu_frac_printed_ops": round(algo_ops_per_mac(nc3, True) * macs / (k3 * 1e-3) / VALU_PEAK, 3),
                **issue_fields(f"matmul_1024_f16_nc{nc3}", k3 * 1e-3, macs),
                "error": exact_error(oracle, A3, B3, C3.cpu().numpy(), nc3, 1024, np.float16, count=1024)}
            log(f"  1024^3 f16 nc={nc3}: {k3:.2f} ms")
    if not args.no_extra and want("linear"):
        log("MC-Linear")
        extra["linear_4096x1024x1024_f16_nc3"] = bench_linear(torch, mcf, oracle, inputs)
    if not args.no_extra and want("exact"):
        log("exact binary16 products (int8 matrix cores)")
        extra["exact"] = bench_exact(torch, mcf, oracle, inputs)
    if not args.no_extra and want("linreg"):
        log("linear-regression gradient descent")
        extra["linreg"] = bench_linreg(torch, mcf, inputs)
    if not args.no_extra and want("scaled"):
        log("binary16 with scaled low components")
        extra["scaled"] = bench_scaled(torch, mcf, oracle, inputs)
    if not args.no_extra and want("f64"):
        log("binary64 components")
        extra["f64"] = bench_f64(torch, mcf, oracle, inputs)
    if not args.no_extra and want("elementwise"):
        log("elementwise")
        extra["elementwise"] = bench_elementwise(torch, mcf, inputs)
    if not args.no_extra and want("splitk"):
        log("K-split products")
        extra["splitk"] = bench_splitk(torch, mcf, inputs)
    if not args.no_extra and want("batched"):
        log("batched products and AddMM")
        extra["batched"] = bench_batched(torch, mcf, inputs)
    if not args.no_extra and want("cpu_oracle") and not args.no_cpu:
        log("CPU oracle on the other workloads (bounded samples)")
        extra["cpu_oracle"] = cpu_oracle_other(oracle, inputs)
    if not args.no_extra:
        line["extra"] = extra
    if not args.no_cpu:
        log("cpu baseline (oracle)")
        line["cpu_baseline"] = cpu_baseline(oracle, A, B, nc)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
