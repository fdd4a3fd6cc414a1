#!/usr/bin/env python3
"""Benchmark of Y = X W^T + R (bf16, fp32 accumulation) on one MI355X.

Workload: the 16-shape sweep M in {1, 64, 512, 4096} x hidden in {2048, 4096,
5120, 8192} (N = K = hidden), residual on, seeds 0-15 -- synthetic stand-ins
for the paper's 16-shape attention-output-projection task.  One step = one
call of the library per shape.

Cold operands: every shape holds enough copies of (X, W, R, Y) to span at
least 1 GiB (4x the 256 MB Infinity Cache) and the calls cycle through them,
so each call reads operands that were last touched a full GiB of traffic
earlier -- they come from HBM.  Timing: the calls over all copies are
captured once in a HIP graph; each timed step replays it between two HIP
events on the capture stream, and per-call time = elapsed / copies (this
keeps host submission cost out of 1-20 us kernels).  The per-shape time is
the median over the timed steps.

Printed JSON line (stdout, last line):
  value     geometric mean over the 16 shapes of TFLOP/s = 2MNK / t
  roofline  the kernel variant with the most time in a step: algorithmic
            FLOPs (MFMA-bound) or bytes (HBM-bound) of its launches divided
            by their summed durations, against the MI355X peak
  cpu_baseline  the CPU oracle (fp64, OpenMP) on a time-bounded row sample
            of the same 16 shapes, same aggregation
Per-shape rows, the geometric mean of per-shape roofline fractions, the
three single-shape gates (decode M=16, prefill 4096^3, square 8192^3 plain),
the general form (alpha, beta, bias, row strides), SwiGLU (the decoder
layer's gate/up projections with the SiLU-multiply fused) and the INT8 forms
(W8A8 with dequantisation, INT8 SwiGLU; against the int8 MFMA peak) on
decoder-layer shapes, and the grouped mixture-of-experts projections are
extra fields of the same line.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2516.6          # 256 CU x 4096 FLOP/clk x 2.4 GHz, dense
PEAK_I8_TOPS = 5033.2              # 256 CU x 8192 OP/clk x 2.4 GHz, dense (int8 and fp8)
PEAK_HBM_GBPS = 8000.0
ROTATE_BYTES = 1 << 30
MAX_COPIES = 256
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def mfma_peak(w):
    """Dense MFMA peak (T op/s) of the workload's operand type."""
    return PEAK_I8_TOPS if getattr(w, "eight_bit", False) else PEAK_BF16_TFLOPS


def roofline_time(w):
    return max(w.flops / (mfma_peak(w) * 1e12), w.algorithmic_bytes / (PEAK_HBM_GBPS * 1e9))


def bound_of(w):
    return "mfma" if w.flops / (mfma_peak(w) * 1e12) >= w.algorithmic_bytes / (PEAK_HBM_GBPS * 1e9) else "hbm"


def geomean(xs):
    return math.exp(sum(math.log(x) for x in xs) / len(xs))


def source_digest(paths):
    h = hashlib.sha256()
    for p in paths:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


# Kernel symbol fragment and threads per workgroup of each 256x256 tile plan
# (rocprofv3 reports symbols).
# Cfg<BM, BN, BK, WAVES_M, WAVES_N, STAGES, WAVES_PER_EU, LAG, M16, AACC>.
PLAN_SYMBOL = {
    "tile_256x256_k64_w8": ("Cfg<256, 256, 64, 2, 4, 2, 2, false, false, false>", 512),
    "tile_256x256_k64_w4_m16a": ("Cfg<256, 256, 64, 2, 2, 2, 1, false, true, true>", 256),
}
# The plan whose HBM traffic the counter runs summarise (the big sweep shapes' plan).
TRAFFIC_PLAN = "tile_256x256_k64_w4_m16a"
KERNEL_SOURCES = ["paper_2608_17071_amd/csrc/tile_kernel.h", "paper_2608_17071_amd/csrc/kernel_tile.hip",
                  "paper_2608_17071_amd/csrc/internal.h"]


def summarize_traffic(pmc_dir, plan, shapes, command):
    """profiles/traffic.json from four rocprofv3 --pmc runs under pmc_dir:
    fetch/ and write/ (FETCH_SIZE, WRITE_SIZE of `bench.py --only <shapes>`),
    copy_fetch/ and copy_write/ (the same counters of --copy-calibration)."""
    import csv
    from paper_2608_17071_amd import workloads as wl

    def per_grid(sub, counter, needle):
        out = {}
        with open(os.path.join(pmc_dir, sub, "p_counter_collection.csv")) as f:
            for r in csv.DictReader(f):
                if r["Counter_Name"] == counter and needle in r["Kernel_Name"]:
                    out.setdefault(int(r["Grid_Size"]), []).append(float(r["Counter_Value"]))
        return {g: sum(v) / len(v) for g, v in out.items()}

    copy_bytes = 1 << 28
    cf = per_grid("copy_fetch", "FETCH_SIZE", "copyBuffer")
    cw = per_grid("copy_write", "WRITE_SIZE", "copyBuffer")
    fetch_scale = copy_bytes / (1024 * max(cf.values()))
    write_scale = copy_bytes / (1024 * max(cw.values()))
    sym, threads = PLAN_SYMBOL[plan]     # a 256x256 tile
    fetch = per_grid("fetch", "FETCH_SIZE", sym)
    write = per_grid("write", "WRITE_SIZE", sym)
    rows, total = [], 0.0
    for name in shapes:
        w = wl.BY_NAME[name]
        # the shapes of one run have distinct grids (work-items = output
        # tiles x threads per workgroup, no split-K for this plan)
        g = -(-w.M // 256) * -(-w.N // 256) * threads
        b = fetch[g] * 1024 * fetch_scale + write[g] * 1024 * write_scale
        total += b
        rows.append({"shape": name, "fetch_kib": fetch[g], "write_kib": write[g], "hbm_bytes": b,
                     "algorithmic_bytes": w.algorithmic_bytes})
    rec = {"kernels": {plan: {
        "bytes_per_launch": total / len(shapes), "shapes": rows,
        "fetch_scale": fetch_scale, "write_scale": write_scale,
        "sources": KERNEL_SOURCES, "source_sha256": source_digest(KERNEL_SOURCES),
        "command": command}}}
    os.makedirs(os.path.dirname(TRAFFIC_FILE), exist_ok=True)
    with open(TRAFFIC_FILE, "w") as f:
        json.dump(rec, f, indent=1)
    print(json.dumps(rec, indent=1))


def measured_traffic(plan_name):
    """HBM bytes per launch from a committed counter summary, if it is current."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    with open(TRAFFIC_FILE) as f:
        rec = json.load(f)
    entry = rec.get("kernels", {}).get(plan_name)
    if not entry:
        return None
    if entry.get("source_sha256") != source_digest(entry.get("sources", [])):
        return None        # kernel changed since the counters were taken
    return entry.get("bytes_per_launch")


class Case:
    def __init__(self, w, ka, torch, rotate=True, plan=None):
        from paper_2608_17071_amd import workloads as wl
        t = wl.make_inputs(w)
        self.w = w
        self.host = t
        x, W = t["X"].cuda(), t["W"].cuda()
        r = t["R"].cuda() if w.residual else None
        set_bytes = w.algorithmic_bytes
        n = 1
        if rotate:
            n = max(2, min(MAX_COPIES, -(-ROTATE_BYTES // set_bytes)))
        self.sets = []
        for i in range(n):
            self.sets.append((x if i == 0 else x.clone(), W if i == 0 else W.clone(),
                              None if r is None else (r if i == 0 else r.clone()),
                              torch.empty(w.M, w.N, dtype=torch.bfloat16, device="cuda")))
        self.force(ka, plan)

    def force(self, ka, plan):
        """Run `plan` (an id) from now on; None: the library's own choice."""
        self.forced = plan
        self.plan = ka.select_plan(self.w.M, self.w.N, self.w.K, self.w.residual) if plan is None else plan
        self.plan_name = ka.plan_name(self.plan)
        self.times = []
        self.graph = None

    def call(self, ka, i):
        x, W, r, y = self.sets[i]
        if self.forced is not None:
            ka.gemm_bf16_with_plan(self.forced, x, W, r, out=y)
        elif r is not None:
            ka.gemm_bf16_residual(x, W, r, out=y)
        else:
            ka.gemm_bf16(x, W, out=y)

    def call_all(self, ka):
        for i in range(len(self.sets)):
            self.call(ka, i)

    def free(self):
        self.sets = []
        self.graph = None


class BlasCase(Case):
    """The same workload through torch's GEMM (hipBLASLt on ROCm), for
    comparison only: identical inputs, operand copies and timing protocol."""

    def __init__(self, w, ka, torch, rotate=True):
        super().__init__(w, ka, torch, rotate)
        self.forced, self.plan, self.plan_name = None, -1, "torch(hipBLASLt)"
        self.torch = torch

    def call(self, ka, i):
        x, W, r, y = self.sets[i]
        if r is not None:
            self.torch.addmm(r, x, W.t(), out=y)
        else:
            self.torch.mm(x, W.t(), out=y)


class GeneralCase(Case):
    """A general-form workload: X read through its row stride, C, bias, alpha, beta."""

    def __init__(self, w, ka, torch, rotate=True, plan=None):
        from paper_2608_17071_amd import workloads as wl
        t = wl.make_general_inputs(w)
        self.w = w
        self.host = t
        xbuf = torch.zeros((w.M, w.ldx), dtype=torch.bfloat16, device="cuda")
        xbuf[:, :w.K] = t["X"].cuda()
        W = t["W"].cuda()
        c = t["C"].cuda() if t["C"] is not None else None
        b = t["bias"].cuda() if t["bias"] is not None else None
        n = 1
        if rotate:
            n = max(2, min(MAX_COPIES, -(-ROTATE_BYTES // w.algorithmic_bytes)))
        self.sets = []
        for i in range(n):
            xb = xbuf if i == 0 else xbuf.clone()
            self.sets.append((xb[:, :w.K], W if i == 0 else W.clone(),
                              None if c is None else (c if i == 0 else c.clone()),
                              torch.empty(w.M, w.N, dtype=torch.bfloat16, device="cuda"), b))
        self.forced = plan
        self.plan = ka.select_plan_ex(w.M, w.N, w.K, w.has_c, w.ldx, w.K, w.N, w.N, w.alpha, w.beta,
                                      w.has_bias) if plan is None else plan
        self.plan_name = ka.plan_name(self.plan)
        self.times = []
        self.graph = None

    def call(self, ka, i):
        x, W, c, y, b = self.sets[i]
        ka.gemm_bf16_ex(x, W, c, b, self.w.alpha, self.w.beta, out=y, plan=self.forced)


class GluCase(Case):
    """A SwiGLU workload: H = silu(X Wg^T) * (X Wu^T)."""

    def __init__(self, w, ka, torch, rotate=True, plan=None):
        from paper_2608_17071_amd import workloads as wl
        t = wl.make_glu_inputs(w)
        self.w = w
        self.host = t
        x, g, u = t["X"].cuda(), t["Wg"].cuda(), t["Wu"].cuda()
        n = 1
        if rotate:
            n = max(2, min(MAX_COPIES, -(-ROTATE_BYTES // w.algorithmic_bytes)))
        self.sets = []
        for i in range(n):
            self.sets.append((x if i == 0 else x.clone(), g if i == 0 else g.clone(), u if i == 0 else u.clone(),
                              torch.empty(w.M, w.N, dtype=torch.bfloat16, device="cuda")))
        self.forced = plan
        self.plan = ka.select_plan_swiglu(w.M, w.N, w.K) if plan is None else plan
        self.plan_name = ka.plan_name(self.plan)
        self.times = []
        self.graph = None

    def call(self, ka, i):
        x, g, u, h = self.sets[i]
        ka.swiglu_bf16(x, g, u, out=h, plan=self.forced)


class I8Case(Case):
    """An INT8 workload (W8A8 linear with dequantisation, or INT8 SwiGLU)."""

    def __init__(self, w, ka, torch, rotate=True, plan=None):
        from paper_2608_17071_amd import workloads as wl
        t = wl.make_i8_inputs(w)
        self.w = w
        self.host = t
        dev = {k: (v.cuda() if v is not None else None) for k, v in t.items()}
        n = 1
        if rotate:
            n = max(2, min(MAX_COPIES, -(-ROTATE_BYTES // w.algorithmic_bytes)))
        self.sets = []
        for i in range(n):
            d = {k: (v if (i == 0 or v is None) else v.clone()) for k, v in dev.items()}
            d["Y"] = torch.empty(w.M, w.N, dtype=torch.bfloat16, device="cuda")
            self.sets.append(d)
        self.forced = plan
        select = ka.select_plan_i8 if w.fmt == "i8" else ka.select_plan_f8
        self.plan = select(w.M, w.N, w.K, w.swiglu) if plan is None else plan
        self.plan_name = ka.plan_name(self.plan)
        self.times = []
        self.graph = None

    def call(self, ka, i):
        d = self.sets[i]
        f8 = self.w.fmt == "f8"
        if self.w.swiglu:
            (ka.swiglu_f8 if f8 else ka.swiglu_i8)(d["qX"], d["sx"], d["qW"], d["sw"], d["qWu"], d["swu"], out=d["Y"],
                                                   plan=self.forced)
        else:
            (ka.gemm_f8 if f8 else ka.gemm_i8)(d["qX"], d["sx"], d["qW"], d["sw"], d["R"], out=d["Y"],
                                               plan=self.forced)


class GroupedCase(Case):
    """A grouped (per-expert) workload over an expert-major padded layout."""

    def __init__(self, w, ka, torch, rotate=True, plan=None):
        from paper_2608_17071_amd import workloads as wl
        t = wl.make_grouped_inputs(w, device="cuda")
        self.w = w
        self.host = t          # device tensors; the CPU baseline copies the experts it samples
        self.Mpad = t["Mpad"]
        dev = {k: t[k] for k in ("X", "W", "Wu", "counts") if k in t}
        n = 1
        if rotate:
            n = max(2, min(MAX_COPIES, -(-ROTATE_BYTES // w.algorithmic_bytes)))
        self.sets = []
        for i in range(n):
            d = {k: (v if i == 0 else v.clone()) for k, v in dev.items()}
            d["Y"] = torch.empty((w.G, self.Mpad, w.N), dtype=torch.bfloat16, device="cuda")
            self.sets.append(d)
        self.forced = plan
        self.plan = ka.select_plan_grouped(w.G, self.Mpad, w.N, w.K, w.swiglu) if plan is None else plan
        self.plan_name = ka.plan_name(self.plan)
        self.times = []
        self.graph = None

    def call(self, ka, i):
        d = self.sets[i]
        if self.w.swiglu:
            ka.swiglu_bf16_grouped(d["X"], d["W"], d["Wu"], d["counts"], out=d["Y"], plan=self.forced)
        else:
            ka.gemm_bf16_grouped(d["X"], d["W"], d["counts"], out=d["Y"], plan=self.forced)


def cpu_baseline_grouped(cases, seconds):
    """The oracle's grouped forms on whole experts 0, 1, ... of each case until
    its time share is used."""
    import numpy as np
    import oracle
    from paper_2608_17071_amd import workloads as wl

    orc = oracle.default()
    per_shape = seconds / len(cases)
    rates, done = [], []
    for c in cases:
        w, h = c.w, c.host
        E = min(w.G, 16)              # the sample never reaches further; only these are copied
        xb, wb = wl.bits(h["X"][:E].cpu()), wl.bits(h["W"][:E].cpu())
        ub = wl.bits(h["Wu"][:E].cpu()) if w.swiglu else None
        cnt = h["counts"][:E].cpu().numpy()
        ops, e, t0 = 0, 0, time.perf_counter()
        while e < E:
            r = int(cnt[e])
            if r:
                gi = np.full(r * w.N, e, dtype=np.int64)
                ri = np.repeat(np.arange(r, dtype=np.int64), w.N)
                ci = np.tile(np.arange(w.N, dtype=np.int64), r)
                orc.grouped_at(xb, wb, ub, cnt, gi, ri, ci)
                ops += (4 if w.swiglu else 2) * r * w.N * w.K
            e += 1
            if time.perf_counter() - t0 >= per_shape:
                break
        rates.append(ops / (time.perf_counter() - t0) / 1e12)
        done.append(e)
    return {
        "value": geomean(rates), "unit": "TFLOP/s (fp64 oracle, grouped forms, geomean over its shapes)",
        "cores": orc.threads(), "kind": "oracle",
        "sample": f"every valid row of experts 0..e-1 of each grouped shape, e = {done} (about {per_shape:.2f} s each)",
    }


def cpu_baseline_i8(cases, seconds):
    """The oracle's INT8 / FP8 forms on rows 0, 1, ... of each case until its time share is used."""
    import numpy as np
    import torch
    import oracle
    from paper_2608_17071_amd import workloads as wl

    orc = oracle.default()
    per_shape = seconds / len(cases)
    rates, rows_done = [], []
    for c in cases:
        w, h = c.w, c.host
        f8 = w.fmt == "f8"

        def raw(t):
            return t.view(torch.uint8).numpy() if f8 else t.numpy()

        qx, sx, qw, sw = raw(h["qX"]), h["sx"].numpy(), raw(h["qW"]), h["sw"].numpy()
        rb = wl.bits(h["R"]) if h["R"] is not None else None
        cols = np.arange(w.N, dtype=np.int64)
        ops, rows, t0 = 0, 0, time.perf_counter()
        while rows < w.M:
            r = np.full(w.N, rows, dtype=np.int64)
            if w.swiglu:
                (orc.f8_swiglu_at if f8 else orc.i8_swiglu_at)(qx, sx, qw, sw, raw(h["qWu"]), h["swu"].numpy(), r,
                                                                cols)
            else:
                (orc.f8_linear_at if f8 else orc.i8_linear_at)(qx, sx, qw, sw, rb, r, cols)
            rows += 1
            ops += (4 if w.swiglu else 2) * w.N * w.K
            if time.perf_counter() - t0 >= per_shape:
                break
        rates.append(ops / (time.perf_counter() - t0) / 1e12)
        rows_done.append(rows)
    return {
        "value": geomean(rates), "unit": "T op/s (oracle: exact int64 sums, fp64 dequantisation; geomean)",
        "cores": orc.threads(), "kind": "oracle",
        "sample": f"whole output rows 0..r-1 of each INT8 shape, r = {rows_done} (about {per_shape:.2f} s each)",
    }


def cpu_baseline_glu(cases, seconds):
    """The oracle's SwiGLU on rows 0, 1, ... of each case until its time share is used."""
    import numpy as np
    import oracle
    from paper_2608_17071_amd import workloads as wl

    orc = oracle.default()
    per_shape = seconds / len(cases)
    rates, rows_done = [], []
    for c in cases:
        w, h = c.w, c.host
        xb, gb, ub = wl.bits(h["X"]), wl.bits(h["Wg"]), wl.bits(h["Wu"])
        cols = np.arange(w.N, dtype=np.int64)
        flops, rows, t0 = 0, 0, time.perf_counter()
        while rows < w.M:
            orc.swiglu_at(xb, gb, ub, np.full(w.N, rows, dtype=np.int64), cols)
            rows += 1
            flops += 4 * w.N * w.K
            if time.perf_counter() - t0 >= per_shape:
                break
        rates.append(flops / (time.perf_counter() - t0) / 1e12)
        rows_done.append(rows)
    return {
        "value": geomean(rates), "unit": "TFLOP/s (fp64 oracle, SwiGLU, geomean over its shapes)",
        "cores": orc.threads(), "kind": "oracle",
        "sample": f"whole output rows 0..r-1 of each SwiGLU shape, r = {rows_done} (about {per_shape:.2f} s each)",
    }


def cpu_baseline_general(cases, seconds):
    """The oracle's general form on rows 0, 1, ... of each case until its time share is used."""
    import numpy as np
    import oracle
    from paper_2608_17071_amd import workloads as wl

    orc = oracle.default()
    per_shape = seconds / len(cases)
    rates, rows_done = [], []
    for c in cases:
        w, h = c.w, c.host
        xb, wb = wl.bits(h["X"]), wl.bits(h["W"])
        cb = wl.bits(h["C"]) if h["C"] is not None else None
        bb = wl.bits(h["bias"]) if h["bias"] is not None else None
        cols = np.arange(w.N, dtype=np.int64)
        flops, rows, t0 = 0, 0, time.perf_counter()
        while rows < w.M:
            orc.linear_ex_at(xb, wb, cb, bb, w.alpha, w.beta, np.full(w.N, rows, dtype=np.int64), cols)
            rows += 1
            flops += 2 * w.N * w.K
            if time.perf_counter() - t0 >= per_shape:
                break
        rates.append(flops / (time.perf_counter() - t0) / 1e12)
        rows_done.append(rows)
    return {
        "value": geomean(rates), "unit": "TFLOP/s (fp64 oracle, general form, geomean over its shapes)",
        "cores": orc.threads(), "kind": "oracle",
        "sample": f"whole output rows 0..r-1 of each general-form shape, r = {rows_done} (about {per_shape:.2f} s each)",
    }


def time_cases(cases, steps, warmup, ka, torch, use_graph=True):
    """Warm up, capture, then time `steps` passes over all cases; returns wall seconds."""
    for c in cases:
        for _ in range(max(1, warmup)):
            c.call_all(ka)       # also allocates any split-K workspace before capture
    torch.cuda.synchronize()
    if use_graph:
        for c in cases:
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                c.call_all(ka)
            c.graph = g
        for c in cases:
            for _ in range(max(1, warmup)):
                c.graph.replay()
        torch.cuda.synchronize()
    t0 = time.perf_counter()
    events = []
    for _ in range(steps):
        for c in cases:
            a = torch.cuda.Event(enable_timing=True)
            b = torch.cuda.Event(enable_timing=True)
            a.record()
            if use_graph:
                c.graph.replay()
            else:
                c.call_all(ka)
            b.record()
            events.append((c, a, b))
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    for c, a, b in events:
        c.times.append(a.elapsed_time(b) * 1e-3 / len(c.sets))
    return wall


def median(xs):
    s = sorted(xs)
    n = len(s)
    return s[n // 2] if n % 2 else 0.5 * (s[n // 2 - 1] + s[n // 2])


def shape_row(c):
    w = c.w
    t = median(c.times)
    extra = {}
    if hasattr(w, "alpha"):
        extra = {"alpha": w.alpha, "beta": w.beta, "C": w.has_c, "bias": w.has_bias, "ldx": w.ldx}
    return {
        "shape": w.name, "M": w.M, "N": w.N, "K": w.K, **extra, "plan": c.plan_name,
        "us": round(t * 1e6, 3), "tflops": round(w.flops / t / 1e12, 3),
        "gbps": round(w.algorithmic_bytes / t / 1e9, 1), "bound": bound_of(w),
        "roofline_frac": round(roofline_time(w) / t, 4),
    }


def cpu_baseline(cases, seconds):
    """The oracle on rows 0, 1, 2, ... of every shape until its time share is used."""
    import numpy as np
    import oracle
    from paper_2608_17071_amd import workloads as wl

    orc = oracle.default()
    per_shape = seconds / len(cases)
    rates, rows_done = [], []
    for c in cases:
        w = c.w
        xb, wb = wl.bits(c.host["X"]), wl.bits(c.host["W"])
        rb = wl.bits(c.host["R"]) if c.host["R"] is not None else None
        cols = np.arange(w.N, dtype=np.int64)
        flops, rows, t0 = 0, 0, time.perf_counter()
        while rows < w.M:
            orc.linear_at(xb, wb, rb, np.full(w.N, rows, dtype=np.int64), cols)
            rows += 1
            flops += 2 * w.N * w.K
            if time.perf_counter() - t0 >= per_shape:
                break
        el = time.perf_counter() - t0
        rates.append(flops / el / 1e12)
        rows_done.append(rows)
    return {
        "value": geomean(rates), "unit": "TFLOP/s (fp64 oracle, geomean over 16 shapes)",
        "cores": orc.threads(), "kind": "oracle",
        "sample": (f"whole output rows 0..r-1 of each of the 16 sweep shapes, r = {rows_done} "
                   f"(about {per_shape:.2f} s per shape), same seeded inputs"),
    }


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def gpu_clocks() -> dict:
    """Current shader (sclk) and memory (mclk) clocks of GPU 0 in MHz, read by
    the SMI tool in a child process (a snapshot between timed regions, not an
    average over them); {} when no tool answers."""
    import re
    import subprocess
    for cmd in (["amd-smi", "metric", "-g", "0", "--clock"], ["rocm-smi", "-d", "0", "--showclocks"]):
        try:
            r = subprocess.run(cmd, capture_output=True, text=True, timeout=30)
        except (OSError, subprocess.SubprocessError):
            continue
        text = r.stdout
        out = {}
        for key, pats in (("sclk_mhz", (r"sclk[^\n(]*\((\d+)\s*Mhz", r"GFX_0:\s*\n\s*CLK:\s*(\d+)\s*MHz")),
                          ("mclk_mhz", (r"mclk[^\n(]*\((\d+)\s*Mhz", r"MEM_0:\s*\n\s*CLK:\s*(\d+)\s*MHz"))):
            for pat in pats:
                m = re.search(pat, text, flags=re.I)
                if m:
                    out[key] = int(m.group(1))
                    break
        if out:
            out["tool"] = cmd[0]
            return out
    return {}


def oracle_config_seconds():
    """Whole-output oracle seconds for the tiny, decode and prefill configs
    with every host thread, and on one thread for tiny and decode (the CPU
    baseline: the oracle's own speed, reported, not a target)."""
    import oracle
    from paper_2608_17071_amd import workloads as wl

    orc = oracle.default()
    threads = orc.threads()
    res = {"threads": threads, "whole_config_seconds": {}, "single_thread_seconds": {}}
    for w in (wl.TINY, wl.DECODE, wl.PREFILL):
        t = wl.make_inputs(w)
        xb, wb, rb = wl.bits(t["X"]), wl.bits(t["W"]), wl.bits(t["R"])
        t0 = time.perf_counter()
        orc.linear(xb, wb, rb)
        res["whole_config_seconds"][w.name] = round(time.perf_counter() - t0, 4)
        if w is not wl.PREFILL:
            orc.set_threads(1)
            t0 = time.perf_counter()
            orc.linear(xb, wb, rb)
            res["single_thread_seconds"][w.name] = round(time.perf_counter() - t0, 4)
            orc.set_threads(threads)
    return res


def compare_plans(names, plans, steps, warmup, ka, torch, rotate=True):
    """Time every plan that can run each workload (or the listed ones) under
    the benchmark's protocol (cold operands, graph replay); one workload's
    operand copies at a time.  Workloads: the sweep and gate configs, the
    general-form and the SwiGLU ones.  Returns one row per workload."""
    from paper_2608_17071_amd import workloads as wl
    all_plans = ka.plan_names()
    rows = []
    for n in names:
        if n in wl.GLU_BY_NAME:
            w = wl.GLU_BY_NAME[n]
            ok = lambda p: ka.plan_supports_swiglu(p, w.M, w.N, w.K)
            make = lambda p: GluCase(w, ka, torch, rotate=rotate, plan=p)
            selected = ka.plan_name(ka.select_plan_swiglu(w.M, w.N, w.K))
            base = None
        elif n in wl.GROUPED_BY_NAME:
            w = wl.GROUPED_BY_NAME[n]
            base = GroupedCase(w, ka, torch, rotate=rotate)      # the selected plan; gives M_pad
            mpad = base.Mpad
            ok = lambda p: ka.plan_supports_grouped(p, w.G, mpad, w.N, w.K, w.swiglu)

            def make(p, base=base):
                base.forced = p
                base.plan = p
                base.plan_name = ka.plan_name(p)
                base.times = []
                base.graph = None
                return base
            selected = base.plan_name
        elif n in wl.GENERAL_BY_NAME:
            w = wl.GENERAL_BY_NAME[n]
            ok = lambda p: ka.plan_supports(p, w.M, w.N, w.K, w.has_c)
            make = lambda p: GeneralCase(w, ka, torch, rotate=rotate, plan=p)
            selected = ka.plan_name(ka.select_plan_ex(w.M, w.N, w.K, w.has_c, w.ldx, w.K, w.N, w.N, w.alpha,
                                                      w.beta, w.has_bias))
            base = None
        else:
            w = wl.BY_NAME[n]
            ok = lambda p: ka.plan_supports(p, w.M, w.N, w.K, w.residual)
            base = Case(w, ka, torch, rotate=rotate)

            def make(p, base=base):
                base.force(ka, p)
                return base
            selected = base.plan_name
        cand = [p for p in (plans or all_plans) if not p.startswith("generic") and ok(all_plans.index(p))]
        times = {}
        for p in cand:
            case = make(all_plans.index(p))
            log(f"  {n} plan {p} ...")
            try:
                time_cases([case], steps, warmup, ka, torch)
            except ka.KernelArcError as e:      # a form the plan cannot compute (strides, scalars)
                log(f"    skipped: {e}")
                continue
            times[p] = round(median(case.times) * 1e6, 3)
            if case is not base:
                case.free()
            del case
            torch.cuda.synchronize()
        if base is not None:
            base.free()
        best = min(times, key=times.get) if times else None
        rows.append({"shape": n, "M": getattr(w, "M", None) or getattr(w, "G", 0) * (mpad if n in wl.GROUPED_BY_NAME else 1),
                     "N": w.N, "K": w.K, "selected": selected, "fastest": best, "us": times})
        log(f"  {n}: selected {selected} {times.get(selected)} us, fastest {best} {times.get(best)} us")
    return rows


def write_plan_table(rows, path, command):
    """Markdown summary of compare_plans: per workload the selected plan, the
    fastest plan and every candidate's time."""
    lines = ["# Plan comparison on MI355X (the benchmark's cold-operand protocol, HIP-graph replay)", "",
             "Command (repository root, on the MI355X):", "", "```", command, "```", "",
             "Per workload: the plan the library selects, the fastest candidate, and the median per-call time of",
             "every plan that can run the shape (generic kernel excluded), in microseconds.", "",
             "| shape | selected | selected us | fastest | fastest us | selected / fastest |",
             "|---|---|---|---|---|---|"]
    for r in rows:
        t = r["us"]
        sel, best = r["selected"], r["fastest"]
        ratio = t[sel] / t[best] if sel in t and best in t and t[best] else float("nan")
        lines.append(f"| {r['shape']} | {sel} | {t.get(sel, float('nan')):.2f} | {best} | "
                     f"{t.get(best, float('nan')):.2f} | {ratio:.3f} |")
    lines += ["", "## Every candidate", ""]
    for r in rows:
        cells = ", ".join(f"{p} {v:.2f}" for p, v in sorted(r["us"].items(), key=lambda kv: kv[1]))
        lines.append(f"- **{r['shape']}** (M={r['M']}, N={r['N']}, K={r['K']}): {cells}")
    with open(path, "w") as f:
        f.write("\n".join(lines) + "\n")


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--hot", action="store_true", help="no rotating copies: hot-cache timing (labelled)")
    ap.add_argument("--no-graph", action="store_true", help="launch eagerly instead of replaying a HIP graph")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--no-gates", action="store_true", help="skip the decode/prefill/square extras")
    ap.add_argument("--no-general", action="store_true",
                    help="skip the general-form shapes (alpha, beta, bias, row strides)")
    ap.add_argument("--no-swiglu", action="store_true",
                    help="skip the SwiGLU gate/up shapes")
    ap.add_argument("--no-int8", action="store_true",
                    help="skip the INT8 (W8A8 with dequantisation) shapes")
    ap.add_argument("--no-grouped", action="store_true",
                    help="skip the grouped (mixture-of-experts) shapes")
    ap.add_argument("--only", default="",
                    help="comma-separated workload names (sweep, gate, general-form or SwiGLU): "
                         "time just these (for profiling one kernel)")
    ap.add_argument("--blas", action="store_true",
                    help="with --only: also time torch's GEMM (hipBLASLt) on the plain shapes, same protocol")
    ap.add_argument("--summarize-traffic", nargs=2, metavar=("PMC_DIR", "SHAPES"),
                    help="write profiles/traffic.json for the dominant plan from counter runs")
    ap.add_argument("--compare-plans", action="store_true",
                    help="time every plan that can run each workload of --only (default: the 20 benchmark "
                         "workloads) under the benchmark's protocol; --plans limits the candidates")
    ap.add_argument("--plans", default="", help="with --compare-plans: comma-separated plan names")
    ap.add_argument("--write-table", default="", help="with --compare-plans: write a markdown summary here")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 256 MiB device copy 10 times (reference for HBM byte counters)")
    args = ap.parse_args()

    if args.summarize_traffic:
        pmc_dir, shapes = args.summarize_traffic
        shapes = shapes.split(",")
        cmd = ("rocprofv3 --pmc FETCH_SIZE (then WRITE_SIZE) -d <dir>/fetch (write) -o p --output-format csv "
               f"-- python bench.py --only {','.join(shapes)} --steps 2 --warmup 1; the same two counters of "
               "python bench.py --copy-calibration into <dir>/copy_fetch, <dir>/copy_write")
        summarize_traffic(pmc_dir, TRAFFIC_PLAN, shapes, cmd)
        return

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: this build has no multi-GPU path "
              "(run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2608_17071_amd import kernelarc as ka
    from paper_2608_17071_amd import workloads as wl

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    torch.cuda.set_device(0)
    if args.copy_calibration:
        a = torch.ones(1 << 28, dtype=torch.uint8, device="cuda")
        b = torch.empty_like(a)
        for _ in range(10):
            b.copy_(a)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes_read": a.numel(), "bytes_written": b.numel(), "launches": 10}))
        return

    if args.compare_plans:
        names = args.only.split(",") if args.only else [w.name for w in wl.SWEEP] + \
            [wl.DECODE.name, wl.PREFILL.name, wl.SQUARE.name]
        plans = args.plans.split(",") if args.plans else None
        rows = compare_plans(names, plans, args.steps, args.warmup, ka, torch, rotate=not args.hot)
        if args.write_table:
            cmd = "python bench.py --compare-plans" + (f" --only {args.only}" if args.only else "") + \
                  (f" --plans {args.plans}" if args.plans else "") + f" --steps {args.steps} --warmup {args.warmup}" + \
                  f" --write-table {args.write_table}"
            write_plan_table(rows, args.write_table, cmd)
        print(json.dumps({"plan_table": rows}), flush=True)
        return

    if args.only:
        def case_of(n):
            if n in wl.GLU_BY_NAME:
                return GluCase(wl.GLU_BY_NAME[n], ka, torch, rotate=not args.hot)
            if n in wl.GENERAL_BY_NAME:
                return GeneralCase(wl.GENERAL_BY_NAME[n], ka, torch, rotate=not args.hot)
            if n in wl.I8_BY_NAME:
                return I8Case(wl.I8_BY_NAME[n], ka, torch, rotate=not args.hot)
            if n in wl.F8_BY_NAME:
                return I8Case(wl.F8_BY_NAME[n], ka, torch, rotate=not args.hot)
            if n in wl.GROUPED_BY_NAME:
                return GroupedCase(wl.GROUPED_BY_NAME[n], ka, torch, rotate=not args.hot)
            return Case(wl.BY_NAME[n], ka, torch, rotate=not args.hot)
        cases = [case_of(n) for n in args.only.split(",")]
        if args.blas:
            cases += [BlasCase(c.w, ka, torch, rotate=not args.hot) for c in list(cases) if type(c) is Case]
        time_cases(cases, args.steps, args.warmup, ka, torch, use_graph=not args.no_graph)
        print(json.dumps({"only": [shape_row(c) for c in cases]}), flush=True)
        return
    log("generating inputs ...")
    sweep = [Case(w, ka, torch, rotate=not args.hot) for w in wl.SWEEP]
    torch.cuda.synchronize()
    clocks = {"before_sweep": gpu_clocks()}
    log(f"timing {len(sweep)} shapes x {args.steps} steps (warmup {args.warmup}) ...")
    wall = time_cases(sweep, args.steps, args.warmup, ka, torch, use_graph=not args.no_graph)
    clocks["after_sweep"] = gpu_clocks()
    rows = [shape_row(c) for c in sweep]
    for r in rows:
        log(f"  {r['shape']:24s} {r['plan']:28s} {r['us']:9.2f} us {r['tflops']:8.1f} TF "
            f"{r['gbps']:7.0f} GB/s  {r['bound']} frac {r['roofline_frac']:.3f}")

    gemm_s_per_step = sum(median(c.times) for c in sweep)
    value = geomean([r["tflops"] for r in rows])
    frac_geo = geomean([r["roofline_frac"] for r in rows])

    # dominant kernel variant: most summed time per step
    by_plan = {}
    for c in sweep:
        d = by_plan.setdefault(c.plan_name, {"t": 0.0, "flops": 0, "bytes": 0, "launches": 0, "cases": []})
        d["t"] += median(c.times)
        d["flops"] += c.w.flops
        d["bytes"] += c.w.algorithmic_bytes
        d["launches"] += 1
        d["cases"].append(c)
    dom_name, dom = max(by_plan.items(), key=lambda kv: kv[1]["t"])
    mfma_bound = sum(roofline_time(c.w) for c in dom["cases"] if bound_of(c.w) == "mfma") >= \
        sum(roofline_time(c.w) for c in dom["cases"] if bound_of(c.w) == "hbm")
    avg_launch = dom["t"] / dom["launches"]
    if mfma_bound:
        achieved = dom["flops"] / dom["launches"] / avg_launch / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s"}
    else:
        achieved = dom["bytes"] / dom["launches"] / avg_launch / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBPS, "unit": "GB/s"}
    roof["frac"] = round(achieved / roof["peak"], 4)
    roof["traffic"] = measured_traffic(dom_name)
    roof["kernel"] = dom_name
    roof["avg_launch_us"] = round(avg_launch * 1e6, 3)
    roof["launches_per_step"] = dom["launches"]
    roof["shapes"] = [c.w.name for c in dom["cases"]]

    gates = {}
    if not args.no_gates:
        for c in sweep:
            c.free()
        extra = [Case(w, ka, torch, rotate=not args.hot) for w in (wl.DECODE, wl.PREFILL, wl.SQUARE)]
        clocks["before_gates"] = gpu_clocks()
        time_cases(extra, args.steps, args.warmup, ka, torch, use_graph=not args.no_graph)
        clocks["after_gates"] = gpu_clocks()
        for c in extra:
            r = shape_row(c)
            gates[c.w.name] = r
            log(f"  {r['shape']:24s} {r['plan']:28s} {r['us']:9.2f} us {r['tflops']:8.1f} TF "
                f"{r['gbps']:7.0f} GB/s  {r['bound']} frac {r['roofline_frac']:.3f}")
        del extra

    # The general form (NEXT row: alpha, beta, bias, row strides) on the
    # decoder layer's residual GEMM sites; reported beside the metric.
    general = None
    if not args.no_general:
        for c in sweep:
            c.free()
        gcases = [GeneralCase(w, ka, torch, rotate=not args.hot) for w in wl.GENERAL]
        time_cases(gcases, args.steps, args.warmup, ka, torch, use_graph=not args.no_graph)
        grows = []
        for c in gcases:
            r = shape_row(c)
            grows.append(r)
            log(f"  {r['shape']:40s} {r['plan']:28s} {r['us']:9.2f} us {r['tflops']:8.1f} TF "
                f"{r['gbps']:7.0f} GB/s  {r['bound']} frac {r['roofline_frac']:.3f}")
        general = {"shapes": grows,
                   "geomean_tflops": round(geomean([r["tflops"] for r in grows]), 3),
                   "geomean_roofline_frac": round(geomean([r["roofline_frac"] for r in grows]), 4)}
        if not args.no_cpu_baseline:
            log("timing the CPU oracle on the general form (~4 s) ...")
            general["cpu_baseline"] = cpu_baseline_general(gcases, 4.0)
        for c in gcases:
            c.free()
        del gcases

    # SwiGLU (NEXT row: the decoder layer's gate/up projections with the
    # SiLU-multiply fused into the epilogue); reported beside the metric.
    swiglu = None
    if not args.no_swiglu:
        for c in sweep:
            c.free()
        scases = [GluCase(w, ka, torch, rotate=not args.hot) for w in wl.GLU]
        time_cases(scases, args.steps, args.warmup, ka, torch, use_graph=not args.no_graph)
        srows = []
        for c in scases:
            r = shape_row(c)
            srows.append(r)
            log(f"  {r['shape']:40s} {r['plan']:28s} {r['us']:9.2f} us {r['tflops']:8.1f} TF "
                f"{r['gbps']:7.0f} GB/s  {r['bound']} frac {r['roofline_frac']:.3f}")
        swiglu = {"op": "H = silu(X Wg^T) * (X Wu^T), FLOPs counted as 4MNK",
                  "shapes": srows,
                  "geomean_tflops": round(geomean([r["tflops"] for r in srows]), 3),
                  "geomean_roofline_frac": round(geomean([r["roofline_frac"] for r in srows]), 4)}
        if not args.no_cpu_baseline:
            log("timing the CPU oracle on SwiGLU (~4 s) ...")
            swiglu["cpu_baseline"] = cpu_baseline_glu(scases, 4.0)
        for c in scases:
            c.free()
        del scases

    # INT8 and FP8 (NEXT row: the precision axis, W8A8 with the
    # dequantisation fused into the epilogue, and the decoder layer's INT8
    # gate/up path with the SwiGLU epilogue); roofline against the dense 8-bit
    # MFMA peak.
    int8 = None
    if not args.no_int8:
        for c in sweep:
            c.free()
        icases = [I8Case(w, ka, torch, rotate=not args.hot) for w in wl.I8 + wl.F8]
        time_cases(icases, args.steps, args.warmup, ka, torch, use_graph=not args.no_graph)
        irows = []
        for c in icases:
            r = shape_row(c)
            irows.append(r)
            log(f"  {r['shape']:40s} {r['plan']:28s} {r['us']:9.2f} us {r['tflops']:8.1f} TOP {r['gbps']:7.0f} GB/s  "
                f"{r['bound']} frac {r['roofline_frac']:.3f}")
        int8 = {"op": "Y = bf16(sx[i] sw[j] sum_k qX qW (+ R)); SwiGLU: silu(sx swg Ag) * (sx swu Au); "
                      "int8 (i8_*) or FP8 E4M3 (f8_*) operands; ops = 2MNK (4MNK for SwiGLU), "
                      "peak = dense 8-bit MFMA",
                "peak_tops": PEAK_I8_TOPS, "shapes": irows,
                "geomean_tops": round(geomean([r["tflops"] for r in irows]), 3),
                "geomean_roofline_frac": round(geomean([r["roofline_frac"] for r in irows]), 4)}
        if not args.no_cpu_baseline:
            log("timing the CPU oracle on INT8 (~4 s) ...")
            int8["cpu_baseline"] = cpu_baseline_i8(icases, 4.0)
        for c in icases:
            c.free()
        del icases

    # Grouped (NEXT row: the mixture-of-experts projections over an
    # expert-major padded layout, one launch per projection).
    grouped = None
    if not args.no_grouped:
        for c in sweep:
            c.free()
        gcs = [GroupedCase(w, ka, torch, rotate=not args.hot) for w in wl.GROUPED]
        time_cases(gcs, args.steps, args.warmup, ka, torch, use_graph=not args.no_graph)
        grows2 = []
        for c in gcs:
            r = shape_row(c)
            r.update({"experts": c.w.G, "top_k": c.w.top_k, "tokens": c.w.T, "M_pad": c.Mpad, "rows": c.w.rows})
            grows2.append(r)
            log(f"  {r['shape']:40s} {r['plan']:28s} {r['us']:9.2f} us {r['tflops']:8.1f} TF {r['gbps']:7.0f} GB/s  "
                f"{r['bound']} frac {r['roofline_frac']:.3f}")
        grouped = {"op": "per expert g: Y[g] = X[g] W[g]^T (SwiGLU: silu(X Wg^T) * (X Wu^T)) on its valid rows; "
                         "FLOPs over valid rows only",
                   "shapes": grows2,
                   "geomean_tflops": round(geomean([r["tflops"] for r in grows2]), 3),
                   "geomean_roofline_frac": round(geomean([r["roofline_frac"] for r in grows2]), 4)}
        if not args.no_cpu_baseline:
            log("timing the CPU oracle on the grouped forms (~4 s) ...")
            grouped["cpu_baseline"] = cpu_baseline_grouped(gcs, 4.0)
        for c in gcs:
            c.free()
        del gcs

    cpu = None
    if not args.no_cpu_baseline:
        log(f"timing the CPU oracle (~{args.cpu_seconds:.0f} s) ...")
        cpu = cpu_baseline(sweep, args.cpu_seconds)
        cpu["cpu_model"] = cpu_model()
        log("timing the CPU oracle on whole configs (tiny, decode, prefill; ~5 s) ...")
        cpu.update(oracle_config_seconds())

    out = {
        "metric": "BF16 TFLOP/s and % of MFMA peak (or % HBM BW) per shape; geomean over sweep",
        "value": round(value, 3),
        "unit": "TFLOP/s (geomean over the 16-shape sweep)",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(gemm_s_per_step * 1e3, 4),
        "wall_ms_per_step_all_copies": round(wall / args.steps * 1e3, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic (seeded; bf16 N(0,1)/sqrt(K) operands, N(0,1) residual)",
        "config": {
            "workload": "sweep16: Y = X W^T + R, M in {1,64,512,4096} x N=K in {2048,4096,5120,8192}, seeds 0-15",
            "cache": "hot (labelled)" if args.hot else "cold: calls rotate over >= 1 GiB of operand copies",
            "launch": "eager" if args.no_graph else "HIP graph replay of one call per operand copy",
            "accumulate": "fp32",
        },
        "sweep_geomean_roofline_frac": round(frac_geo, 4),
        "gpu_clocks_mhz": clocks,
        "roofline": roof,
        "cpu_baseline": cpu,
        "shapes": rows,
        "gates": gates,
        "general": general,
        "swiglu": swiglu,
        "int8": int8,
        "grouped": grouped,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
