#!/usr/bin/env python3
"""Benchmark of the FP8 gauge-orbit evaluation on one MI355X.

One step = the whole hot path once for the headline workload, the largest
projection shape: three-level Strassen (8x8x8, 343 products) on A
8192x27648 (Student-t(3), 32 outlier channels x1000) times B 27648x5120
(N(0, 0.015^2)), for 512 sign variants sampled from its orbit: scheme
preparation (the gauge action on the host), the float64 reference, the
classical FP8 baseline with its error, and for every variant the FP8
operands, the 343 block products, the reconstruction and its error on the
device.  Inputs are resident in HBM before timing starts.  Other workloads
(--workload) are the smaller projection shapes.

Prints one JSON line on stdout (progress goes to stderr):
  value  = classical-equivalent FP8 TFLOP/s = G * 2MNK / t,
  roofline = the kernel class with the most time in the timed region, its
             achieved rate from HIP events around each of its launches,
  pipeline = the whole orbit against the matrix-core and HBM ceilings
             (algorithmic flops and bytes per step over the step time),
  cpu_baseline = the oracle on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HEADLINE = "strassen3_8192x27648x5120_sign512"
PEAK_FP8_TFLOPS = 5000.0     # MI355X dense FP8 matrix peak
PEAK_BF16_TFLOPS = 2500.0    # MI355X dense bf16 matrix peak
PEAK_HBM_GBS = 8000.0        # MI355X HBM3E


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def default_chunk(w):
    """Gauges per orbit launch: 16 for three-level schemes, 32 otherwise.
    Measured on one machine at a time, the three-level workload's step took
    1.0-2.3% less at 16 than at 32 (mostly in the block products; 8 was
    slower than 32, 64 as fast as 32), and the two-level 2048 x 4096 x 4096
    step 6% more at 16 than at 32."""
    return 16 if w.levels >= 3 else 32


def kernel_work(cls, w, geo, chunk, G, fused=False):
    """Algorithmic work per step of one kernel class, summed over its launches
    (the orbit's chunks and the classical baseline's single launch), and the
    class's roofline bound.  `fused`: the per-tensor schedule over several
    chunks, where each chunk's codes are formed in one pass with the next
    chunk's maxima (the maxima class then runs for the first chunk only).
    Units of work:
      block_gemm: 2*Mb*Nb*Kb flops per block product; G*R products for the
                  orbit plus the classical product 2*M*N*K;
      recon:      per gauge, R*Mb*Nb fp32 products read; per launch, the
                  M*N float64 reference read once (the gauges of a launch
                  share it; C is not written); the classical baseline reads
                  M*N products and writes C;
      form_amax:  each launch reads one operand once in fp32 (A, or B^T):
                  the classical baseline's and, per chunk, the orbit's (the
                  first chunk's only when fused);
      form_quant: each launch reads one operand and writes its FP8 codes;
      reference:  reads A and B in fp32, writes C_ref in float64.
    """
    gm, gk, gn, R = geo
    M, N, K = w.M, w.N, w.K
    Mb, Kb, Nb = M // gm, K // gk, N // gn
    chunks = -(-G // chunk)
    ops = (M * K + N * K) * 4.0
    if cls == "block_gemm":
        return "mfma", G * R * 2.0 * Mb * Nb * Kb + 2.0 * M * N * K, "TFLOP/s"
    if cls == "recon":
        return "hbm", G * R * Mb * Nb * 4.0 + chunks * M * N * 8.0 + M * N * 8.0, "GB/s"
    if cls == "form_amax":
        return "hbm", (2 if fused else chunks + 1) * ops, "GB/s"
    if cls == "form_quant":
        return "hbm", (chunks + 1) * ops + G * R * (Mb * Kb + Nb * Kb) + (M * K + N * K), "GB/s"
    if cls == "reference":
        return "hbm", ops + M * N * 8.0, "GB/s"
    raise ValueError(cls)


def profiled_traffic(cls, workload, steps_work):
    """HBM bytes per step of a kernel class from the committed rocprofv3
    counter summary (profiles/traffic_<class>_<workload>.txt: FETCH_SIZE and
    WRITE_SIZE passes, calibrated with a plain 1 GiB copy).  None when there
    is no summary or the kernel sources changed since it was taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", f"traffic_{cls}_{workload}.txt")
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if line.startswith("#") or ":" not in line:
            continue
        k, v = line.split(":", 1)
        kv[k.strip()] = v.strip()
    h = hashlib.sha256()
    for src in kv.get("sources", "").split(","):
        h.update(open(os.path.join(ROOT, src), "rb").read())
    if h.hexdigest() != kv.get("sources_sha256"):
        return None
    rd, wr = float(kv["read_bytes_per_step"]), float(kv["write_bytes_per_step"])
    launches = float(kv["dispatches_per_step"])
    return dict(bytes_per_step=rd + wr, read_bytes_per_step=rd, write_bytes_per_step=wr,
                algorithmic_bytes_per_step=steps_work, bytes_per_launch=(rd + wr) / launches,
                algorithmic_bytes_per_launch=steps_work / launches,
                source=os.path.relpath(path, ROOT))


def gemm_bytes(w, geo, G):
    """Algorithmic HBM bytes per step of the block products: FP8 operands read
    once and fp32 products written once (orbit), plus the classical product."""
    gm, gk, gn, R = geo
    Mb, Kb, Nb = w.M // gm, w.K // gk, w.N // gn
    return G * R * (Mb * Kb + Nb * Kb + 4.0 * Mb * Nb) + (w.M * w.K + w.N * w.K + 4.0 * w.M * w.N)


def cpu_model():
    """The host CPU's model name (first entry of /proc/cpuinfo), or None."""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def library_gemm(w, geo, dev, iters=5):
    """The vendor library's GEMMs (torch, which calls hipBLASLt) on the shapes
    of the block products, after the timed region: one gauge's R products as
    one bf16 batched product (bf16 out), and the flat M x K x N product in
    bf16 and with the FP8 instructions (E4M3, unit scales, fp32 out; their
    sums are not exact, unlike the library's own block products).  Operands
    are random, contiguous and resident; times are HIP-event averages."""
    import torch
    gm, gk, gn, R = geo
    Mb, Kb, Nb = w.M // gm, w.K // gk, w.N // gn
    g = torch.Generator(device=dev)
    g.manual_seed(0)

    def timed(fn):
        for _ in range(2):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(iters):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / iters

    res = {}
    a = torch.randn((R, Mb, Kb), generator=g, device=dev, dtype=torch.bfloat16)
    b = torch.randn((R, Kb, Nb), generator=g, device=dev, dtype=torch.bfloat16)
    ms = timed(lambda: torch.bmm(a, b))
    res["bmm_bf16_one_gauge"] = dict(shape=[R, Mb, Kb, Nb], ms=round(ms, 4),
                                     tflops=round(2.0 * R * Mb * Kb * Nb / ms / 1e9, 1))
    del a, b
    a = torch.randn((w.M, w.K), generator=g, device=dev, dtype=torch.bfloat16)
    b = torch.randn((w.K, w.N), generator=g, device=dev, dtype=torch.bfloat16)
    flat = 2.0 * w.M * w.K * w.N
    ms = timed(lambda: a @ b)
    res["mm_bf16_flat"] = dict(shape=[w.M, w.K, w.N], ms=round(ms, 4),
                               tflops=round(flat / ms / 1e9, 1))
    a8 = a.to(torch.float8_e4m3fn)
    b8 = b.t().contiguous().to(torch.float8_e4m3fn).t()
    one = torch.ones((), device=dev)
    ms = timed(lambda: torch._scaled_mm(a8, b8, one, one, out_dtype=torch.float32))
    res["scaled_mm_fp8_flat"] = dict(shape=[w.M, w.K, w.N], ms=round(ms, 4),
                                     tflops=round(flat / ms / 1e9, 1))
    del a, b, a8, b8
    torch.cuda.empty_cache()
    return res


def library_hbm(dev, iters=10):
    """What plain passes over 4 GiB of fp32 reach in torch's own kernels:
    a maximum per row of 4096 (reads), a fill (writes) and a copy (reads
    and writes), in GB/s of bytes moved; HIP-event averages."""
    import torch
    n = 1 << 30
    x = torch.ones(n, dtype=torch.float32, device=dev)
    y = torch.empty_like(x)

    def rate(fn, nbytes):
        for _ in range(2):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(iters):
            fn()
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / iters
        return dict(ms=round(ms, 4), gbs=round(nbytes / ms / 1e6, 1))

    res = dict(row_max_read=rate(lambda: x.view(-1, 4096).amax(dim=1), 4 * n),
               fill_write=rate(lambda: y.fill_(1.0), 4 * n),
               copy_read_write=rate(lambda: y.copy_(x), 8 * n))
    del x, y
    torch.cuda.empty_cache()
    return res


# Classical-equivalent flops the oracle is given per gauge in the CPU sample:
# at about 0.04 TFLOP/s on 16 host cores this is about 8 s per gauge.
CPU_SAMPLE_FLOPS = 4e11


def cpu_sample_rows(w, gm):
    """Rows of A the CPU sample uses: all of them, or the first M / f for the
    least power of two f that brings 2 (M / f) N K under CPU_SAMPLE_FLOPS
    while M / f stays a multiple of the grid's m^L."""
    rows = w.M
    while 2.0 * rows * w.N * w.K > CPU_SAMPLE_FLOPS and rows % (2 * gm) == 0:
        rows //= 2
    return rows


def cpu_baseline(w, A, B, gauges, scale_mode=0, budget_s=10.0):
    """The oracle (plain C, OpenMP) on the first gauges of the workload's
    orbit, one after another until about budget_s seconds have passed (at
    least one, at most 16).  On the largest shapes one gauge would take
    about a minute, so the sample keeps the workload's K, N, scheme and
    gauges and takes the first rows of A (cpu_sample_rows); the rate is
    classical-equivalent flops of the sample over its time."""
    import oracle
    from oracle import scheme_ops as so
    from oracle import schemes as osch

    base = osch.BASE_SCHEMES[w.scheme]()
    gm = base.m ** w.levels
    rows = cpu_sample_rows(w, gm)
    As = A[:rows]
    t = 0.0
    n = 0
    dims = None
    while n < min(16, len(gauges)) and (n == 0 or t < budget_s):
        g = gauges[n]
        s = so.gauge(so.power(base, w.levels), *g) if w.gauge_kind == "sign" else \
            so.power(so.gauge(base, *g), w.levels)
        tabs, dims = oracle.flatten_f32(s)
        t0 = time.perf_counter()
        if scale_mode & ~0xff:  # the repairs (group schedule)
            oracle.lowp_matmul_repaired(As, B, tabs, dims, flags=(scale_mode >> 8) & 3)
        else:
            oracle.lowp_matmul(As, B, tabs, dims, scale_mode=scale_mode)
        t += time.perf_counter() - t0
        n += 1
    cores = oracle.default_threads()
    shape = (f"the full {w.M}x{w.K}x{w.N} shape" if rows == w.M else
             f"the first {rows} of the {w.M} rows of A ({rows}x{w.K}x{w.N}; same B, scheme "
             f"and gauges)")
    return dict(value=n * 2.0 * rows * w.N * w.K / t / 1e12, unit="TFLOP/s (classical-equivalent)",
                cores=cores, cpu_model=cpu_model(), kind="oracle",
                sample=f"the first {n} of {w.G} gauge variants on {shape}: FP8 operands, "
                       f"{dims[3]} block products, reconstruction each; {t:.2f} s; the float64 "
                       f"reference is not included")


def pipeline_work(w, geo, G, chunk):
    """Algorithmic work of one step's orbit (all G gauges): the block
    products' matrix flops, and the least HBM traffic of the schedule with
    materialized products: per gauge the FP8 operands written and read once
    and the fp32 products written and read once; per launch of `chunk`
    gauges the float64 reference read once (operand inputs, read once per
    chunk, are left out)."""
    gm, gk, gn, R = geo
    Mb, Kb, Nb = w.M // gm, w.K // gk, w.N // gn
    flops = G * R * 2.0 * Mb * Nb * Kb
    hbm = (G * (2.0 * R * (Mb * Kb + Nb * Kb) + 2.0 * 4.0 * R * Mb * Nb)
           + -(-G // chunk) * 8.0 * w.M * w.N)
    return flops, hbm


# The paper's integer timings (App. E, one H20 at 4096 x 4096 x 4096 from
# prequantized codes and scales): classical int8 563-774 us over groups of
# 128/256/512; one Strassen level (code bound 63) 2.04/3.17/2.09x as long as
# classical int8; two levels (code bound 31, groups of 256) 27.9x.
PAPER_INT8_RATIO = {("strassen1", 128): 2.04, ("strassen1", 256): 3.17, ("strassen1", 512): 2.09,
                    ("strassen2", 256): 27.9}


def int8_bench(args):
    """Classical int8 and the certified fast realizations at 4096^3: the
    upper median of 30 timed calls (HIP events), each after zeroing a 256 MB
    buffer so no operand stays in the caches, after 8 warmup calls; the fast
    outputs are checked bit for bit against the classical ones."""
    import numpy as np
    import torch
    from paper_2609_39816_amd import fm

    n = args.int8_size
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    rng = np.random.default_rng(20261202)
    A = torch.from_numpy(rng.standard_normal((n, n)).astype(np.float32)).to(dev)
    B = torch.from_numpy(rng.standard_normal((n, n)).astype(np.float32)).to(dev)
    flush = torch.empty(64 << 20, dtype=torch.float32, device=dev)
    s = fm.Scheme.base("strassen")

    def timed(fn):
        for _ in range(8):
            fn()
        ts = []
        for _ in range(30):
            flush.zero_()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1) * 1e3)
        return float(np.sort(ts)[len(ts) // 2])

    rows = []
    configs = ([("strassen1", 1, 63, 64, g, False) for g in (128, 256, 512)] +
               [("strassen2", 2, 31, 32, 256, False), ("strassen2", 2, 127, 32, 128, True)])
    classical_us = {}
    for name, levels, b, h, g, corr in configs:
        Ac, dA = fm.int8_quantize(A, g, b)
        BTc, dB = fm.int8_quantize(B.t().contiguous(), g, b)
        out_c = torch.empty((n, n), dtype=torch.float32, device=dev)
        out_f = torch.empty_like(out_c)
        us_c = timed(lambda: fm.int8_matmul_classical(Ac, dA, BTc, dB, g, out=out_c))
        # the scheme's tables and tile schedule are prepared once, outside
        # the timed calls (the kernels are timed, as in App. E)
        plan = fm.Int8Plan(s, n, n, n, levels, g, h, b, b, correct=corr, device=dev)
        us_f = timed(lambda: plan.run(Ac, dA, BTc, dB, out=out_f))
        fm.status(plan.ws)
        same = bool(torch.equal(out_c.view(torch.int32), out_f.view(torch.int32)))
        classical_us[(b, g)] = us_c
        rows.append(dict(scheme=name, corrected=corr, code_bound=b, group=g, block_inner=h,
                         classical_us=round(us_c, 1),
                         fast_us=round(us_f, 1), ratio=round(us_f / us_c, 3),
                         paper_ratio=None if corr else PAPER_INT8_RATIO.get((name, g)),
                         classical_tops=round(2.0 * n ** 3 / us_c / 1e6, 1),
                         bit_identical=same))
        log(f"[bench] int8 {name}{' corrected' if corr else ''} b={b} g={g}: classical {us_c:.1f} us, fast {us_f:.1f} us, "
            f"ratio {us_f / us_c:.3f}, bits equal {same}")
    out = {"metric": "certified int8 matmul time relative to classical int8 (4096^3, upper median)",
           "value": rows[3]["ratio"], "unit": "x classical int8 (two-level Strassen, b=31, g=256)",
           "higher_is_better": False, "n_gpus": 1, "data": "synthetic",
           "config": {"workload": f"int8_{n}x{n}x{n}", "M": n, "K": n, "N": n},
           "vs_baseline": round(rows[3]["ratio"] / PAPER_INT8_RATIO[("strassen2", 256)], 4),
           "rows": rows}
    print(json.dumps(out), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default=HEADLINE)
    ap.add_argument("--chunk", type=int, default=None,
                    help="gauges per launch, rounded down to G / 2^k (default: default_chunk of "
                         "the workload; 0: the whole orbit in one launch)")
    ap.add_argument("--fmt", default=None)
    ap.add_argument("--scale-mode", default="tensor", choices=["tensor", "rowcol", "group"],
                    help="scale granularity of the FP8 rounding of block sums")
    ap.add_argument("--repair", default="none", choices=["none", "rows", "weights", "both"],
                    help="repairs of the group schedule (with --scale-mode group)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-timing", action="store_true", help="do not bracket kernels with events")
    ap.add_argument("--int8", action="store_true",
                    help="time the integer path (classical int8 and the certified realizations)")
    ap.add_argument("--int8-size", type=int, default=4096)
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run a plain 1 GiB device copy (reference for HBM byte counters)")
    ap.add_argument("--library-gemm", action="store_true",
                    help="also time the vendor library's GEMMs (torch on hipBLASLt) on the "
                         "block-product shapes, and torch's plain HBM passes (a row maximum, "
                         "a fill, a copy of 4 GiB), as context for the kernels' rooflines")
    args = ap.parse_args()
    if args.gpus != 1:
        print(json.dumps({"error": "this benchmark runs on one GPU only; the gauge orbit would "
                                   "shard over GPUs by gauge (see the design notes)",
                          "n_gpus": args.gpus}))
        sys.exit(2)

    if args.int8:
        int8_bench(args)
        return

    import numpy as np
    import torch

    import synthetic as sy
    from paper_2609_39816_amd import fm

    w = sy.WORKLOADS[args.workload]
    fmt_name = args.fmt or w.fmts[0]
    fmt = fm.FMTS[fmt_name]
    smode = {"tensor": fm.SCALE_TENSOR, "rowcol": fm.SCALE_ROWCOL, "group": fm.SCALE_GROUP}[
        args.scale_mode]
    if args.repair != "none":
        if smode != fm.SCALE_GROUP:
            sys.exit("the repairs belong to the group schedule: add --scale-mode group")
        smode |= {"rows": fm.REPAIR_ROWS, "weights": fm.REPAIR_WEIGHTS,
                  "both": fm.REPAIR_ROWS | fm.REPAIR_WEIGHTS}[args.repair]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    log(f"[bench] workload {w.name}: generating inputs")
    A, B = sy.operands(w)
    gauges = sy.gauges(w)
    G = len(gauges)
    At = torch.from_numpy(A).to(dev)
    Bt = torch.from_numpy(B).to(dev)

    base = fm.Scheme.base(w.scheme)
    if w.gauge_kind == "sign":
        flat = base.kron(w.levels) if w.levels > 1 else base
        levels = 1
    else:
        flat = base
        levels = w.levels
    classical = fm.Scheme.base("classical")
    geo = flat.flat_dims(levels)
    req = default_chunk(w) if args.chunk is None else args.chunk
    # the orbit runs in chunks of G / 2^k gauges: the largest such that its
    # workspace fits, here the largest not above the request
    chunk = G
    while req > 0 and chunk > max(1, req):
        chunk = max(1, chunk // 2)
    if req > 0 and chunk != req:
        log(f"[bench] {req} gauges per launch requested: the orbit runs {chunk} (G / 2^k)")
    # per-tensor scales over several chunks: codes and the next chunk's maxima in one pass
    fused = smode == fm.SCALE_TENSOR and chunk < G
    ws = fm.workspace(fm.workspace_size(flat, w.M, w.N, w.K, levels, G, chunk, smode))
    ws_cl = fm.workspace(fm.workspace_size(classical, w.M, w.N, w.K, 1, 1, 1, smode))
    ws_err = fm.workspace(fm.lib.fm_error_workspace_size(w.M, w.N))
    Cref = torch.empty((w.M, w.N), dtype=torch.float64, device=dev)
    C_cl = torch.empty((w.M, w.N), dtype=torch.float32, device=dev)
    log(f"[bench] workspace {ws.numel() / 1e9:.2f} GB, chunk {chunk}, family "
        f"{flat.kernel_family(levels)}")

    def step():
        # device work that needs no host preparation goes first, so the host
        # gauge action below overlaps it
        fm.reference_f64(At, Bt, out=Cref)
        fm.matmul_lowp(classical, At, Bt, 1, fmt, ws=ws_cl, out=C_cl, scale_mode=smode)
        hips = (flat if w.gauge_kind == "sign" else base).gauge_orbit(gauges)
        errs = fm.orbit_eval(hips, At, Bt, Cref, levels, fmt, ws=ws, scale_mode=smode)
        st = fm.error_stats(C_cl, Cref, ws=ws_err)
        return errs / st["rel_fro"], st["rel_fro"]

    if args.copy_calibration:
        x = torch.ones(1 << 28, dtype=torch.float32, device=dev)
        y = torch.empty_like(x)
        y.copy_(x)
        torch.cuda.synchronize()
        log("[bench] copy calibration: 1 GiB read + 1 GiB written by one copy kernel")
        del x, y
    for i in range(args.warmup):
        step()
        log(f"[bench] warmup {i + 1}/{args.warmup} done")
    torch.cuda.synchronize()
    if not args.no_timing:
        fm.timing_reset()
        fm.timing_enable(True)
    t0 = time.perf_counter()
    for i in range(args.steps):
        ratios, err_cl = step()
        log(f"[bench] step {i + 1}/{args.steps} done")
    torch.cuda.synchronize()
    t = (time.perf_counter() - t0) / args.steps
    roof = None
    per_class = {}
    if not args.no_timing:
        fm.timing_enable(False)
        for cls in fm.TIMED_CLASSES:
            n, ms = fm.timing_read(cls)
            per_class[cls] = dict(launches=n, total_ms=ms)
        fm.timing_reset()
        dom = max(per_class, key=lambda c: per_class[c]["total_ms"])
        n, ms = per_class[dom]["launches"], per_class[dom]["total_ms"]
        bound, work, unit = kernel_work(dom, w, geo, chunk, G, fused)
        # achieved = work per launch / average launch duration = work / time
        avg_s = ms / 1e3 / max(1, n)
        tot_s = ms / 1e3 / args.steps
        peak_note = None
        if unit == "TFLOP/s":
            # the default arithmetic widens the FP8 codes exactly to bf16 and
            # multiplies with the bf16 matrix instructions: their peak is the
            # kernel's ceiling; the FP8 instructions' peak is reported beside it
            fp8_mfma = fm.get_block_product_arithmetic() == fm.ACC_FP8
            achieved = work / tot_s / 1e12
            peak = PEAK_FP8_TFLOPS if fp8_mfma else PEAK_BF16_TFLOPS
            peak_note = dict(instruction="FP8 matrix instructions" if fp8_mfma
                             else "bf16 matrix instructions on exactly widened FP8 codes",
                             fp8_peak=PEAK_FP8_TFLOPS,
                             frac_of_fp8_peak=round(achieved / PEAK_FP8_TFLOPS, 4))
        else:
            achieved, peak = work / tot_s / 1e9, PEAK_HBM_GBS
        # the byte counters were taken for the per-tensor schedule only
        traffic = (profiled_traffic(dom, w.name, gemm_bytes(w, geo, G))
                   if dom == "block_gemm" and smode == fm.SCALE_TENSOR else None)
        roof = dict(bound=bound, kernel=dom, achieved=round(achieved, 2), peak=peak, unit=unit,
                    frac=round(achieved / peak, 4),
                    traffic=(round(traffic["bytes_per_step"] / (n / args.steps))
                             if traffic else None),
                    traffic_detail=traffic, peak_basis=peak_note,
                    avg_launch_ms=round(avg_s * 1e3, 4), launches_per_step=n / args.steps)
        log("[bench] per-class kernel time per step (ms): " +
            ", ".join(f"{c} {v['total_ms'] / args.steps:.2f} ({v['launches'] // args.steps} launches)"
                      for c, v in per_class.items()))

    flops = G * 2.0 * w.M * w.N * w.K
    value = flops / t / 1e12
    mfma_flops, hbm_bytes = pipeline_work(w, geo, G, chunk)
    # the whole orbit against both ceilings: its block products' matrix
    # flops over the step time against the matrix peak of the instruction
    # issued (and the FP8 peak), and its least HBM traffic over the step time
    # against the HBM peak; per kernel class, achieved rates from the HIP
    # event times of its launches
    fp8_mfma = fm.get_block_product_arithmetic() == fm.ACC_FP8
    pipe = dict(mfma_flops_per_step=mfma_flops, hbm_bytes_per_step=hbm_bytes,
                mfma_tflops=round(mfma_flops / t / 1e12, 2),
                frac_of_mfma_peak=round(mfma_flops / t / 1e12 /
                                        (PEAK_FP8_TFLOPS if fp8_mfma else PEAK_BF16_TFLOPS), 4),
                frac_of_fp8_peak=round(mfma_flops / t / 1e12 / PEAK_FP8_TFLOPS, 4),
                hbm_gbs=round(hbm_bytes / t / 1e9, 1),
                frac_of_hbm_peak=round(hbm_bytes / t / 1e9 / PEAK_HBM_GBS, 4))
    per_class_rate = {}
    for cls, v in per_class.items():
        if v["total_ms"] <= 0:
            continue
        bound, work, unit = kernel_work(cls, w, geo, chunk, G, fused)
        secs = v["total_ms"] / 1e3 / args.steps
        if unit == "TFLOP/s":
            per_class_rate[cls] = dict(ms_per_step=round(secs * 1e3, 3),
                                       tflops=round(work / secs / 1e12, 1))
        else:
            per_class_rate[cls] = dict(ms_per_step=round(secs * 1e3, 3),
                                       gbs=round(work / secs / 1e9, 1),
                                       frac_of_hbm_peak=round(work / secs / 1e9 / PEAK_HBM_GBS, 4))
    st = dict(min=float(ratios.min()), median=float(np.sort(ratios)[len(ratios) // 2]),
              max=float(ratios.max()), identity=float(ratios[0]))
    out = {
        "metric": "classical-equiv FP8 TFLOP/s (2MNK/t) + gauge-scheme evals/sec; % of MFMA peak",
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(t * 1e3, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": fmt_name,
        "data": "synthetic",
        "config": {"workload": w.name, "M": w.M, "K": w.K, "N": w.N, "scheme": w.scheme,
                   "levels": w.levels, "gauges": G, "gauge_kind": w.gauge_kind, "fmt": fmt_name,
                   "chunk": chunk, "scale_mode": args.scale_mode, "repair": args.repair,
                   "parallelism": "none (1 GPU)"},
        "evals_per_s": round(G / t, 1),
        "pct_mfma_peak_classical_equiv": round(100 * value / PEAK_FP8_TFLOPS, 2),
        "pct_mfma_peak_actual": round(100 * mfma_flops / t / 1e12 / PEAK_FP8_TFLOPS, 2),
        "classical_fp8_rel_fro": err_cl,
        "ratio_stats": st,
        "roofline": roof,
        "pipeline": pipe,
        "kernel_classes": per_class_rate,
    }
    if args.library_gemm:
        log("[bench] library GEMMs on the block-product shapes")
        out["library_gemm"] = library_gemm(w, geo, dev)
        out["library_hbm"] = library_hbm(dev)
    if not args.no_cpu_baseline:
        log("[bench] oracle baseline on the host cores")
        out["cpu_baseline"] = cpu_baseline(w, A, B, gauges, smode)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
