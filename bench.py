#!/usr/bin/env python3
"""Benchmark: emulated FP64 GEMM (Ozaki Scheme II, round to nearest) on one
MI355X, through the C ABI.

One step = one full ozaki25_dgemm_ex call: exponent scans, deconstruction of
both operands into planes, the per-modulus products and the CRT
reconstruction, on synthetic seeded inputs that are already resident in HBM.
The headline line is the published 12-modulus set (e4m3 planes, 36 FP8-MFMA
limb products with FP32 accumulation and the modular epilogue); the same run
also times the all-byte 15-modulus set of Sec. 5.1 (int8 planes, 15 int8-MFMA
products) on the same inputs and reports it under "all_byte_set".
``--moduli a15`` makes the all-byte set the headline instead; ``--quantiser
tz`` times the truncating quantiser.  Each set also reports "stored_planes":
the per-call time of ozaki25_dgemm_planes on planes made once (storage mode
P); the headline set also "graph_replay": one call captured in a HIP graph
and replayed.  Prints one JSON line.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload square] [--moduli s12|a15]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import workloads  # noqa: E402

# MI355X published peaks
HBM_PEAK_GBS = 8000.0
FP8_PEAK_TOPS = 5000.0
INT8_PEAK_TOPS = 5000.0
FP64_PEAK_TFLOPS = 78.6

# per modulus set: products per output, plane bytes per input element,
# residue bytes per output (the fused path's internal products), peak
SETS = {
    "s12": dict(id=0, oracle_set=0, r=12, products=36, plane_bytes=30, cres_bytes=24,
                peak=FP8_PEAK_TOPS, dtype="fp8", moduli="published 12-modulus set",
                route="e4m3 MFMA, fp32 accumulate", gemm_kernel="residue_gemm_kernel<int16>",
                persistent_kernel="residue_gemm_persistent_kernel<int16>",
                dec_kernel="deconstruct_kernel<0>+<1>",
                fused_kernel="fused_pub_kernel", fused_products=30,
                note="fp8 ops (1 MAC = 2 ops): 36 limb products x 2mnk per launch; peak is the dense fp8 rate"),
    "a15": dict(id=1, oracle_set=1, r=15, products=15, plane_bytes=15, cres_bytes=15,
                peak=INT8_PEAK_TOPS, dtype="int8", moduli="all-byte 15-modulus set (Sec. 5.1 candidate A)",
                route="int8 MFMA, int32 accumulate", gemm_kernel="residue_gemm_bytes_kernel<int8>",
                persistent_kernel="residue_gemm_bytes_persistent_kernel<int8>",
                dec_kernel="deconstruct_bytes_kernel<0>+<1>",
                fused_kernel="fused_bytes_kernel", fused_products=15,
                note="int8 ops (1 MAC = 2 ops): 15 residue products x 2mnk per launch; peak is the dense int8 rate"),
}
COUNTER_FILES = {"s12": os.path.join(ROOT, "profiles", "residue_gemm_square_counters.txt"),
                 "a15": os.path.join(ROOT, "profiles", "residue_gemm_bytes_square_counters.txt")}
GEMM_SOURCE = os.path.join(ROOT, "paper_2609_09095_amd", "csrc", "residue_gemm.hip")
DEC_COUNTERS = os.path.join(ROOT, "profiles", "deconstruct_square_counters.txt")
DEC_SOURCES = [os.path.join(ROOT, "paper_2609_09095_amd", "csrc", f) for f in ("scan.hip", "deconstruct.hip")]


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def source_hash(path):
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def sources_hash(paths):
    h = hashlib.sha256()
    for path in paths:
        with open(path, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def counter_value(path, w, digest, key):
    """A value from a committed rocprofv3 counter summary, or None if it is
    absent, for another workload, or taken on another version of the kernel
    sources (digest)."""
    if not os.path.exists(path):
        return None
    kv = {}
    with open(path) as f:
        for line in f:
            if ":" in line and not line.startswith("#"):
                k, val = line.split(":", 1)
                kv[k.strip()] = val.strip()
    try:
        if kv.get("workload") != w.name or kv.get("source_sha256_16") != digest:
            return None
        return float(kv[key])
    except (KeyError, ValueError):
        return None


def measured_traffic(w, moduli):
    """HBM bytes per residue-GEMM launch (FETCH_SIZE and WRITE_SIZE, scaled)."""
    return counter_value(COUNTER_FILES[moduli], w, source_hash(GEMM_SOURCE), "hbm_bytes_per_launch")


def measured_deconstruction(w, moduli, scan_ms, dec_ms):
    """Bytes the exponent scans and the deconstruction of both operands move
    between L2 and the memory side per call (FETCH_SIZE + WRITE_SIZE, scaled),
    and that rate over the two stages' time as a fraction of the HBM peak.
    The deconstruction of a run re-reads what its scan just read, mostly from
    the last-level cache, which these counters do not tell apart from HBM:
    the fraction is an upper bound on HBM use."""
    b = counter_value(DEC_COUNTERS, w, sources_hash(DEC_SOURCES), f"hbm_bytes_per_call_{moduli}")
    if b is None:
        return {"measured_bytes": None, "measured_frac": None}
    return {"measured_bytes": b,
            "measured_frac": round(b / ((scan_ms + dec_ms) * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
            "measured_note": "bytes beyond L2 (HBM or the last-level cache); an upper bound on HBM use"}


def cpu_baseline(A, B, w, rows, cols, cfg):
    """The oracle as it stands on `rows` x `cols` outputs of the workload at
    full k, its output rows dealt over host threads (one oracle call per
    block of rows; the oracle's C calls release the GIL)."""
    import concurrent.futures as cf
    import oracle
    oracle.build(force=False)
    threads = max(1, min(16, os.cpu_count() or 1, rows))
    cidx = np.arange(cols)
    blocks = np.array_split(np.arange(rows), threads)
    t0 = time.perf_counter()
    with cf.ThreadPoolExecutor(max_workers=threads) as ex:
        for f in [ex.submit(oracle.dgemm, A, B, rows=b, cols=cidx, want_planes=False, set=cfg["oracle_set"])
                  for b in blocks]:
            f.result()
    dt = time.perf_counter() - t0
    flops = 2.0 * rows * cols * w.k
    return {"value": flops / dt / 1e12, "unit": "TFLOPS", "cores": threads, "kind": "oracle",
            "sample": f"{rows} rows of A x {cols} columns of B of the {w.name} workload, full k={w.k} "
                      f"(exponent scan, quantise, residues, {cfg['r']} int64 residue GEMMs, Garner, "
                      f"rounding, exact-product check), {dt:.1f} s on {threads} threads"}


def vendor_lowp_gemm(torch, w, cfg, steps):
    """The vendor library's dense low-precision GEMM on one residue product's
    shape (m x k times k x n, limb-sized integer data): hipBLASLt e4m3 through
    torch._scaled_mm for the published set, int8 through torch._int_mm for the
    all-byte set.  A practical reference for the residue GEMM's rate, not part
    of the emulated path."""
    dev = torch.device("cuda:0")
    g = torch.Generator(device=dev)
    g.manual_seed(7)
    A = torch.randint(-22, 23, (w.m, w.k), dtype=torch.int8, device=dev, generator=g)
    Bt = torch.randint(-22, 23, (w.n, w.k), dtype=torch.int8, device=dev, generator=g)
    if cfg["dtype"] == "fp8":
        Af = A.to(torch.float32).to(torch.float8_e4m3fn)
        Bf = Bt.to(torch.float32).to(torch.float8_e4m3fn)
        one = torch.tensor(1.0, device=dev)
        fn = lambda: torch._scaled_mm(Af, Bf.t(), scale_a=one, scale_b=one, out_dtype=torch.bfloat16)  # noqa: E731
        lib_name = "hipBLASLt e4m3 x e4m3 -> bf16 (torch._scaled_mm)"
    else:
        fn = lambda: torch._int_mm(A, Bt.t())  # noqa: E731
        lib_name = "int8 x int8 -> int32 (torch._int_mm)"
    try:
        fn()
        torch.cuda.synchronize()
        # one untimed call first, so that the GPU is busy when the start event
        # is reached and the timed calls run back to back (otherwise the host's
        # latency for the first call falls inside the timed range)
        steps = max(steps, 20)
        s0, s1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        fn()
        s0.record()
        for _ in range(steps):
            fn()
        s1.record()
        torch.cuda.synchronize()
        ms = s0.elapsed_time(s1) / steps
    except Exception as e:  # the library may lack a solution for the shape
        return {"library": lib_name, "error": str(e)[:200]}
    tops = 2.0 * w.m * w.n * w.k / (ms * 1e-3) / 1e12
    return {"library": lib_name, "ms_per_call": round(ms, 4), "achieved": round(tops, 3),
            "peak": cfg["peak"], "frac": round(tops / cfg["peak"], 4),
            "unit": "TFLOP/s" if cfg["dtype"] == "fp8" else "TOP/s"}


def time_set(oz, torch, w, Ad, Bd, Cd, cfg, steps, warmup, quant):
    """Mean ms per step and per stage of ozaki25_dgemm_ex for one modulus set."""
    ws = torch.empty(oz.ozaki25_dgemm_workspace_size(w.m, w.n, w.k, cfg["id"]), dtype=torch.uint8,
                     device=Ad.device)

    def step(events=None):
        oz.ozaki25_dgemm_ex(Ad, Bd, Cd, subtract=w.subtract, workspace=ws, stage_events=events,
                            set=cfg["id"], quantiser=quant)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(oz.NUM_STAGE_EVENTS)] for _ in range(steps)]
    for row in ev:
        for e in row:
            e.record()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for i in range(steps):
        step(ev[i])
    end.record()
    torch.cuda.synchronize()
    ms = start.elapsed_time(end) / steps
    stage = np.array([[row[j].elapsed_time(row[j + 1]) for j in range(oz.NUM_STAGE_EVENTS - 1)] for row in ev])
    median = float(np.median([row[0].elapsed_time(row[-1]) for row in ev]))
    del ws
    return ms, stage.mean(axis=0).tolist(), median


def time_accurate(oz, torch, w, Ad, Bd, Cd, C0d, cfg, steps, warmup, quant):
    """ms per step and per stage of ozaki25_dgemm_accurate (the accurate
    mode: magnitude digits, bound product and shifts, then the same stages
    as the fast mode with those exponents)."""
    ws = torch.empty(oz.ozaki25_dgemm_accurate_workspace_size(w.m, w.n, w.k, cfg["id"]), dtype=torch.uint8,
                     device=Ad.device)

    def step(events=None):
        oz.ozaki25_dgemm_accurate(Ad, Bd, Cd, subtract=w.subtract, workspace=ws, stage_events=events,
                                  set=cfg["id"], quantiser=quant)

    if C0d is not None:
        Cd.copy_(C0d)
    for _ in range(warmup):
        step()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(oz.NUM_STAGE_EVENTS)] for _ in range(steps)]
    for row in ev:
        for e in row:
            e.record()
    torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for i in range(steps):
        step(ev[i])
    end.record()
    torch.cuda.synchronize()
    ms = start.elapsed_time(end) / steps
    stage = np.array([[row[j].elapsed_time(row[j + 1]) for j in range(oz.NUM_STAGE_EVENTS - 1)] for row in ev])
    del ws
    st = stage.mean(axis=0).tolist()
    return {"ms_per_step": round(ms, 4), "value": round(w.flops / (ms * 1e-3) / 1e12, 3), "unit": "TFLOPS",
            "stage_ms": dict(zip(("exponents", "deconstruct", "residue_gemm", "reconstruct"),
                                 [round(x, 4) for x in st])),
            "note": "ozaki25_dgemm_accurate: per-row/column shifts from the int8 magnitude-bound "
                    "product (one extra product) instead of the fixed t(k)"}


def time_planes(oz, torch, w, Ad, Bd, Cd, cfg, steps, quant):
    """Storage mode P: ms per ozaki25_dgemm_planes call on planes made once."""
    planesA, expsA = oz.ozaki25_deconstruct(0, Ad, set=cfg["id"], quantiser=quant)
    planesB, expsB = oz.ozaki25_deconstruct(1, Bd, set=cfg["id"], quantiser=quant)
    ws = torch.empty(oz.ozaki25_dgemm_planes_workspace_size(w.m, w.n, w.k, cfg["id"]), dtype=torch.uint8,
                     device=Ad.device)

    def step():
        oz.ozaki25_dgemm_planes(w.k, planesA, expsA, planesB, expsB, Cd, subtract=w.subtract,
                                workspace=ws, set=cfg["id"])

    step()
    torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(steps):
        step()
    end.record()
    torch.cuda.synchronize()
    ms = start.elapsed_time(end) / steps
    del planesA, planesB, ws
    return ms


def time_graph(oz, torch, w, Ad, Bd, Cd, cfg, steps, quant):
    """ms per replay of a HIP graph that captured one ozaki25_dgemm_ex call
    (caller workspace: the call enqueues kernels only)."""
    ws = torch.empty(oz.ozaki25_dgemm_workspace_size(w.m, w.n, w.k, cfg["id"]), dtype=torch.uint8,
                     device=Ad.device)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        oz.ozaki25_dgemm_ex(Ad, Bd, Cd, subtract=w.subtract, workspace=ws, set=cfg["id"], quantiser=quant)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        oz.ozaki25_dgemm_ex(Ad, Bd, Cd, subtract=w.subtract, workspace=ws, set=cfg["id"], quantiser=quant)
    g.replay()
    torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(steps):
        g.replay()
    end.record()
    torch.cuda.synchronize()
    ms = start.elapsed_time(end) / steps
    del g, ws
    return ms


def fused(w):
    """Storage mode F for A (the library's choice for at most 128 columns and
    at least 1024 rows): A is quantised inside the product kernel, so there
    is no deconstruction stage to price against HBM."""
    return w.n <= 128 and w.m >= 1024


def rates(w, cfg, ms, stages):
    scan_ms, dec_ms, gemm_ms, rec_ms = stages
    elems = w.m * w.k + w.k * w.n
    dec_bytes = elems * (8 + cfg["plane_bytes"])
    rec_bytes = w.m * w.n * (cfg["cres_bytes"] + 8 + (8 if w.subtract else 0))
    gemm_ops = 2.0 * (cfg["fused_products"] if fused(w) else cfg["products"]) * w.m * w.n * w.k
    return dict(tflops=w.flops / (ms * 1e-3) / 1e12, gemm_ops=gemm_ops,
                gemm_tops=gemm_ops / (gemm_ms * 1e-3) / 1e12, dec_bytes=dec_bytes,
                dec_gbs=dec_bytes / (dec_ms * 1e-3) / 1e9,
                stage_gbs=(dec_bytes + elems * 8) / ((dec_ms + scan_ms) * 1e-3) / 1e9,
                rec_gbs=rec_bytes / (rec_ms * 1e-3) / 1e9,
                roof=cfg["peak"] / cfg["products"])


def dec_roofline(w, cfg, rt, moduli, scan_ms, dec_ms):
    if fused(w):
        return {"bound": "hbm", "kernel": None, "achieved": None, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": None, "bytes_per_call": None,
                "note": "storage mode F for A: no planes of A are made (the product kernel " + cfg["fused_kernel"]
                        + " quantises A); the scan stage holds A's exponent scan, the deconstruct stage B's"}
    return {"bound": "hbm", "kernel": cfg["dec_kernel"], "achieved": round(rt["dec_gbs"], 1),
            "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(rt["dec_gbs"] / HBM_PEAK_GBS, 4),
            "bytes_per_call": rt["dec_bytes"], "stage_with_scan_gbs": round(rt["stage_gbs"], 1),
            **measured_deconstruction(w, moduli, scan_ms, dec_ms)}


def gemm_kernel_name(w, cfg):
    """The residue GEMM kernel the library launches for this shape: the
    compact product of either set takes its persistent form (one block per
    CU walking tiles) at short k, an even count of at most 16 K stages of
    128, with at least two output tiles per CU (512 x 128 tiles for n <= 128,
    256 x 256 otherwise, per modulus)."""
    import torch
    nstage = -(-w.k // 128)
    bm, bn = (512, 128) if w.n <= 128 else (256, 256)
    tiles = cfg["r"] * -(-w.m // bm) * -(-w.n // bn)
    cus = torch.cuda.get_device_properties(0).multi_processor_count // 8 * 8
    if 2 <= nstage <= 16 and nstage % 2 == 0 and cus >= 8 and tiles >= 2 * cus:
        return cfg["persistent_kernel"]
    return cfg["gemm_kernel"]


def gemm_roofline(w, cfg, rt, moduli):
    unit = "TFLOP/s" if cfg["dtype"] == "fp8" else "TOP/s"
    r = {"bound": "mfma", "kernel": cfg["fused_kernel"] if fused(w) else gemm_kernel_name(w, cfg),
         "achieved": round(rt["gemm_tops"], 2), "peak": cfg["peak"], "unit": unit,
         "frac": round(rt["gemm_tops"] / cfg["peak"], 4),
         "traffic": None if fused(w) else measured_traffic(w, moduli), "ops_per_launch": rt["gemm_ops"],
         "note": cfg["note"]}
    if fused(w):
        r["note"] = (f"storage mode F: {cfg['fused_products']} products x 2mnk per launch, in units of the "
                     "peak's dtype (the published set: 3 e4m3 digit products per square modulus and one fp16 "
                     "residue product per nonsquare one, counted twice as fp16 runs at half the fp8 rate); "
                     "the kernel is bound by converting A (VALU), not by the matrix cores")
    return r


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="square", choices=sorted(workloads.WORKLOADS))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-native", action="store_true")
    ap.add_argument("--baseline-rows", type=int, default=4096,
                    help="rows of A in the oracle's timed sample (all of them when fewer)")
    ap.add_argument("--baseline-cols", type=int, default=1024,
                    help="columns of B in the oracle's timed sample (all of them when fewer)")
    ap.add_argument("--calibration-copy", action="store_true",
                    help="copy 1 GiB device to device once before the run (a known-size kernel "
                         "for scaling rocprofv3 FETCH_SIZE / WRITE_SIZE counters)")
    ap.add_argument("--moduli", default="s12", choices=sorted(SETS),
                    help="modulus set of the headline line (the other one is reported alongside)")
    ap.add_argument("--only", action="store_true", help="time the headline modulus set only")
    ap.add_argument("--quantiser", default="rn", choices=["rn", "tz"],
                    help="quantiser of Eq. (scale): round to nearest (default) or toward zero")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py runs on one GPU only; --gpus {args.gpus} is not supported "
              "(the emulated DGEMM shards by output panels, but this build measures one GPU)",
              file=sys.stderr)
        return 2

    import torch
    import paper_2609_09095_amd as oz
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 2
    oz.lib()

    w = workloads.WORKLOADS[args.workload]
    log(f"[bench] generating {w.name} inputs m={w.m} n={w.n} k={w.k} s={w.s}")
    A, B, C0 = workloads.make_inputs(w)
    dev = torch.device("cuda:0")
    Ad = torch.from_numpy(A).to(dev)
    Bd = torch.from_numpy(B).to(dev)
    C0d = torch.from_numpy(C0).to(dev) if C0 is not None else None
    Cd = C0d.clone() if C0d is not None else torch.empty((w.m, w.n), dtype=torch.float64, device=dev)
    torch.cuda.synchronize()

    if args.calibration_copy:
        src = torch.ones(1 << 27, dtype=torch.float64, device=dev)   # 1 GiB
        dst = torch.empty_like(src)
        torch.mul(src, 1.0, out=dst)   # an elementwise kernel: 1 GiB in, 1 GiB out
        torch.cuda.synchronize()
        del src, dst
        log("[bench] calibration copy: 1 GiB read, 1 GiB written")

    cfg = SETS[args.moduli]
    quant = oz.TZ if args.quantiser == "tz" else oz.RN
    log(f"[bench] {cfg['moduli']}: warmup {args.warmup}, timing {args.steps} steps")
    ms, stages, ms_median = time_set(oz, torch, w, Ad, Bd, Cd, cfg, args.steps, args.warmup, quant)
    scan_ms, dec_ms, gemm_ms, rec_ms = stages
    rt = rates(w, cfg, ms, stages)
    log(f"[bench] {ms:.3f} ms/step; scan {scan_ms:.3f} deconstruct {dec_ms:.3f} gemm {gemm_ms:.3f} "
        f"reconstruct {rec_ms:.3f} ms")

    other = None
    if not args.only:
        name = "a15" if args.moduli == "s12" else "s12"
        ocfg = SETS[name]
        if C0d is not None:
            Cd.copy_(C0d)
        log(f"[bench] {ocfg['moduli']}: warmup {args.warmup}, timing {args.steps} steps")
        oms, ostages, _ = time_set(oz, torch, w, Ad, Bd, Cd, ocfg, args.steps, args.warmup, quant)
        ort = rates(w, ocfg, oms, ostages)
        log(f"[bench] {oms:.3f} ms/step; stages {[round(x, 3) for x in ostages]}")
        other = {
            "moduli": ocfg["moduli"], "route": ocfg["route"], "dtype": ocfg["dtype"],
            "value": round(ort["tflops"], 3), "unit": "TFLOPS", "ms_per_step": round(oms, 4),
            "stage_ms": dict(zip(("scan", "deconstruct", "residue_gemm", "reconstruct"),
                                 [round(x, 4) for x in ostages])),
            "roofline": gemm_roofline(w, ocfg, ort, name),
            "roofline_deconstruct": dec_roofline(w, ocfg, ort, name, ostages[0], ostages[1]),
            "emulation_roof_tflops": round(ort["roof"], 2),
            "emulation_roof_frac": round(ort["tflops"] / ort["roof"], 4),
        }
        if C0d is not None:
            Cd.copy_(C0d)
        pms = time_planes(oz, torch, w, Ad, Bd, Cd, ocfg, args.steps, quant)
        other["stored_planes"] = {"ms_per_call": round(pms, 4), "value": round(w.flops / (pms * 1e-3) / 1e12, 3),
                                  "unit": "TFLOPS"}
        log(f"[bench] {ocfg['moduli']}: accurate mode")
        other["accurate_mode"] = time_accurate(oz, torch, w, Ad, Bd, Cd, C0d, ocfg, args.steps, args.warmup,
                                               quant)

    if C0d is not None:
        Cd.copy_(C0d)
    log("[bench] stored planes (mode P)")
    pms = time_planes(oz, torch, w, Ad, Bd, Cd, cfg, args.steps, quant)
    log(f"[bench] {cfg['moduli']}: accurate mode")
    acc = time_accurate(oz, torch, w, Ad, Bd, Cd, C0d, cfg, args.steps, args.warmup, quant)
    log(f"[bench] accurate mode {acc['ms_per_step']:.3f} ms/step; stages {acc['stage_ms']}")
    if C0d is not None:
        Cd.copy_(C0d)
    log("[bench] graph replay")
    gms = time_graph(oz, torch, w, Ad, Bd, Cd, cfg, args.steps, quant)

    native = None
    vendor = None
    if not args.no_native:
        log("[bench] native FP64 " + ("addmm (C - A.B)" if w.subtract else "matmul"))
        if w.subtract:
            Cn = C0d.clone()
            fn = lambda: torch.addmm(C0d, Ad, Bd, beta=1.0, alpha=-1.0, out=Cn)  # noqa: E731
        else:
            Cn = torch.empty((w.m, w.n), dtype=torch.float64, device=dev)
            fn = lambda: torch.matmul(Ad, Bd, out=Cn)  # noqa: E731
        fn()
        torch.cuda.synchronize()
        reps = 3 if w.flops > 1e11 else 20
        s0, s1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        fn()  # untimed: the GPU is busy when the start event is reached
        s0.record()
        for _ in range(reps):
            fn()
        s1.record()
        torch.cuda.synchronize()
        native = w.flops / (s0.elapsed_time(s1) / reps * 1e-3) / 1e12
        del Cn
        log("[bench] vendor low-precision GEMM on one residue product's shape")
        vendor = vendor_lowp_gemm(torch, w, cfg, args.steps)
        if vendor.get("achieved"):
            per_product = rt["gemm_tops"]
            vendor["residue_gemm_over_vendor"] = round(per_product / vendor["achieved"], 4)

    result = {
        "metric": "emulated FP64 TFLOPS (2mnk/s) + deconstruction GB/s vs HBM/MFMA roofs",
        "value": round(rt["tflops"], 3),
        "unit": "TFLOPS",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "ms_per_step_median": round(ms_median, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg["dtype"],
        "data": "synthetic",
        "config": {"workload": f"{w.name}: C {'-=' if w.subtract else '='} A.B, m={w.m} n={w.n} k={w.k}, "
                               f"entries (U-0.5)exp({w.s} N), seed {w.seed}",
                   "m": w.m, "n": w.n, "k": w.k, "moduli": cfg["moduli"], "quantiser": args.quantiser.upper(),
                   "route": cfg["route"]},
        "roofline": gemm_roofline(w, cfg, rt, args.moduli),
        "roofline_deconstruct": dec_roofline(w, cfg, rt, args.moduli, scan_ms, dec_ms),
        "roofline_reconstruct": {"bound": "hbm", "achieved": round(rt["rec_gbs"], 1), "peak": HBM_PEAK_GBS,
                                 "unit": "GB/s", "frac": round(rt["rec_gbs"] / HBM_PEAK_GBS, 4)},
        "stage_ms": {"scan": round(scan_ms, 4), "deconstruct": round(dec_ms, 4), "residue_gemm": round(gemm_ms, 4),
                     "reconstruct": round(rec_ms, 4)},
        "emulation_roof_tflops": round(rt["roof"], 2),
        "emulation_roof_frac": round(rt["tflops"] / rt["roof"], 4),
        "stored_planes": {"ms_per_call": round(pms, 4), "value": round(w.flops / (pms * 1e-3) / 1e12, 3),
                          "unit": "TFLOPS",
                          "note": "storage mode P: ozaki25_dgemm_planes on planes deconstructed once "
                                  "(residue products + reconstruction per call)"},
        "accurate_mode": acc,
        "graph_replay": {"ms_per_call": round(gms, 4), "value": round(w.flops / (gms * 1e-3) / 1e12, 3),
                         "unit": "TFLOPS",
                         "note": "one ozaki25_dgemm_ex call captured in a HIP graph, replayed"},
        "native_fp64_tflops": round(native, 2) if native else None,
        "vendor_lowp_gemm": vendor,
        "native_fp64_peak_tflops": FP64_PEAK_TFLOPS,
        "paper_context": "modelled Rubin projections (no measurement in the paper): 473 TFLOPS roof, 182-235 TFLOPS floors",
    }
    if other is not None:
        result["all_byte_set" if args.moduli == "s12" else "published_set"] = other
    del Ad, Bd, Cd, C0d
    torch.cuda.empty_cache()
    if not args.no_cpu_baseline:
        rows = min(args.baseline_rows, w.m)
        cols = min(args.baseline_cols, w.n)
        log(f"[bench] cpu baseline: oracle on {rows}x{cols} outputs")
        result["cpu_baseline"] = cpu_baseline(A, B, w, rows, cols, cfg)
    else:
        result["cpu_baseline"] = None
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
