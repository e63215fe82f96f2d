#!/usr/bin/env python3
"""LoRA-linear forward + backward throughput on one MI355X.

One step = lora_linear_fwd + lora_linear_bwd (the whole path: fused forward
GEMM, dU, dB and dA token reductions, dX GEMM, finalize) for every projection
of the workload -- by default the three Llama-2-7B shapes (q_proj 2048 x 4096
x 4096 r 8, up_proj 4096 x 11008 x 4096 r 16, down_proj 8192 x 4096 x 11008
r 64) back to back -- on synthetic bf16 inputs.  Inputs are resident in HBM
before timing starts; when one step's operands fit the 256 MB Infinity Cache,
successive steps rotate over several copies so every step reads from HBM.

Prints one JSON line: whole-job TFLOP/s (algorithmic flops 4mnk + 6mr(n+k) per
projection), the fraction of the bf16 dense matrix-core peak, per-projection
forward and backward call times, the host's enqueue time per step (one step
into an idle stream; and over the timed loop, where a full launch queue makes
it follow the GPU time), a roofline
entry for the dominant kernel (the forward call of the projection with the
most forward flops, timed live with HIP events on its stream; its kernels come
from the library's own launch plan) and the fp64 CPU oracle's throughput on
the host as a baseline.  With --dropout P a step is the *_dropout entry
points instead, each projection's keep mask drawn afresh on the device
(lora_dropout_keep_mask) at the top of the step, inside the timed region.
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

PEAK_BF16_TFLOPS = 2500.0    # MI355X dense bf16 matrix-core peak
PEAK_HBM_GBS = 8000.0        # MI355X HBM3E
MALL_BYTES = 256 << 20       # Infinity Cache
KERNEL_SOURCES = ["paper_2403_11366_amd/csrc/lora_fwd.hip", "paper_2403_11366_amd/csrc/lora_device.hpp",
                  "paper_2403_11366_amd/csrc/lora_plan.hpp", "paper_2403_11366_amd/csrc/lora_launch.hpp"]


def forward_plan(s, dropout: bool = False):
    """The forward launches the library makes for shape s (its own plan query)."""
    import paper_2403_11366_amd as lora
    return lora.lora_linear_plan("fwd_dropout" if dropout else "fwd", s.m, s.n, s.k, s.r)


def short_kernel(name: str) -> str:
    """'lora::lora_fwd_kernel<...>' -> 'lora_fwd_kernel'."""
    return name.split("::")[-1].split("<")[0]


def dominant_shape(shapes):
    """The projection whose forward GEMM has the most flops: its forward call is
    the roofline entry of a multi-projection step."""
    return max(shapes, key=lambda s: 2 * s.m * s.n * s.k + 2 * s.m * s.k * s.r + 2 * s.m * s.n * s.r)


def traffic_file(workload: str) -> str:
    """Committed HBM-traffic record of the forward call of the dominant shape of `workload`."""
    from lora_synth import CONFIGS
    s0 = dominant_shape(CONFIGS[workload])
    kname = short_kernel(forward_plan(s0)[-1]["kernel"])
    return os.path.join(ROOT, "profiles", f"{kname}_{s0.name}_traffic.json")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_source_hash() -> str:
    """Hash of the forward kernel's sources with comments and blank space
    removed, so that only a change of the code itself retires a traffic
    record."""
    import re
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel)) as f:
            text = f.read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        h.update(" ".join(text.split()).encode())
    return h.hexdigest()[:16]


def measured_traffic(workload: str):
    """HBM bytes per forward call of the dominant shape from the committed
    rocprofv3 counter runs, if they were taken on the current kernel source;
    else None."""
    try:
        with open(traffic_file(workload)) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("kernel_source_sha") != kernel_source_hash():
        return None
    return rec.get("hbm_bytes_per_launch")


def summarize_traffic(root: str, workload: str, copy_mib: int):
    """Turn four rocprofv3 --pmc runs into HBM bytes per forward call of the
    dominant shape of `workload` (the sum over the call's kernels).

    root/{fwd_fetch,fwd_write,copy_fetch,copy_write}/ hold the counter CSVs of
    `--only fwd` and `--only copy` runs with FETCH_SIZE and WRITE_SIZE (KiB per
    dispatch).  Each forward reading is scaled by known/measured for a plain
    copy of copy_mib MiB (which reads and writes exactly that many bytes)."""
    import csv
    import glob

    def per_dispatch(sub, counter, name_part):
        vals = {}
        for f in glob.glob(os.path.join(root, sub, "**", "*counter_collection.csv"), recursive=True):
            for r in csv.DictReader(open(f)):
                if r["Counter_Name"] == counter and name_part in r["Kernel_Name"]:
                    vals[r["Dispatch_Id"]] = vals.get(r["Dispatch_Id"], 0.0) + float(r["Counter_Value"])
        if not vals:
            raise SystemExit(f"no {counter} rows for {name_part} under {root}/{sub}")
        v = sorted(vals.values())
        return v[len(v) // 2], len(v)

    from lora_synth import CONFIGS
    s0 = dominant_shape(CONFIGS[workload])
    kernels = [x["kernel"] for x in forward_plan(s0)]
    f_fwd = w_fwd = 0.0
    counts = []
    for kname in kernels:
        fv, nf = per_dispatch("fwd_fetch", "FETCH_SIZE", kname)
        wv, nw = per_dispatch("fwd_write", "WRITE_SIZE", kname)
        f_fwd, w_fwd = f_fwd + fv, w_fwd + wv
        counts.append([nf, nw])
    f_cpy, _ = per_dispatch("copy_fetch", "FETCH_SIZE", "")
    w_cpy, _ = per_dispatch("copy_write", "WRITE_SIZE", "")
    known_kib = copy_mib * 1024.0
    sf, sw = known_kib / f_cpy, known_kib / w_cpy
    fetch_b = f_fwd * sf * 1024.0
    write_b = w_fwd * sw * 1024.0
    rec = {"workload": workload, "shape": s0.name, "kernels": kernels, "kernel_source_sha": kernel_source_hash(),
           "fetch_kib_raw": f_fwd, "write_kib_raw": w_fwd, "copy_mib": copy_mib,
           "copy_fetch_kib_raw": f_cpy, "copy_write_kib_raw": w_cpy,
           "fetch_scale": sf, "write_scale": sw,
           "hbm_fetch_bytes_per_launch": fetch_b, "hbm_write_bytes_per_launch": write_b,
           "hbm_bytes_per_launch": fetch_b + write_b, "dispatches": counts}
    out = traffic_file(workload)
    os.makedirs(os.path.dirname(out), exist_ok=True)
    with open(out, "w") as f:
        json.dump(rec, f, indent=1)
    print(json.dumps(rec))


def algorithmic_units(s, launch):
    """(unit, amount) of one launch of shape s: flops for the matrix-core GEMMs,
    bytes for the HBM-bound kernels (the algorithmic minimum: each operand read
    once, each output written once; split-K partial traffic not credited)."""
    m, n, k, r = s.m, s.n, s.k, s.r
    name = launch["kernel"]
    c0, c1 = launch["cols"]
    if "lora_fwd_kernel" in name or "lora_fwd_ks_kernel" in name:
        cols = c1 - c0
        upre = name.startswith("lora::lora_fwd_kernel") and name.split(",")[6].strip() == "true"
        u = 0 if (upre or c0 > 0) else 2 * m * k * r
        return "flop", 2 * m * cols * k + 2 * m * cols * r + u
    if "lora_bwd_dx_kernel" in name:
        return "flop", 2 * m * (n + r) * (c1 - c0)
    if "lora_u_kernel" in name:
        return "byte", 2 * m * k + 2 * r * k + 4 * m * r
    if "lora_bwd_du_kernel" in name or "lora_bwd_du_dma_kernel" in name:
        return "byte", 2 * m * n + 2 * n * r + 4 * m * r
    if "lora_tokred_kernel" in name or "lora_tokred_dma_kernel" in name:
        return "byte", (2 * m * n + 4 * m * r + 4 * n * r) + (2 * m * k + 4 * m * r + 4 * r * k)
    return None, None


def summarize_counters(root: str, workload: str, copy_mib: int):
    """Per-kernel table from rocprofv3 runs of one single-projection workload
    under root/: trace/ (--kernel-trace --stats), fetch/ and write/ (--pmc
    FETCH_SIZE, WRITE_SIZE), mfma/ (--pmc SQ_VALU_MFMA_BUSY_CYCLES
    SQ_BUSY_CYCLES GRBM_GUI_ACTIVE SQ_INSTS_MFMA), lds/ (--pmc SQ_INSTS_LDS
    SQ_LDS_BANK_CONFLICT SQ_LDS_IDX_ACTIVE), copy_fetch/ and copy_write/ (the
    copy of copy_mib MiB that calibrates FETCH_SIZE and WRITE_SIZE).  Prints
    markdown: per kernel of the workload's plan, its average duration, the
    algorithmic rate against its roofline, the counter-measured HBM bytes and
    rate, and matrix-core and LDS figures."""
    import csv
    import glob
    from lora_synth import CONFIGS
    (s,) = CONFIGS[workload]

    def rows(sub, pattern):
        out = []
        for f in glob.glob(os.path.join(root, sub, "**", pattern), recursive=True):
            out += list(csv.DictReader(open(f)))
        return out

    def counter(sub, name, kname):
        per = {}
        for r_ in rows(sub, "*counter_collection.csv"):
            if r_["Counter_Name"] == name and kname in r_["Kernel_Name"]:
                per[r_["Dispatch_Id"]] = per.get(r_["Dispatch_Id"], 0.0) + float(r_["Counter_Value"])
        if not per:
            return None
        v = sorted(per.values())
        return v[len(v) // 2]

    durations = {}
    for r_ in rows("trace", "*kernel_stats.csv"):
        nm = r_["Name"][5:] if r_["Name"].startswith("void ") else r_["Name"]
        durations[nm] = (int(r_["Calls"]), float(r_["AverageNs"]) / 1e3)

    def duration(kname):
        hits = [(c, d) for nm, (c, d) in durations.items() if nm.startswith(kname + "(") or nm == kname]
        return hits[0] if hits else (0, None)

    f_cpy, w_cpy = counter("copy_fetch", "FETCH_SIZE", ""), counter("copy_write", "WRITE_SIZE", "")
    sf = copy_mib * 1024.0 / f_cpy if f_cpy else None
    sw = copy_mib * 1024.0 / w_cpy if w_cpy else None
    import paper_2403_11366_amd as lora
    launches = lora.lora_linear_plan("fwd", s.m, s.n, s.k, s.r) + lora.lora_linear_plan("bwd", s.m, s.n, s.k, s.r)
    print(f"| kernel | calls | avg us | algorithmic | rate | of peak | HBM bytes (counters) | HBM GB/s "
          f"| MFMA flops executed / algorithmic | MFMA busy | shader clock | LDS bank conflicts / LDS instr |")
    print("|---|---|---|---|---|---|---|---|---|---|---|---|")
    for x in launches:
        kname = x["kernel"]
        calls, us = duration(kname)
        unit, amount = algorithmic_units(s, x)
        rate = frac = None
        if us and unit == "flop":
            rate = amount / (us * 1e-6) / 1e12
            frac = rate / PEAK_BF16_TFLOPS
        elif us and unit == "byte":
            rate = amount / (us * 1e-6) / 1e9
            frac = rate / PEAK_HBM_GBS
        fb, wb = counter("fetch", "FETCH_SIZE", kname), counter("write", "WRITE_SIZE", kname)
        hbm = (fb * sf + wb * sw) * 1024.0 if (fb is not None and wb is not None and sf and sw) else None
        mfma = counter("mfma", "SQ_VALU_MFMA_BUSY_CYCLES", kname)
        mops = counter("mfma", "SQ_INSTS_VALU_MFMA_MOPS_BF16", kname)
        busy = counter("mfma", "GRBM_GUI_ACTIVE", kname)
        lds_i, lds_c = counter("lds", "SQ_INSTS_LDS", kname), counter("lds", "SQ_LDS_BANK_CONFLICT", kname)
        # GRBM_GUI_ACTIVE reads as the sum over the 8 XCDs of their busy cycles;
        # SQ_VALU_MFMA_BUSY_CYCLES as the sum over all 1024 SIMDs of the cycles
        # their matrix pipe is busy (32 per 32x32x16 bf16 instruction).  Busy
        # fraction: per-SIMD matrix-pipe cycles over the per-XCD busy cycles.
        mfma_pct = 100.0 * mfma / (busy / 8 * 1024) if (mfma and busy) else None
        # (GRBM_GUI_ACTIVE also counts the dispatch's ramp: a clock only for long kernels)
        clock = busy / 8 / (us * 1e-6) / 1e9 if (busy and us and us > 100) else None
        executed = mops * 512 / amount if (mops and unit == "flop") else None
        cols = "" if x["tile"] == (0, 0) else f" cols [{x['cols'][0]}, {x['cols'][1]})"
        fmt = lambda v, p: "-" if v is None else f"{v:.{p}f}"
        print(f"| `{kname}`{cols} | {calls} | {fmt(us, 2)} | {amount / 1e9:.2f} G{unit} "
              f"| {fmt(rate, 1)} {'TFLOP/s' if unit == 'flop' else 'GB/s'} | {fmt(frac, 3)} "
              f"| {fmt(None if hbm is None else hbm / 1e6, 1)} MB | {fmt(None if (hbm is None or not us) else hbm / (us * 1e-6) / 1e9, 0)} "
              f"| {fmt(executed, 3)} | {fmt(mfma_pct, 1)}% | {fmt(clock, 2)} GHz "
              f"| {fmt(None if not lds_i else lds_c / lds_i, 3)} |")


def host_cpu():
    """(threads this process may use, CPU model) of the host."""
    cores = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else (os.cpu_count() or 1)
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return cores, model


def cpu_baseline(shape, seconds: float, drop=None):
    """Time the fp64 oracle (as it stands) on this host for `shape`, on every
    core of the process's affinity mask: its plain-loop form (float64 loops
    over the index definitions, OpenMP over output rows), or with LoRA dropout
    at rate `drop` its numpy form (the loop form has no dropout variant).
    Whole forward + backward passes are repeated until `seconds` have passed."""
    import oracle
    from lora_synth import gen_inputs, gen_keep_mask
    cores, model = host_cpu()
    t = gen_inputs(shape)
    if drop is None:
        from oracle import loops
        loops.build()
        kind = "plain fp64 loops (oracle/lora_loops.c, OpenMP over output rows)"

        def one():
            loops.lora_forward_loops(t["X"], t["W"], t["A"], t["B"], shape.alpha, threads=cores)
            loops.lora_backward_loops(t["dY"], t["X"], t["W"], t["A"], t["B"], shape.alpha, threads=cores)
    else:
        keep = gen_keep_mask(shape.m, shape.k, drop, shape.seed + 1)
        kind = "numpy fp64 (one matmul per formula line)"

        def one():
            oracle.lora_forward_dropout(t["X"], t["W"], t["A"], t["B"], keep, drop, shape.alpha)
            oracle.lora_backward_dropout(t["dY"], t["X"], t["W"], t["A"], t["B"], keep, drop, shape.alpha)
    runs, t0 = 0, time.perf_counter()
    while True:
        one()
        runs += 1
        el = time.perf_counter() - t0
        if el >= seconds or runs >= 50:
            break
    per = el / runs
    return {"value": shape.flops_fwd_bwd / per / 1e12, "unit": "TFLOP/s", "cores": int(cores),
            "kind": "oracle", "cpu_model": model,
            "sample": f"{runs} full fwd+bwd of {shape.name} (m={shape.m} n={shape.n} k={shape.k} "
                      f"r={shape.r}) by the oracle's {kind}, {el:.1f} s total, {per:.2f} s each"}


def cpu_baseline_merge(shape, seconds: float):
    """Time the fp64 oracle's merge (as it stands) on this host for `shape`."""
    import oracle
    from lora_synth import gen_inputs
    threads, model = host_cpu()
    t = gen_inputs(shape)
    runs, t0 = 0, time.perf_counter()
    while True:
        oracle.lora_merge_bf16(t["W"], t["A"], t["B"], shape.alpha, 1)
        runs += 1
        el = time.perf_counter() - t0
        if el >= seconds or runs >= 50:
            break
    per = el / runs
    nbytes = 2 * 2 * shape.n * shape.k + 2 * shape.r * (shape.n + shape.k)
    return {"value": nbytes / per / 1e9, "unit": "GB/s", "cores": int(threads), "kind": "oracle", "cpu_model": model,
            "sample": f"{runs} merges of {shape.name} (n={shape.n} k={shape.k} r={shape.r}) in fp64 "
                      f"numpy/OpenBLAS with exact bf16 rounding, {el:.1f} s total, {per:.3f} s each"}


def bench_merge(args, shapes, stream):
    """Merge throughput: W_out = W + s B A for every projection of the workload,
    out of place, over rotating copies of W past the Infinity Cache.  Bytes are
    the algorithmic ones: W read, W_out written, A and B read."""
    import torch
    import paper_2403_11366_amd as lora
    from paper_2403_11366_amd.device_io import bits_to_device
    from lora_synth import gen_inputs
    dev = "cuda"
    per_set = sum(2 * 2 * s.n * s.k for s in shapes)
    nsets = max(2, math.ceil(2 * MALL_BYTES / per_set))
    proj = []
    for s in shapes:
        t = gen_inputs(s)
        W = bits_to_device(t["W"], dev)
        A, B = bits_to_device(t["A"], dev), bits_to_device(t["B"], dev)
        Ws = [W] + [W.clone() for _ in range(nsets - 1)]
        Os = [torch.empty_like(W) for _ in range(nsets)]
        proj.append((s, Ws, Os, A, B))
    torch.cuda.synchronize()

    def run(i):
        for s, Ws, Os, A, B in proj:
            lora.lora_linear_merge(Ws[i % nsets], A, B, Os[i % nsets], s.alpha, 1, stream=stream)

    for i in range(args.warmup):
        run(i)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record(stream)
    for i in range(args.steps):
        run(i)
    ev1.record(stream)
    torch.cuda.synchronize()
    us = ev0.elapsed_time(ev1) / args.steps * 1e3
    nbytes = sum(2 * 2 * s.n * s.k + 2 * s.r * (s.n + s.k) for s in shapes)
    gbs = nbytes / (us * 1e-6) / 1e9
    log(f"[bench] merge {us:.1f} us per step, {gbs:.0f} GB/s")
    cpu = None if args.no_cpu_baseline else cpu_baseline_merge(shapes[0], args.cpu_seconds)
    rec = {
        "metric": "LoRA merge W + s B A GB/s (HBM), Llama-2 projection shapes, 1 GPU",
        "value": round(gbs, 1), "unit": "GB/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(us / 1e3, 4), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": args.config, "op": "merge",
                   "projections": [{"name": s.name, "n": s.n, "k": s.k, "r": s.r, "alpha": s.alpha}
                                   for s in shapes],
                   "input_sets": nsets, "bytes_per_step": nbytes},
        "roofline": {"bound": "hbm", "kernel": "lora_merge_kernel", "achieved": round(gbs, 1),
                     "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": round(gbs / PEAK_HBM_GBS, 4),
                     "traffic": None, "bytes_per_launch": nbytes // len(shapes) if len(shapes) == 1 else None,
                     "avg_launch_us": round(us / len(shapes), 2)},
        "cpu_baseline": cpu,
    }
    print(json.dumps(rec), flush=True)


def bench_grouped(args, shapes, groups, stream):
    """Train step of a decoder layer whose projections that read one input run
    as a group (q, k, v and gate, up: lora_linear_group_fwd / _bwd, one forward
    launch and one dX launch per group); the others run alone.  Same
    algorithmic flops as the per-projection step."""
    import torch
    import paper_2403_11366_amd as lora
    from paper_2403_11366_amd.device_io import bits_to_device
    from lora_synth import gen_group_inputs
    dev = "cuda"
    per_set = sum(2 * (s.m * s.k + s.n * s.k + s.r * s.k + s.n * s.r + s.m * s.n) for s in shapes)
    nsets = max(1, math.ceil(2 * MALL_BYTES / per_set))
    log(f"[bench] {args.config} grouped {groups}: {nsets} input set(s)")
    work = []
    for members in groups:
        gs = [shapes[i] for i in members]
        s0 = gs[0]
        t = gen_group_inputs(gs)
        base = {"X": bits_to_device(t["X"], dev)}
        for key in ("W", "A", "B", "dY"):
            base[key] = [bits_to_device(v, dev) for v in t[key]]
        sets = [base] + [{key: (v.clone() if key == "X" else [x.clone() for x in v]) for key, v in base.items()}
                         for _ in range(nsets - 1)]
        ns = [s.n for s in gs]
        out = {"Y": [torch.empty((s0.m, n), dtype=torch.bfloat16, device=dev) for n in ns],
               "U": [torch.empty((s0.m, s0.r), dtype=torch.float32, device=dev) for _ in ns],
               "dX": torch.empty((s0.m, s0.k), dtype=torch.bfloat16, device=dev),
               "dA": [torch.empty((s0.r, s0.k), dtype=torch.float32, device=dev) for _ in ns],
               "dB": [torch.empty((n, s0.r), dtype=torch.float32, device=dev) for n in ns],
               "ws": torch.empty(lora.lora_linear_group_bwd_workspace_size(ns, s0.m, s0.k, s0.r),
                                 dtype=torch.uint8, device=dev)}
        work.append((gs, sets, out))
    torch.cuda.synchronize()

    def fwd(i, gs, sets, out):
        d = sets[i % len(sets)]
        lora.lora_linear_group_fwd(d["X"], d["W"], d["A"], d["B"], out["Y"], out["U"], gs[0].alpha, stream=stream)

    def bwd(i, gs, sets, out):
        d = sets[i % len(sets)]
        lora.lora_linear_group_bwd(d["dY"], d["X"], d["W"], d["A"], d["B"], out["U"], out["dX"], out["dA"],
                                   out["dB"], out["ws"], gs[0].alpha, stream=stream)

    def step(i):
        for gs, sets, out in work:
            fwd(i, gs, sets, out)
            bwd(i, gs, sets, out)

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(i)
    torch.cuda.synchronize()
    ms_per_step = (time.perf_counter() - t0) / args.steps * 1e3
    flops = sum(s.flops_fwd_bwd for s in shapes)
    tflops = flops / (ms_per_step / 1e3) / 1e12
    log(f"[bench] grouped {ms_per_step * 1e3:.1f} us/step, {tflops:.1f} TFLOP/s")
    # dominant kernel: the forward launch of the largest group, HIP events on its stream
    gi = max(range(len(work)), key=lambda j: sum(s.n for s in work[j][0]))
    gs, sets, out = work[gi]
    reps = max(20, args.steps)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record(stream)
    for i in range(reps):
        fwd(i, gs, sets, out)
    ev1.record(stream)
    torch.cuda.synchronize()
    fwd_us = ev0.elapsed_time(ev1) / reps * 1e3
    m, k, r = gs[0].m, gs[0].k, gs[0].r
    k1 = sum(2 * m * s.n * k + 2 * m * k * r + 2 * m * s.n * r for s in gs)
    achieved = k1 / (fwd_us * 1e-6) / 1e12
    rec = {
        "metric": "LoRA-linear fwd+bwd TFLOP/s + % bf16 MFMA peak, Llama-2 layer with grouped projections, 1 GPU",
        "value": round(tflops, 2), "unit": "TFLOP/s", "pct_bf16_mfma_peak": round(100 * tflops / PEAK_BF16_TFLOPS, 2),
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": args.config, "groups": [[shapes[i].name for i in g] for g in groups],
                   "input_sets": nsets, "flops_per_step": flops},
        "roofline": {"bound": "mfma", "kernel": "lora_fwd_kernel (group " + "+".join(s.name for s in gs) + ")",
                     "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(achieved / PEAK_BF16_TFLOPS, 4), "traffic": None, "flops_per_launch": k1,
                     "avg_launch_us": round(fwd_us, 2)},
        "cpu_baseline": None,
    }
    print(json.dumps(rec), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=100)
    ap.add_argument("--config", default="llama2_7b_shapes")
    ap.add_argument("--cpu-seconds", type=float, default=5.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--only", choices=["fwd", "copy"], default=None,
                    help="run only forward launches, or only a plain device copy (for counter runs)")
    ap.add_argument("--copy-mib", type=int, default=512)
    ap.add_argument("--op", choices=["train", "merge"], default="train",
                    help="train: forward + backward (the default measurement); merge: the "
                         "merge W + s B A of each projection's adapter into its weight")
    ap.add_argument("--dropout", type=float, default=None, metavar="P",
                    help="train with LoRA dropout at rate P on the adapter input (the *_dropout "
                         "entry points; each step draws a fresh keep mask on the device with "
                         "lora_dropout_keep_mask, inside the timed step)")
    ap.add_argument("--grouped", action="store_true",
                    help="run the projections that read one input (q, k, v; gate, up) as groups "
                         "(workloads with a layer grouping only)")
    ap.add_argument("--fused-bwd", action="store_true",
                    help="backward through lora_linear_bwd_fused (dU and dB inside the dX GEMM; "
                         "rank <= 16, no dropout)")
    ap.add_argument("--summarize-counters", metavar="DIR", default=None,
                    help="print the per-kernel counter table of the rocprofv3 runs under DIR and exit")
    ap.add_argument("--summarize-traffic", metavar="DIR", default=None,
                    help="write the HBM-traffic record from counter runs under DIR and exit")
    args = ap.parse_args()

    if args.summarize_counters:
        summarize_counters(args.summarize_counters, args.config, args.copy_mib)
        return
    if args.summarize_traffic:
        summarize_traffic(args.summarize_traffic, args.config, args.copy_mib)
        return

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(the LoRA linear would shard over tokens with an all-reduce of dA and dB; "
              "not built here). Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    import paper_2403_11366_amd as lora
    from lora_synth import CONFIGS, gen_inputs
    from paper_2403_11366_amd.device_io import bits_to_device

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    lora.load_library()
    if args.only == "copy":
        n = args.copy_mib << 20
        src = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(args.steps):
            dst.copy_(src)
        torch.cuda.synchronize()
        log(f"[bench] {args.steps} copies of {args.copy_mib} MiB done")
        return
    shapes = CONFIGS[args.config]
    if args.fused_bwd and (args.dropout is not None or args.grouped or any(s.r > 16 for s in shapes)):
        sys.exit("--fused-bwd: rank <= 16 without dropout or grouping only")
    dev = "cuda"
    stream = torch.cuda.current_stream()
    if args.op == "merge":
        bench_merge(args, shapes, stream)
        return
    if args.grouped:
        from lora_synth import LAYER_GROUPS
        if args.config not in LAYER_GROUPS or args.dropout is not None:
            sys.exit(f"--grouped needs a layer workload ({', '.join(LAYER_GROUPS)}) and no dropout")
        bench_grouped(args, shapes, LAYER_GROUPS[args.config], stream)
        return

    # ---- inputs resident in HBM, rotated over enough copies to exceed the MALL
    drop = args.dropout
    per_set = sum(2 * (s.m * s.k + s.n * s.k + s.r * s.k + s.n * s.r + s.m * s.n) for s in shapes)
    nsets = max(1, math.ceil(2 * MALL_BYTES / per_set))
    log(f"[bench] {args.config}: {len(shapes)} projection(s), {nsets} input set(s) of {per_set / 2**20:.0f} MiB")
    proj = []
    for s in shapes:
        t = gen_inputs(s)
        base = {key: bits_to_device(v, dev) for key, v in t.items()}
        sets = [base] + [{key: v.clone() for key, v in base.items()} for _ in range(nsets - 1)]
        out = {
            "Y": torch.empty((s.m, s.n), dtype=torch.bfloat16, device=dev),
            "U": torch.empty((s.m, s.r), dtype=torch.float32, device=dev),
            "dX": torch.empty((s.m, s.k), dtype=torch.bfloat16, device=dev),
            "dA": torch.empty((s.r, s.k), dtype=torch.float32, device=dev),
            "dB": torch.empty((s.n, s.r), dtype=torch.float32, device=dev),
            "ws": torch.empty((lora.lora_linear_bwd_fused_workspace_size if args.fused_bwd
                               else lora.lora_linear_bwd_workspace_size)(s.m, s.n, s.k, s.r),
                              dtype=torch.uint8, device=dev),
        }
        if drop is not None:   # the step's keep mask, drawn on the device at the top of each step
            out["keep"] = torch.empty((s.m, s.k // 8), dtype=torch.uint8, device=dev)
            lora.lora_dropout_keep_mask(s.seed, 0, drop, out["keep"])
        proj.append((s, sets, out))
    torch.cuda.synchronize()

    def fwd(i, s, sets, out):
        d = sets[i % len(sets)]
        if drop is not None:
            lora.lora_linear_fwd_dropout(d["X"], d["W"], d["A"], d["B"], out["keep"], drop, out["Y"], out["U"],
                                         s.alpha, stream=stream)
            return
        lora.lora_linear_fwd(d["X"], d["W"], d["A"], d["B"], out["Y"], out["U"], s.alpha, stream=stream)

    def bwd(i, s, sets, out):
        d = sets[i % len(sets)]
        if drop is not None:
            lora.lora_linear_bwd_dropout(d["dY"], d["X"], d["W"], d["A"], d["B"], out["U"], out["keep"], drop,
                                         out["dX"], out["dA"], out["dB"], out["ws"], s.alpha, stream=stream)
            return
        (lora.lora_linear_bwd_fused if args.fused_bwd else lora.lora_linear_bwd)(
            d["dY"], d["X"], d["W"], d["A"], d["B"], out["U"], out["dX"], out["dA"], out["dB"], out["ws"],
            s.alpha, stream=stream)

    def step(i):
        for s, sets, out in proj:
            if drop is not None:   # a fresh mask per step: the next m k / 8 counters of the projection's seed
                lora.lora_dropout_keep_mask(s.seed, (i + 1) * (s.m * s.k // 8), drop, out["keep"], stream=stream)
            fwd(i, s, sets, out)
            bwd(i, s, sets, out)

    if args.only == "fwd":   # counter runs: the dominant shape's forward call only
        s_dom = dominant_shape(shapes)
        for i in range(args.warmup + args.steps):
            for s_, sets_, out_ in proj:
                if s_ is s_dom:
                    fwd(i, s_, sets_, out_)
        torch.cuda.synchronize()
        log(f"[bench] {args.warmup + args.steps} forward calls of {s_dom.name} done")
        return

    # ---- whole path
    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    # host cost of enqueueing one step into an idle stream (the launches
    # return before the GPU work ends): median over 10 steps, each begun after
    # a synchronisation, so a full launch queue cannot hold the host back
    host_us = []
    for i in range(10):
        torch.cuda.synchronize()
        t_h = time.perf_counter()
        step(i)
        host_us.append((time.perf_counter() - t_h) * 1e6)
    torch.cuda.synchronize()
    host_us.sort()
    enqueue_idle_us = host_us[len(host_us) // 2]
    log(f"[bench] warmup {args.warmup} steps done; timing {args.steps} steps")
    # HIP events split the timed steps into 5 repetitions (recorded on the
    # stream, no synchronisation inside the timed region); the host clock also
    # notes when the last step has been enqueued.
    nrep = 5 if args.steps >= 5 else 1
    marks = [round(j * args.steps / nrep) for j in range(nrep + 1)]
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(nrep + 1)]
    t0 = time.perf_counter()
    evs[0].record(stream)
    for i in range(args.steps):
        step(i)
        if i + 1 in marks:
            evs[marks.index(i + 1)].record(stream)
    t_enq = time.perf_counter()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ms_per_step = elapsed / args.steps * 1e3
    enqueue_us = (t_enq - t0) / args.steps * 1e6
    rep_ms = [evs[j].elapsed_time(evs[j + 1]) / (marks[j + 1] - marks[j]) for j in range(nrep)]
    flops = sum(s.flops_fwd_bwd for s, _, _ in proj)
    tflops = flops / (ms_per_step / 1e3) / 1e12
    log(f"[bench] {ms_per_step * 1e3:.1f} us/step, {tflops:.1f} TFLOP/s (host enqueue {enqueue_us:.1f} us/step)")

    # ---- per projection: the forward and the backward call, each timed with
    # HIP events recorded on the stream they are launched on
    reps = max(20, args.steps)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    def timed(fn, s, sets, out):
        for i in range(3):
            fn(i, s, sets, out)
        ev0.record(stream)
        for i in range(reps):
            fn(i, s, sets, out)
        ev1.record(stream)
        torch.cuda.synchronize()
        return ev0.elapsed_time(ev1) / reps * 1e3

    per_shape = []
    for s, sets, out in proj:
        f_us, b_us = timed(fwd, s, sets, out), timed(bwd, s, sets, out)
        k1 = 2 * s.m * s.n * s.k + 2 * s.m * s.k * s.r + 2 * s.m * s.n * s.r
        per_shape.append({"name": s.name, "fwd_us": round(f_us, 2), "bwd_us": round(b_us, 2),
                          "tflops": round(s.flops_fwd_bwd / ((f_us + b_us) * 1e-6) / 1e12, 2),
                          "fwd_frac": round(k1 / (f_us * 1e-6) / 1e12 / PEAK_BF16_TFLOPS, 4),
                          "fwd_kernels": [x["kernel"] for x in forward_plan(s, drop is not None)],
                          "bwd_kernels": [x["kernel"] for x in lora.lora_linear_plan(
                              ("bwd_dropout" if drop is not None else "bwd_fused" if args.fused_bwd else "bwd"),
                              s.m, s.n, s.k, s.r)]})
        log(f"[bench] {s.name}: forward call {f_us:.1f} us, backward call {b_us:.1f} us")

    # ---- roofline entry: the forward call of the projection with the most
    # forward flops (one GEMM launch, or a U pass and/or two column ranges,
    # all inside the timed call, as its plan lists)
    s0 = dominant_shape([s for s, _, _ in proj])
    e0 = next(e for e in per_shape if e["name"] == s0.name)
    fwd_us = e0["fwd_us"]
    k1_flops = 2 * s0.m * s0.n * s0.k + 2 * s0.m * s0.k * s0.r + 2 * s0.m * s0.n * s0.r
    achieved = k1_flops / (fwd_us * 1e-6) / 1e12
    kernel_label = " + ".join(e0["fwd_kernels"])
    traffic = measured_traffic(args.config) if drop is None else None

    cpu = None
    if not args.no_cpu_baseline:
        c0 = min((s for s, _, _ in proj), key=lambda s: s.flops_fwd_bwd)
        log(f"[bench] timing the fp64 oracle on the host ({c0.name}, at least {args.cpu_seconds:.0f} s)")
        cpu = cpu_baseline(c0, args.cpu_seconds, drop)

    rec = {
        "metric": "LoRA-linear fwd+bwd TFLOP/s + % bf16 MFMA peak, Llama-2-7B shapes, 1 GPU"
                  + ("" if drop is None else f", LoRA dropout p={drop}"),
        "value": round(tflops, 2),
        "unit": "TFLOP/s",
        "pct_bf16_mfma_peak": round(100 * tflops / PEAK_BF16_TFLOPS, 2),
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": args.config,
                   "projections": [{"name": s.name, "m": s.m, "n": s.n, "k": s.k, "r": s.r,
                                    "alpha": s.alpha} for s in shapes],
                   "input_sets": nsets, "flops_per_step": flops, "lora_dropout": drop,
                   "backward": "lora_linear_bwd_fused" if args.fused_bwd else "lora_linear_bwd",
                   "operands": "bf16 in, fp32 accumulate; Y, dX bf16; U, dA, dB fp32"},
        "roofline": {"bound": "mfma", "kernel": kernel_label, "shape": s0.name,
                     "achieved": round(achieved, 2),
                     "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                     "traffic": traffic, "flops_per_launch": k1_flops, "avg_launch_us": round(fwd_us, 2)},
        "per_projection": per_shape,
        "host_enqueue_us_per_step": round(enqueue_idle_us, 2),
        "host_enqueue_timed_us_per_step": round(enqueue_us, 2),
        "repetitions": {"count": nrep, "ms_per_step": [round(x, 4) for x in rep_ms],
                        "median": round(sorted(rep_ms)[nrep // 2], 4),
                        "std": round((sum((x - sum(rep_ms) / nrep) ** 2 for x in rep_ms) / nrep) ** 0.5, 4)},
        "cpu_baseline": cpu,
    }
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
