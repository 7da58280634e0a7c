#!/usr/bin/env python3
"""Benchmark of the quantized linear-layer stack on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--chain]

One step = one pass of eb_qlinear_stack over every projection of every layer
of the workload (graph-replayed), with weights, activations and outputs
already resident in HBM.  The default workload is batch-1 decode of one token
through a 32-layer 7B-class stack with Q4_0 weights (4096->12288 QKV,
4096->4096 O, 4096->22016 gate+up, 11008->4096 down; fp16 activations, fp32
outputs).

With --chain (workloads with a gate/up projection) the layers run as a
dependent decoder-layer chain through one fp32 residual stream h: QKV on
RMSNorm(h), O adding into h (attention is outside the path: its output is a
seeded input per layer), gate/up on RMSNorm(h) with the SiLU-gated product,
down adding into h; every step fused into its projection's launch (section
3.2, operator fusion).

Prints ONE JSON line:
  value          whole-pass algorithmic throughput (GB/s for the bandwidth-bound
                 workloads, TFLOP/s for the prefill workloads)
  ms_per_step    milliseconds per backbone pass (HIP events around K passes)
  roofline       the dominant kernel's algorithmic rate per launch against the
                 MI355X peak: its launches are graph-replayed back to back and
                 HIP events on the launch stream give the average duration
  cpu_baseline   the CPU oracle timed on a bounded sample of the same workload
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = ("qlinear HBM GB/s (M=1) and MFMA TFLOP/s (M≥512) vs MI355X peak; "
          "ms/backbone pass")
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E
PEAK_MFMA_16BIT_TFLOPS = 2500.0  # MI355X dense bf16 / fp16 matrix
RIDGE_FLOP_PER_BYTE = PEAK_MFMA_16BIT_TFLOPS * 1e12 / (PEAK_HBM_GBS * 1e9)  # 312.5
MAX_HOST_THREADS = 16


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--warmup-seconds", type=float, default=0.5,
                    help="keep warming up until this much time has passed as well (the "
                         "GPU takes some tens of milliseconds of load to reach its "
                         "steady clock)")
    ap.add_argument("--workload", default="q4_0_decode_7b")
    ap.add_argument("--chain", action="store_true",
                    help="run the layers as a dependent decoder-layer chain with fused "
                         "RMSNorm / residual / SiLU-gate steps")
    ap.add_argument("--cpu-layers", type=int, default=None, help="layers in the oracle sample")
    ap.add_argument("--cpu-rows", type=int, default=None, help="activation rows in the oracle sample")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="oracle time the CPU baseline sample is sized to")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="BYTES",
                    help="first run a plain device-to-device copy of BYTES (for scaling "
                         "rocprofv3 FETCH_SIZE / WRITE_SIZE counters)")
    return ap.parse_args()


def weight_bytes(qtype, n, k):
    return n * (k // 32) * (34 if qtype == "q8_0" else 18)


def op_bytes(qtype, m, n, k):
    return weight_bytes(qtype, n, k) + 2 * m * k + 4 * m * n


def load_traffic(workload, kernel):
    """HBM bytes per launch from committed rocprofv3 counter runs
    (profiles/traffic.json, written by paper_2607_02501_amd.traffic), if they
    were taken on the current kernel sources; otherwise None."""
    from paper_2607_02501_amd.srchash import family, kernel_sources_sha

    path = os.path.join(ROOT, "profiles", "traffic.json")
    try:
        with open(path) as fh:
            rec = json.load(fh).get(workload, {}).get(kernel)
    except (OSError, ValueError):
        return None
    if not rec or rec.get("kernel_sources_sha") != kernel_sources_sha(
            family(rec.get("kernel_symbol", ""))):
        return None
    return rec.get("hbm_bytes_per_launch")


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}, WORLD_SIZE {world}): "
              "this build has no multi-GPU path; run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2607_02501_amd import eb
    from paper_2607_02501_amd import workloads as W

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    wl = W.WORKLOADS[args.workload]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.calibrate_copy:
        src = torch.ones(args.calibrate_copy // 4, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"[bench] calibration copy of {args.calibrate_copy} bytes done")
        del src, dst

    # ---- resident inputs: quantized weights, activations, outputs ----------
    t_setup = time.time()
    qws = {}
    for layer in range(wl.layers):
        for p, (_, k, n) in enumerate(wl.projections):
            w = W.weights(wl, layer, p, dev)
            qws[layer, p] = eb.quantize(w, wl.qtype)
            del w
    entries, meta = [], []
    if args.chain:
        entries, meta, chain_bytes = chain_entries(wl, W, qws, dev, torch)
    else:
        for step in range(wl.steps):
            for layer in range(wl.layers):
                for p, (pname, k, n) in enumerate(wl.projections):
                    x = W.activations(wl, layer, p, dev, step=step)
                    y = torch.empty((wl.m, n), dtype=torch.float32, device=dev)
                    entries.append((qws[layer, p], x, y))
                    meta.append((pname, wl.m, n, k))
    ops = eb.make_ops(entries)
    torch.cuda.synchronize()
    log(f"[bench] {wl.name}{' chain' if args.chain else ''}: {len(entries)} ops per pass, "
        f"{eb.stack_launches(ops)} launches per pass, setup {time.time() - t_setup:.1f}s")

    bytes_pass = chain_bytes if args.chain else sum(op_bytes(wl.qtype, m, n, k) for (_, m, n, k) in meta)
    wbytes_pass = sum(weight_bytes(wl.qtype, n, k) for (_, m, n, k) in meta)
    flops_pass = sum(2 * m * n * k for (_, m, n, k) in meta)
    mfma_bound = wl.m >= 512

    # ---- timed region: K graph-replayed passes -----------------------------
    warm, t_warm = 0, time.time()
    while warm < args.warmup or time.time() - t_warm < args.warmup_seconds:
        eb.qlinear_stack(ops)
        warm += 1
        if warm % 8 == 0:
            torch.cuda.synchronize()
    torch.cuda.synchronize()
    args.warmup = warm
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(args.steps):
        eb.qlinear_stack(ops)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    log(f"[bench] timed {args.steps} passes: {ms:.4f} ms/pass")

    if args.chain:
        finish_chain(args, wl, W, dev, ops, entries, meta, bytes_pass, wbytes_pass, flops_pass, ms,
                     mfma_bound, eb, torch)
        return

    # ---- per-kernel durations ------------------------------------------------
    # Ops that run the same kernel instance (same path, formats, m and k) form
    # one stack, graph-replayed back to back (independent m == 1 ops become one
    # fused launch); HIP events on the launch stream bracket `reps` replays, so
    # the average launch duration excludes host launch cost and agrees with
    # rocprofv3's per-kernel average.
    groups = {}
    for ent, (pname, m, n, k) in zip(entries, meta):
        key = (eb.auto_path(wl.qtype, wl.x_dtype, m, n, k), m, k)
        groups.setdefault(key, []).append((ent, m, n, k))
    kinds = {}
    for key, items in groups.items():
        gops = eb.make_ops([e for e, *_ in items])
        for _ in range(2):
            eb.qlinear_stack(gops)
        torch.cuda.synchronize()
        reps = max(3, min(50, 2000 // len(items)))
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            eb.qlinear_stack(gops)
        b.record()
        torch.cuda.synchronize()
        kinds[key] = {"ms": a.elapsed_time(b) / reps, "launches": eb.stack_launches(gops),
                      "ops": len(items),
                      "bytes": sum(op_bytes(wl.qtype, m, n, k) for _, m, n, k in items),
                      "flops": sum(2 * m * n * k for _, m, n, k in items)}
    eb.stack_cache_clear()
    dom = max(kinds, key=lambda p: kinds[p]["ms"])
    dk = kinds[dom]
    avg_ms = dk["ms"] / dk["launches"]
    path = dom[0]
    kernel_name = f"{path}_{wl.qtype}_{'f16' if wl.x_dtype == torch.float16 else 'bf16'}_m{dom[1]}_k{dom[2]}"
    for p, d in kinds.items():
        log(f"[bench] kernel {p}: {d['ops']} ops in {d['launches']} launches/pass, "
            f"avg {1e3 * d['ms'] / d['launches']:.2f} us, "
            f"{d['bytes'] / d['ms'] / 1e6:.1f} GB/s, {d['flops'] / d['ms'] / 1e9:.2f} TFLOP/s")
    # the roofline that bounds a kernel is set by its arithmetic intensity,
    # not by which path runs it (m = 50 on the MFMA path is HBM-bound)
    if dk["flops"] / dk["bytes"] > RIDGE_FLOP_PER_BYTE:
        achieved = dk["flops"] / dk["launches"] / (avg_ms * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_MFMA_16BIT_TFLOPS,
                "unit": "TFLOP/s", "frac": round(achieved / PEAK_MFMA_16BIT_TFLOPS, 4)}
    else:
        achieved = dk["bytes"] / dk["launches"] / (avg_ms * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBS, 4)}
    roof["kernel"] = kernel_name
    roof["avg_launch_us"] = round(avg_ms * 1e3, 3)
    roof["launches_per_pass"] = dk["launches"]
    roof["ops_per_launch"] = dk["ops"] / dk["launches"]
    roof["algorithmic_per_launch"] = (dk["flops"] if roof["bound"] == "mfma" else dk["bytes"]) // dk["launches"]
    roof["traffic"] = load_traffic(wl.name, kernel_name)

    if mfma_bound:
        value, unit = flops_pass / (ms * 1e-3) / 1e12, "TFLOP/s"
    else:
        value, unit = bytes_pass / (ms * 1e-3) / 1e9, "GB/s"

    # ---- CPU oracle on a bounded sample ------------------------------------
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(args, wl, W, dev, mfma_bound)

    out = {
        "metric": METRIC, "value": round(value, 2), "unit": unit, "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": f"{wl.qtype} weights x {'f16' if wl.x_dtype == torch.float16 else 'bf16'} "
                 "activations, f32 accumulate",
        "data": "synthetic (seeded N(0,0.02) weights, N(0,1) activations)",
        "config": {"workload": wl.name, "m": wl.m, "layers": wl.layers, "steps": wl.steps,
                   "ops_per_pass": len(entries), "weight_bytes_per_pass": wbytes_pass,
                   "algorithmic_bytes_per_pass": bytes_pass, "flops_per_pass": flops_pass,
                   "graph_replay": os.environ.get("EB_STACK_GRAPH", "1") != "0",
                   "output": "f32"},
        "roofline": roof,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


def chain_entries(wl, W, qws, dev, torch):
    """Stack entries of the dependent decoder-layer chain (see the module
    docstring) and its algorithmic bytes per pass: weights, the residual
    stream read by each normalisation and residual addition and written by
    each addition, the attention stand-in, the QKV and gated outputs and
    their re-reads, the normalisation weights."""
    names = [p[0] for p in wl.projections]
    if names[2] != "gate_up":
        raise SystemExit(f"--chain needs a gate/up projection; {wl.name} has {names}")
    (_, d, n_qkv), _, (_, _, n_gu), (_, f, _) = wl.projections
    m, xdt = wl.m, wl.x_dtype
    xs = 2
    h = W.normal((m, d), W.seed_of(wl.wid, 4095, 15, 3), dev)
    qkv = torch.empty((m, n_qkv), dtype=xdt, device=dev)
    act = torch.empty((m, n_gu // 2), dtype=xdt, device=dev)
    entries, meta, nbytes = [], [], 0
    # normalisation weights belong to the layer (the same in every step)
    gammas = [(1.0 + 0.1 * W.normal((d,), W.seed_of(wl.wid, layer, 0, 2), dev),
               1.0 + 0.1 * W.normal((d,), W.seed_of(wl.wid, layer, 2, 2), dev))
              for layer in range(wl.layers)]
    for step in range(wl.steps):
        for layer in range(wl.layers):
            g1, g2 = gammas[layer]
            attn = W.activations(wl, layer, 1, dev, step=step)
            entries += [
                (qws[layer, 0], h, qkv, dict(x_dtype=xdt, prologue="rmsnorm", norm_weight=g1, eps=1e-5)),
                (qws[layer, 1], attn, h, dict(epilogue="add", residual=h)),
                (qws[layer, 2], h, act, dict(x_dtype=xdt, prologue="rmsnorm", norm_weight=g2,
                                             eps=1e-5, epilogue="glu")),
                (qws[layer, 3], act, h, dict(epilogue="add", residual=h)),
            ]
            for p, (pname, k, n) in enumerate(wl.projections):
                meta.append((pname, m, n, k))
                nbytes += weight_bytes(wl.qtype, n, k)
            nbytes += (m * d * 4 + d * 4 + m * n_qkv * xs          # QKV: h, g, qkv out
                       + m * d * xs + 2 * m * d * 4                # O: attention, h read and write
                       + m * d * 4 + d * 4 + m * (n_gu // 2) * xs  # gate/up: h, g, gated out
                       + m * f * xs + 2 * m * d * 4)               # down: gated in, h read and write
    return entries, meta, nbytes


def finish_chain(args, wl, W, dev, ops, entries, meta, bytes_pass, wbytes_pass, flops_pass, ms,
                 mfma_bound, eb, torch):
    """JSON line of a chain run: the chain's launches depend on each other, so
    the roofline is the whole pass against the peak (no per-kernel groups)."""
    launches = eb.stack_launches(ops)
    eb.stack_cache_clear()
    if mfma_bound:
        value, unit = flops_pass / (ms * 1e-3) / 1e12, "TFLOP/s"
        roof = {"bound": "mfma", "achieved": round(value, 2), "peak": PEAK_MFMA_16BIT_TFLOPS,
                "unit": "TFLOP/s", "frac": round(value / PEAK_MFMA_16BIT_TFLOPS, 4)}
    else:
        value, unit = bytes_pass / (ms * 1e-3) / 1e9, "GB/s"
        roof = {"bound": "hbm", "achieved": round(value, 1), "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": round(value / PEAK_HBM_GBS, 4)}
    roof.update({"kernel": "decoder-layer chain, all launches of a pass",
                 "avg_launch_us": round(ms * 1e3 / launches, 3), "launches_per_pass": launches,
                 "ops_per_launch": round(len(entries) / launches, 3),
                 "algorithmic_per_launch": (flops_pass if mfma_bound else bytes_pass) // launches,
                 "traffic": None})
    log(f"[bench] chain: {launches} launches per pass, {value:.1f} {unit} over the pass")
    cpu = None if args.no_cpu_baseline else cpu_baseline_chain(args, wl, W, dev, mfma_bound)
    out = {
        "metric": METRIC, "value": round(value, 2), "unit": unit, "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": f"{wl.qtype} weights x {'f16' if wl.x_dtype == torch.float16 else 'bf16'} "
                 "activations, f32 accumulate, f32 residual stream",
        "data": "synthetic (seeded N(0,0.02) weights, N(0,1) attention outputs and stream)",
        "config": {"workload": wl.name + "_chain", "m": wl.m, "layers": wl.layers,
                   "steps": wl.steps, "ops_per_pass": len(entries),
                   "weight_bytes_per_pass": wbytes_pass, "algorithmic_bytes_per_pass": bytes_pass,
                   "flops_per_pass": flops_pass,
                   "graph_replay": os.environ.get("EB_STACK_GRAPH", "1") != "0",
                   "fused_steps": "rmsnorm prologue, residual add, silu-gated gate/up"},
        "roofline": roof,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


def cpu_baseline_chain(args, wl, W, dev, mfma_bound):
    """The oracle's fused projections along the same chain (its own residual
    stream, binary64, the first rows), layer after layer until about
    --cpu-seconds of oracle time."""
    import numpy as np
    import torch

    from oracle import oracle as O

    orc = O.get()
    cores = min(O.available_cores(), MAX_HOST_THREADS)
    rows = min(args.cpu_rows or (wl.m if wl.m <= 8 else 8), wl.m)
    qt = O.Q8_0 if wl.qtype == "q8_0" else O.Q4_0
    xt = O.X_F16 if wl.x_dtype == torch.float16 else O.X_BF16
    (_, d, n_qkv), _, (_, _, n_gu), (_, f, _) = wl.projections
    h = W.normal((wl.m, d), W.seed_of(wl.wid, 4095, 15, 3), dev)[:rows].cpu().numpy().astype(np.float64)
    secs, nbytes, flops, ops, layers = 0.0, 0, 0, 0, 0

    def bits(t):
        return t.cpu().contiguous().view(torch.int16).numpy().view(np.uint16)

    def timed(fn):
        nonlocal secs
        t = time.perf_counter()
        r = fn()
        secs += time.perf_counter() - t
        return r

    for layer in range(wl.layers):
        if secs >= args.cpu_seconds:
            break
        layers += 1
        blocks = [orc.quantize(qt, W.weights(wl, layer, p, dev).cpu().numpy(), nthreads=cores)
                  for p in range(4)]
        g1 = (1.0 + 0.1 * W.normal((d,), W.seed_of(wl.wid, layer, 0, 2), dev)).cpu().numpy()
        g2 = (1.0 + 0.1 * W.normal((d,), W.seed_of(wl.wid, layer, 2, 2), dev)).cpu().numpy()
        attn = bits(W.activations(wl, layer, 1, dev)[:rows])
        h32 = h.astype(np.float32)
        timed(lambda: orc.fused_qlinear(qt, blocks[0], n_qkv, d, h32, xt, prologue="rmsnorm",
                                        gamma=g1, eps=1e-5, nthreads=cores))
        h = timed(lambda: orc.fused_qlinear(qt, blocks[1], d, d, attn, xt, epilogue="add",
                                            residual=h, nthreads=cores))[0]
        h32 = h.astype(np.float32)
        act = timed(lambda: orc.fused_qlinear(qt, blocks[2], n_gu, d, h32, xt, prologue="rmsnorm",
                                              gamma=g2, eps=1e-5, epilogue="glu", nthreads=cores))[0]
        actw = orc.round_x16(act, xt)
        h = timed(lambda: orc.fused_qlinear(qt, blocks[3], d, f, actw, xt, epilogue="add",
                                            residual=h, nthreads=cores))[0]
        ops += 4
        for (_, k, n) in wl.projections:
            nbytes += op_bytes(wl.qtype, rows, n, k)
            flops += 2 * rows * n * k
    sample = (f"{ops} fused projection calls: the chain through the first {layers} of "
              f"{wl.layers} layers, {rows} of {wl.m} activation rows; {secs:.1f}s of oracle time")
    log(f"[bench] cpu oracle: {sample}")
    if mfma_bound:
        return {"value": round(flops / secs / 1e12, 6), "unit": "TFLOP/s", "cores": cores,
                "kind": "oracle", "sample": sample}
    return {"value": round(nbytes / secs / 1e9, 4), "unit": "GB/s", "cores": cores,
            "kind": "oracle", "sample": sample}


def cpu_baseline(args, wl, W, dev, mfma_bound):
    """Time the CPU oracle (binary64 qlinear over its own quantization of the
    same seeded weights) on a bounded sample of the workload: its projections
    layer by layer (cycling over the layers already quantized when the
    workload is shorter than the time target) on the first rows of x, until
    about --cpu-seconds of timed oracle work has been done."""
    import numpy as np
    import torch

    from oracle import oracle as O

    orc = O.get()
    cores = min(O.available_cores(), MAX_HOST_THREADS)
    max_layers = min(args.cpu_layers or wl.layers, wl.layers)
    rows = min(args.cpu_rows or (wl.m if wl.m <= 8 else 8), wl.m)
    qt = O.Q8_0 if wl.qtype == "q8_0" else O.Q4_0
    xt = O.X_F16 if wl.x_dtype == torch.float16 else O.X_BF16
    cache, cache_bytes = [], 0
    secs, nbytes, flops, ops, layers_seen = 0.0, 0, 0, 0, 0

    def run(blocks, xb, n, k):
        nonlocal secs, nbytes, flops, ops
        t = time.perf_counter()
        orc.qlinear(qt, blocks, n, k, xb, xt, nthreads=cores)
        secs += time.perf_counter() - t
        nbytes += op_bytes(wl.qtype, rows, n, k)
        flops += 2 * rows * n * k
        ops += 1

    for layer in range(max_layers):
        if secs >= args.cpu_seconds:
            break
        layers_seen += 1
        for p, (_, k, n) in enumerate(wl.projections):
            w = W.weights(wl, layer, p, dev).cpu().numpy()
            x = W.activations(wl, layer, p, dev)[:rows]
            xb = x.cpu().contiguous().view(torch.int16).numpy().view(np.uint16)
            blocks = orc.quantize(qt, w, nthreads=cores)  # untimed: weights load once
            del w
            run(blocks, xb, n, k)
            if cache_bytes + blocks.nbytes <= (2 << 30):
                cache.append((blocks, xb, n, k))
                cache_bytes += blocks.nbytes
    while secs < args.cpu_seconds and cache:
        for blocks, xb, n, k in cache:
            run(blocks, xb, n, k)
            if secs >= args.cpu_seconds:
                break
    sample = (f"{ops} projection calls over the first {layers_seen} of {wl.layers} layers "
              f"({len(wl.projections)} projections each, cycling), {rows} of {wl.m} "
              f"activation rows; {secs:.1f}s of oracle time")
    log(f"[bench] cpu oracle: {sample}")
    model = ""
    try:
        with open("/proc/cpuinfo") as fh:
            model = next((l.split(":", 1)[1].strip() for l in fh if l.startswith("model name")), "")
    except OSError:
        pass
    if mfma_bound:
        return {"value": round(flops / secs / 1e12, 6), "unit": "TFLOP/s", "cores": cores,
                "kind": "oracle", "sample": sample, "cpu_model": model}
    return {"value": round(nbytes / secs / 1e9, 4), "unit": "GB/s", "cores": cores,
            "kind": "oracle", "sample": sample, "cpu_model": model}


if __name__ == "__main__":
    main()
