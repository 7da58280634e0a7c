#!/usr/bin/env python3
"""Benchmark of the quantized linear-layer stack on one MI355X.

    python bench.py [--steps K] [--warmup W]                  # every workload, one JSON line
    python bench.py --workload NAME [--chain] [--steps K] ... # one workload (profiling runs)

One step = one pass of eb_qlinear_stack over every projection of every layer
of a workload (graph-replayed), with weights, activations and outputs already
resident in HBM.  Workloads (seeded synthetic inputs of the shapes in
paper_2607_02501_amd/workloads.py):

  q8_0_m1_2048              one Q8_0 2048x2048 decode linear (128 distinct copies per pass)
  q4_0_decode_7b            batch-1 decode through a 32-layer 7B-class Q4_0 stack
  q6_s_decode_7b            the same decode stack in the 6-bit Q6_S format
  q8_0_vlm_prefill_816      VLM-backbone prefill, m = 816, 18 layers of d = 2048
  q6_s_vlm_prefill_816      the same prefill in the 6-bit Q6_S format
  q8_0_action_expert_50x10  action-expert denoising, m = 50, 18 layers x 10 steps
  q4_0_video_wam_4096       video world-action backbone, m = 4096, 28 layers of d = 3072

A "_chain" variant runs the layers as a dependent decoder-layer chain through
one fp32 residual stream h: QKV on RMSNorm(h), O adding into h (attention is
outside the path: its output is a seeded input per layer), gate/up on
RMSNorm(h) with the SiLU-gated product, down adding into h; every step fused
into its projection's launch (section 3.2, operator fusion).  That is a real
backbone pass: each projection waits for the one before.  The independent
variant gives every projection its own activations, so the stack may fuse
them into few launches (a bandwidth / matrix-core rate, not a pass time).

With no --workload, bench.py measures every workload (independent, and the
chain where the workload has a gate/up projection), the dependent batch-1
decode chain last, and prints ONE JSON line whose headline (value,
ms_per_step, roofline, cpu_baseline) is that decode chain -- the ms per
backbone pass of autoregressive action-token decode -- with every other
measurement under "configs".

Per workload:
  value          whole-pass algorithmic throughput (GB/s for the bandwidth-bound
                 workloads, TFLOP/s for the matrix-core-bound ones)
  ms_per_step    milliseconds per pass (HIP events around K passes)
  roofline       the dominant kernel's algorithmic rate per launch against the
                 MI355X peak, from HIP events on the launch stream around
                 graph replays of that kernel's launches alone (see kernel_groups)
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
PEAK_MFMA_INT8_TOPS = 5000.0     # MI355X dense int8 matrix
RIDGE_FLOP_PER_BYTE = PEAK_MFMA_16BIT_TFLOPS * 1e12 / (PEAK_HBM_GBS * 1e9)  # 312.5
MAX_HOST_THREADS = 16

# every workload, in run order; the headline (decode chain) last
ALL_CONFIGS = [("q8_0_m1_2048", False), ("q4_0_video_wam_4096", False),
               ("q8_0_vlm_prefill_816", False), ("q8_0_vlm_prefill_816", True),
               ("q8_0_action_expert_50x10", False), ("q8_0_action_expert_50x10", True),
               ("q4_0_decode_7b", False), ("q4_0_decode_7b", True),
               ("q6_s_decode_7b", False), ("q6_s_decode_7b", True), ("q6_s_vlm_prefill_816", False)]
HEADLINE = ("q4_0_decode_7b", True)


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=3, help="untimed passes before the timed ones")
    ap.add_argument("--settle-seconds", type=float, default=0.5,
                    help="before the first workload, keep the GPU busy with device copies for "
                         "this long (its clock takes some tens of milliseconds of load to settle); "
                         "no pass of any workload is run for it")
    ap.add_argument("--workload", default=None, help="measure this workload only")
    ap.add_argument("--chain", action="store_true",
                    help="with --workload: the dependent decoder-layer chain")
    ap.add_argument("--multirate", action="store_true",
                    help="measure only the multi-rate control tick (VLM backbone + action expert)")
    ap.add_argument("--int8", action="store_true",
                    help="with --workload: the int8-activation prefill path, op by op")
    ap.add_argument("--no-int8", action="store_true",
                    help="leave the int8 prefill measurements out of the full run")
    ap.add_argument("--no-multirate", action="store_true",
                    help="leave the multi-rate control tick out of the full run")
    ap.add_argument("--cpu-rows", type=int, default=None, help="activation rows in the oracle sample")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="oracle time the headline CPU baseline sample is sized to")
    ap.add_argument("--cpu-seconds-other", type=float, default=2.0,
                    help="oracle time of the other workloads' CPU baseline samples")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-kernel-groups", action="store_true",
                    help="skip the per-kernel roofline timing (profiling runs)")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="BYTES",
                    help="first run a plain device-to-device copy of BYTES (for scaling "
                         "rocprofv3 FETCH_SIZE / WRITE_SIZE counters)")
    return ap.parse_args()


def weight_bytes(qtype, n, k):
    return n * (k // {"q8_0": 32, "q4_0": 32, "q6_s": 256}[qtype]) * {"q8_0": 34, "q4_0": 18, "q6_s": 210}[qtype]


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


def cpu_model():
    try:
        with open("/proc/cpuinfo") as fh:
            return next((l.split(":", 1)[1].strip() for l in fh if l.startswith("model name")), "")
    except OSError:
        return ""


# ---------------------------------------------------------------------------
# Workload entries
# ---------------------------------------------------------------------------

def independent_entries(wl, W, qws, dev, torch):
    """Every projection of every layer (and step) with its own activations."""
    entries, meta = [], []
    for step in range(wl.steps):
        for layer in range(wl.layers):
            for p, (pname, k, n) in enumerate(wl.projections):
                x = W.activations(wl, layer, p, dev, step=step)
                y = torch.empty((wl.m, n), dtype=torch.float32, device=dev)
                entries.append((qws[layer, p], x, y))
                meta.append((pname, p, wl.m, n, k))
    nbytes = sum(op_bytes(wl.qtype, m, n, k) for (_, _, m, n, k) in meta)
    return entries, meta, nbytes


def chain_entries(wl, W, qws, dev, torch):
    """Stack entries of the dependent decoder-layer chain (see the module
    docstring) and its algorithmic bytes per pass: weights, the residual
    stream read by each normalisation and residual addition and written by
    each addition, the attention stand-in, the QKV and gated outputs and
    their re-reads, the normalisation weights."""
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
                meta.append((pname, p, m, n, k))
                nbytes += weight_bytes(wl.qtype, n, k)
            nbytes += (m * d * 4 + d * 4 + m * n_qkv * xs          # QKV: h, g, qkv out
                       + m * d * xs + 2 * m * d * 4                # O: attention, h read and write
                       + m * d * 4 + d * 4 + m * (n_gu // 2) * xs  # gate/up: h, g, gated out
                       + m * f * xs + 2 * m * d * 4)               # down: gated in, h read and write
    return entries, meta, nbytes


def chain_op_bytes(wl, p):
    """Algorithmic bytes of projection p of one chain layer (as chain_entries)."""
    (_, d, n_qkv), _, (_, _, n_gu), (_, f, _) = wl.projections
    m, xs = wl.m, 2
    _, k, n = wl.projections[p]
    extra = [m * d * 4 + d * 4 + m * n_qkv * xs, m * d * xs + 2 * m * d * 4,
             m * d * 4 + d * 4 + m * (n_gu // 2) * xs, m * f * xs + 2 * m * d * 4][p]
    return weight_bytes(wl.qtype, n, k) + extra


# ---------------------------------------------------------------------------
# Timing
# ---------------------------------------------------------------------------

def time_replays(eb, torch, ops, reps, warm=2):
    """ms per eb_qlinear_stack replay, from HIP events on the launch stream."""
    for _ in range(warm):
        eb.qlinear_stack(ops)
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(reps):
        eb.qlinear_stack(ops)
    b.record()
    torch.cuda.synchronize()
    return a.elapsed_time(b) / reps


def roofline_of(flops, nbytes, launches, ms, label, extra=None):
    """The rate of one kernel group against the peak that bounds it (set by
    arithmetic intensity, not by the path that runs it)."""
    avg_ms = ms / launches
    if flops / nbytes > RIDGE_FLOP_PER_BYTE:
        achieved = flops / launches / (avg_ms * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_MFMA_16BIT_TFLOPS,
                "unit": "TFLOP/s", "frac": round(achieved / PEAK_MFMA_16BIT_TFLOPS, 4)}
        per = flops // launches
    else:
        achieved = nbytes / launches / (avg_ms * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBS, 4)}
        per = nbytes // launches
    roof.update({"kernel": label, "avg_launch_us": round(avg_ms * 1e3, 3),
                 "algorithmic_per_launch": per})
    if extra:
        roof.update(extra)
    return roof


def kernel_groups(args, wl, chain, entries, meta, eb, torch):
    """Per-kernel timing.  Independent workloads: ops that run the same kernel
    instance (same path, m and k) form one stack, graph-replayed back to back
    (independent m == 1 ops become one fused launch, small-m ops one fused
    MFMA launch, large-m ops one grouped launch).  A grouped launch whose ops'
    last row tile would be mostly padding hands those rows to a fused small-m
    launch beside it; its group is timed on the rows it keeps (whole 256-row
    tiles), so the figure is that one launch.  Chains: the ops of one
    projection (every layer, every step) form one stack; they depend on each
    other through the residual stream, so they run as lone launches exactly
    as in the pass (an MFMA projection's launch unit is its product plus its
    split-K reduction).  HIP events bracket the replays, so the average launch
    duration excludes host cost and compares with rocprofv3's kernel times.
    Returns the dominant group's roofline and every group's line."""
    groups = {}
    for ent, (pname, p, m, n, k) in zip(entries, meta):
        key = ("proj", p, pname) if chain else (eb.auto_path(wl.qtype, wl.x_dtype, m, n, k), m, k)
        groups.setdefault(key, []).append((ent, p, m, n, k))
    kinds = {}
    for key, items in groups.items():
        if chain:
            gops = eb.make_ops([e for e, *_ in items])
            nbytes = chain_op_bytes(wl, key[1]) * len(items)
            flops = sum(2 * m * n * k for _, _, m, n, k in items)
            rows_note = None
        else:
            m = items[0][2]
            keep = m - m % 256 if (m > 128 and m % 256) else m
            ents = []
            for (qw, x, y), _, mm, n, k in items:
                ents.append((qw, x[:keep], y[:keep]))
            gops = eb.make_ops(ents)
            nbytes = sum(op_bytes(wl.qtype, keep, n, k) for _, _, _, n, k in items)
            flops = sum(2 * keep * n * k for _, _, _, n, k in items)
            rows_note = keep if keep != m else None
        launches = eb.stack_launches(gops)
        reps = max(3, min(50, 2000 // len(items)))
        ms = time_replays(eb, torch, gops, reps)
        kinds[key] = {"ms": ms, "launches": launches, "ops": len(items), "bytes": nbytes,
                      "flops": flops, "rows": rows_note}
        del gops
        eb.stack_cache_clear()
    lines = {}
    for key, d in kinds.items():
        name = f"{key[2]} projection" if chain else f"{key[0]} m={key[1]} k={key[2]}"
        lines[name] = {"ops": d["ops"], "launches_per_replay": d["launches"],
                       "ms_per_replay": round(d["ms"], 4),
                       "GB/s": round(d["bytes"] / d["ms"] / 1e6, 1),
                       "TFLOP/s": round(d["flops"] / d["ms"] / 1e9, 2)}
        if d["rows"]:
            lines[name]["rows_kept"] = d["rows"]
        log(f"[bench] kernel group {name}: {d['ops']} ops in {d['launches']} launches per replay, "
            f"{d['ms']:.4f} ms, {lines[name]['GB/s']} GB/s, {lines[name]['TFLOP/s']} TFLOP/s")
    dom = max(kinds, key=lambda q: kinds[q]["ms"])
    dk = kinds[dom]
    xs = "f16" if wl.x_dtype == torch.float16 else "bf16"
    if chain:
        label = f"chain_{wl.qtype}_{xs}_m{wl.m}_{dom[2]}"
        desc = (f"{dom[2]} projection of the chain, lone launches "
                f"({dk['launches'] // dk['ops']} per projection)")
    else:
        label = f"{dom[0]}_{wl.qtype}_{xs}_m{dom[1]}_k{dom[2]}"
        desc = (f"{dom[0]} path, m = {dom[1]}, k = {dom[2]}: {dk['ops']} ops in {dk['launches']} "
                f"launch(es) per replay")
        if dk["rows"]:
            desc += f" (rows 0..{dk['rows'] - 1}; the last {dom[1] - dk['rows']} rows run beside it)"
    roof = roofline_of(dk["flops"], dk["bytes"], dk["launches"], dk["ms"], label,
                       {"description": desc, "launches_per_replay": dk["launches"],
                        "ops_per_replay": dk["ops"]})
    roof["traffic"] = load_traffic(wl.name + ("_chain" if chain else ""), label)
    return roof, lines


# ---------------------------------------------------------------------------
# CPU baseline (the oracle on a bounded sample)
# ---------------------------------------------------------------------------

def cpu_baseline(args, wl, W, dev, mfma_bound, seconds):
    """Time the CPU oracle (binary64 qlinear over its own quantization of the
    same seeded weights) on a bounded sample of the workload: its projections
    layer by layer (cycling over the layers already quantized when the
    workload is shorter than the time target) on the first rows of x, until
    about `seconds` of timed oracle work has been done."""
    import numpy as np
    import torch

    from oracle import oracle as O

    orc = O.get()
    cores = min(O.available_cores(), MAX_HOST_THREADS)
    rows = min(args.cpu_rows or (wl.m if wl.m <= 8 else 8), wl.m)
    qt = {"q8_0": O.Q8_0, "q4_0": O.Q4_0, "q6_s": O.Q6_S}[wl.qtype]
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

    for layer in range(wl.layers):
        if secs >= seconds:
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
    while secs < seconds and cache:
        for blocks, xb, n, k in cache:
            run(blocks, xb, n, k)
            if secs >= seconds:
                break
    sample = (f"{ops} projection calls over the first {layers_seen} of {wl.layers} layers "
              f"({len(wl.projections)} projections each, cycling), {rows} of {wl.m} "
              f"activation rows; {secs:.1f}s of oracle time")
    log(f"[bench] cpu oracle {wl.name}: {sample}")
    if mfma_bound:
        return {"value": round(flops / secs / 1e12, 6), "unit": "TFLOP/s", "cores": cores,
                "kind": "oracle", "sample": sample, "cpu_model": cpu_model()}
    return {"value": round(nbytes / secs / 1e9, 4), "unit": "GB/s", "cores": cores,
            "kind": "oracle", "sample": sample, "cpu_model": cpu_model()}


def cpu_baseline_chain(args, wl, W, dev, mfma_bound, seconds):
    """The oracle's fused projections along the same chain (its own residual
    stream, binary64, the first rows), layer after layer until about
    `seconds` of oracle time."""
    import numpy as np
    import torch

    from oracle import oracle as O

    orc = O.get()
    cores = min(O.available_cores(), MAX_HOST_THREADS)
    rows = min(args.cpu_rows or (wl.m if wl.m <= 8 else 8), wl.m)
    qt = {"q8_0": O.Q8_0, "q4_0": O.Q4_0, "q6_s": O.Q6_S}[wl.qtype]
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

    cache, cache_bytes = [], 0

    def layer_inputs(layer):
        blocks = [orc.quantize(qt, W.weights(wl, layer, p, dev).cpu().numpy(), nthreads=cores)
                  for p in range(4)]
        g1 = (1.0 + 0.1 * W.normal((d,), W.seed_of(wl.wid, layer, 0, 2), dev)).cpu().numpy()
        g2 = (1.0 + 0.1 * W.normal((d,), W.seed_of(wl.wid, layer, 2, 2), dev)).cpu().numpy()
        attn = bits(W.activations(wl, layer, 1, dev)[:rows])
        return blocks, g1, g2, attn

    def run_layer(inputs):
        nonlocal h, ops, nbytes, flops
        blocks, g1, g2, attn = inputs
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

    # the chain through the layers (weights quantized untimed, as loaded once),
    # then again through the layers kept in memory (up to 2 GB of blocks) until
    # the time target is reached
    for layer in range(wl.layers):
        if secs >= seconds:
            break
        layers += 1
        inputs = layer_inputs(layer)
        run_layer(inputs)
        nb = sum(b.nbytes for b in inputs[0])
        if cache_bytes + nb <= (2 << 30):
            cache.append(inputs)
            cache_bytes += nb
    while secs < seconds and cache:
        for inputs in cache:
            run_layer(inputs)
            if secs >= seconds:
                break
    sample = (f"{ops} fused projection calls: the chain through the first {layers} of "
              f"{wl.layers} layers (then again through the first {len(cache)}, cycling), "
              f"{rows} of {wl.m} activation rows; {secs:.1f}s of oracle time")
    log(f"[bench] cpu oracle {wl.name} chain: {sample}")
    if mfma_bound:
        return {"value": round(flops / secs / 1e12, 6), "unit": "TFLOP/s", "cores": cores,
                "kind": "oracle", "sample": sample, "cpu_model": cpu_model()}
    return {"value": round(nbytes / secs / 1e9, 4), "unit": "GB/s", "cores": cores,
            "kind": "oracle", "sample": sample, "cpu_model": cpu_model()}


def cpu_single_thread(W, dev):
    """The oracle on one thread: one 2048 x 2048 Q8_0 projection at m = 1
    (the first copy of the single-linear workload), repeated for about 2 s."""
    import numpy as np
    import torch

    from oracle import oracle as O

    orc = O.get()
    wl = W.WORKLOADS["q8_0_m1_2048"]
    _, k, n = wl.projections[0]
    blocks = orc.quantize(O.Q8_0, W.weights(wl, 0, 0, dev).cpu().numpy(), nthreads=1)
    xb = W.activations(wl, 0, 0, dev).cpu().contiguous().view(torch.int16).numpy().view(np.uint16)
    secs, calls = 0.0, 0
    while secs < 2.0:
        t = time.perf_counter()
        orc.qlinear(O.Q8_0, blocks, n, k, xb, O.X_F16, nthreads=1)
        secs += time.perf_counter() - t
        calls += 1
    return {"value": round(calls * op_bytes("q8_0", 1, n, k) / secs / 1e9, 4), "unit": "GB/s",
            "gflops": round(calls * 2 * n * k / secs / 1e9, 4), "cores": 1,
            "sample": f"{calls} calls of one 2048x2048 Q8_0 projection at m = 1, {secs:.1f}s"}


# ---------------------------------------------------------------------------
# One workload
# ---------------------------------------------------------------------------

def run_workload(args, name, chain, cpu_seconds, eb, W, torch, dev):
    wl = W.WORKLOADS[name]
    names = [p[0] for p in wl.projections]
    if chain and names[2] != "gate_up":
        raise SystemExit(f"--chain needs a gate/up projection; {wl.name} has {names}")
    t_setup = time.time()
    qws = {}
    for layer in range(wl.layers):
        for p, (_, k, n) in enumerate(wl.projections):
            w = W.weights(wl, layer, p, dev)
            qws[layer, p] = eb.quantize(w, wl.qtype)
            del w
    if chain:
        entries, meta, bytes_pass = chain_entries(wl, W, qws, dev, torch)
    else:
        entries, meta, bytes_pass = independent_entries(wl, W, qws, dev, torch)
    ops = eb.make_ops(entries)
    torch.cuda.synchronize()
    launches = eb.stack_launches(ops)
    label = wl.name + ("_chain" if chain else "")
    log(f"[bench] {label}: {len(entries)} ops per pass, {launches} launches per pass, "
        f"setup {time.time() - t_setup:.1f}s")
    wbytes_pass = sum(weight_bytes(wl.qtype, n, k) for (_, _, m, n, k) in meta)
    flops_pass = sum(2 * m * n * k for (_, _, m, n, k) in meta)
    mfma_bound = flops_pass / bytes_pass > RIDGE_FLOP_PER_BYTE

    # ---- timed region: W warmup passes, then K graph-replayed passes ---------
    for _ in range(args.warmup):
        eb.qlinear_stack(ops)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(args.steps):
        eb.qlinear_stack(ops)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    log(f"[bench] {label}: {args.warmup} warmup passes, {args.steps} timed passes: {ms:.4f} ms/pass")
    eb.stack_cache_clear()

    if mfma_bound:
        value, unit = flops_pass / (ms * 1e-3) / 1e12, "TFLOP/s"
    else:
        value, unit = bytes_pass / (ms * 1e-3) / 1e9, "GB/s"
    roof, lines = (None, None) if args.no_kernel_groups else kernel_groups(
        args, wl, chain, entries, meta, eb, torch)
    cpu = None
    if not args.no_cpu_baseline and cpu_seconds > 0:
        cpu = (cpu_baseline_chain if chain else cpu_baseline)(args, wl, W, dev, mfma_bound, cpu_seconds)
    xs = "f16" if wl.x_dtype == torch.float16 else "bf16"
    out = {
        "ms_per_step": round(ms, 5), "value": round(value, 2), "unit": unit,
        "steps": args.steps, "warmup": args.warmup, "launches_per_pass": launches,
        "dtype": f"{wl.qtype} weights x {xs} activations, f32 accumulate"
                 + (", f32 residual stream" if chain else ""),
        "config": {"workload": label, "m": wl.m, "layers": wl.layers, "steps": wl.steps,
                   "ops_per_pass": len(entries), "weight_bytes_per_pass": wbytes_pass,
                   "algorithmic_bytes_per_pass": bytes_pass, "flops_per_pass": flops_pass,
                   "graph_replay": os.environ.get("EB_STACK_GRAPH", "1") != "0",
                   "dependent_chain": chain,
                   **({"fused_steps": "rmsnorm prologue, residual add, silu-gated gate/up"}
                      if chain else {})},
        "roofline": roof, "kernel_groups": lines, "cpu_baseline": cpu,
    }
    del entries, ops, qws
    torch.cuda.empty_cache()
    return out


def run_int8(args, name, eb, W, torch, dev):
    """The int8-activation prefill path (EB_PATH_MFMA_I8) over every projection
    of an independent large-m workload, one eb_qlinear_fused_ws call per op in
    layer order (each op: the activation-quantization launch, then the int8
    product launch), timed with HIP events on the launch stream.  TOP/s
    against the dense int8 peak; ms per pass."""
    import ctypes

    wl = W.WORKLOADS[name]
    qws = {(layer, p): eb.quantize(W.weights(wl, layer, p, dev), wl.qtype)
           for layer in range(wl.layers) for p in range(len(wl.projections))}
    entries, meta, _ = independent_entries(wl, W, qws, dev, torch)
    ops = eb.make_ops(entries)
    need = max(int(eb.lib.eb_qlinear_workspace_bytes(ctypes.byref(ops[i]), eb.EB_PATH_MFMA_I8))
               for i in range(len(ops)))
    ws = torch.empty(need, dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream().cuda_stream
    fn, wp = eb.lib.eb_qlinear_fused_ws, ws.data_ptr()
    refs = [ctypes.byref(ops[i]) for i in range(len(ops))]

    def one_pass():
        for r in refs:
            st = fn(r, eb.EB_PATH_MFMA_I8, wp, need, stream)
            if st != 0:
                raise SystemExit(f"eb_qlinear_fused_ws (int8 path) failed: {st}")

    for _ in range(max(1, args.warmup // 5)):
        one_pass()
    torch.cuda.synchronize()
    steps = max(1, args.steps // 5)
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(steps):
        one_pass()
    b.record()
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / steps
    flops = sum(2 * m * n * k for (_, _, m, n, k) in meta)
    tops = flops / (ms * 1e-3) / 1e12
    log(f"[bench] {name} int8 path: {ms:.4f} ms/pass, {tops:.1f} TOP/s")
    del entries, ops, qws, ws
    torch.cuda.empty_cache()
    return {"ms_per_step": round(ms, 5), "value": round(tops, 2), "unit": "TOP/s", "steps": steps,
            "launches_per_pass": 2 * len(meta),
            "dtype": f"{wl.qtype} weight codes x int8 activation blocks, i32 block products, f32 accumulate",
            "config": {"workload": name + "_int8", "m": wl.m, "layers": wl.layers,
                       "ops_per_pass": len(meta), "flops_per_pass": flops,
                       "graph_replay": False, "dependent_chain": False},
            "roofline": {"bound": "mfma", "achieved": round(tops, 2), "peak": PEAK_MFMA_INT8_TOPS,
                         "unit": "TOP/s", "frac": round(tops / PEAK_MFMA_INT8_TOPS, 4),
                         "note": "whole pass incl. the activation-quantization launches"}}


def run_multirate(args, eb, W, torch, dev):
    """Control ticks of a VLM-backboned policy with a flow-matching action
    expert (include/eb_multirate.h): the backbone module is the dependent
    816-row prefill chain (18 layers, d = 2048), refreshed every R ticks; the
    expert module is one denoising step of the 50-row action-expert chain
    (18 layers, d = 1024), run 10 times every tick.  Reports ms per tick
    averaged over whole refresh cycles for R = 1, 2, 4, and the refresh and
    reuse ticks of R = 4 separately."""
    import dataclasses

    wb = W.WORKLOADS["q8_0_vlm_prefill_816"]
    we = dataclasses.replace(W.WORKLOADS["q8_0_action_expert_50x10"], steps=1)
    mods_ops = []
    for wl in (wb, we):
        qws = {(layer, p): eb.quantize(W.weights(wl, layer, p, dev), wl.qtype)
               for layer in range(wl.layers) for p in range(len(wl.projections))}
        entries, _, _ = chain_entries(wl, W, qws, dev, torch)
        mods_ops.append((eb.make_ops(entries), entries, qws))
    b_ops, e_ops = mods_ops[0][0], mods_ops[1][0]
    out = {"unit": "ms/tick", "expert_steps_per_tick": 10,
           "modules": {"backbone": "q8_0_vlm_prefill_816 chain (period R)",
                       "expert": "q8_0_action_expert_50x10 chain, one step (10 per tick)"}}
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    cycles = max(1, args.steps // 10)
    for R in (1, 2, 4):
        mods = eb.make_modules([(b_ops, R, 0, 1), (e_ops, 1, 0, 10)])
        for t in range(R):          # warm-up cycle: plans built, graphs captured
            eb.multirate_tick(mods, t, dev)
        torch.cuda.synchronize()
        a.record()
        for c in range(cycles):
            for t in range(R):
                eb.multirate_tick(mods, t, dev)
        b.record()
        torch.cuda.synchronize()
        out[f"R{R}"] = round(a.elapsed_time(b) / (cycles * R), 4)
        if R == 4:
            per = []
            for t in range(2):
                torch.cuda.synchronize()
                a.record()
                for _ in range(cycles):
                    eb.multirate_tick(mods, t, dev)
                b.record()
                torch.cuda.synchronize()
                per.append(a.elapsed_time(b) / cycles)
            out["refresh_tick_ms"], out["reuse_tick_ms"] = round(per[0], 4), round(per[1], 4)
        log(f"[bench] multi-rate tick, backbone every {R} ticks: {out[f'R{R}']:.4f} ms/tick")
        del mods
    # without reuse the backbone would run before every denoising step
    out["no_reuse_estimate_ms"] = round(10 * (out["refresh_tick_ms"] - out["reuse_tick_ms"])
                                        + out["reuse_tick_ms"], 4)
    eb.stack_cache_clear()
    del mods_ops
    torch.cuda.empty_cache()
    return out


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}, WORLD_SIZE {world}): "
              "there is no multi-GPU path; run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2607_02501_amd import eb
    from paper_2607_02501_amd import workloads as W

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
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
    if args.settle_seconds > 0:
        a = torch.empty(64 << 20, dtype=torch.uint8, device=dev)
        b = torch.empty_like(a)
        t0 = time.time()
        while time.time() - t0 < args.settle_seconds:
            for _ in range(16):
                b.copy_(a)
            torch.cuda.synchronize()
        del a, b

    common = {"metric": METRIC, "n_gpus": 1, "higher_is_better": True, "scaling": "weak",
              "vs_baseline": None,
              "data": "synthetic (seeded N(0,0.02) weights, N(0,1) activations and stream)"}
    if args.workload and args.int8:
        print(json.dumps({**common, **run_int8(args, args.workload, eb, W, torch, dev)}), flush=True)
        return
    if args.workload:
        r = run_workload(args, args.workload, args.chain, args.cpu_seconds, eb, W, torch, dev)
        print(json.dumps({**common, **r}), flush=True)
        return
    if args.multirate:
        print(json.dumps({**common, "multirate": run_multirate(args, eb, W, torch, dev)}), flush=True)
        return

    results = {}
    for name, chain in ALL_CONFIGS:
        head = (name, chain) == HEADLINE
        secs = args.cpu_seconds if head else args.cpu_seconds_other
        results[name + ("_chain" if chain else "")] = run_workload(args, name, chain, secs, eb, W,
                                                                    torch, dev)
    if not args.no_int8:
        for name in ("q4_0_video_wam_4096", "q8_0_vlm_prefill_816"):
            results[name + "_int8"] = run_int8(args, name, eb, W, torch, dev)
    if not args.no_multirate:
        results["multirate_vla_tick"] = run_multirate(args, eb, W, torch, dev)
    head = results.pop(HEADLINE[0] + "_chain")
    if head["cpu_baseline"] is not None:
        head["cpu_baseline"]["single_thread"] = cpu_single_thread(W, dev)
    out = {**common, **head, "configs": results}
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
