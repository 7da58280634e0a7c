"""Measure the GEMV / MFMA crossover in m (the dispatch table of eb_qlinear).

For each (format, k, n) and m, times both kernel paths on the GPU: R distinct
weight copies of the op are run as one captured graph (one launch per op), so the time per op includes what a
graph pays per launch.
Prints a markdown table; the smallest m at which the MFMA path is faster is
the crossover.  Usage: python -m paper_2607_02501_amd.crossover [--out FILE]
"""
from __future__ import annotations

import argparse
import os
import sys

SHAPES = [("q4_0", "f16", 4096, 4096), ("q4_0", "f16", 4096, 12288), ("q4_0", "f16", 11008, 4096),
          ("q8_0", "bf16", 2048, 2048), ("q8_0", "bf16", 1024, 8192), ("q8_0", "bf16", 4096, 1024),
          ("q8_0", "bf16", 2048, 32768)]
MS = [1, 2, 3, 4, 5, 6, 8, 12, 16, 24, 32, 48, 64]


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--out", default=None)
    ap.add_argument("--reps", type=int, default=5)
    args = ap.parse_args()
    import torch

    from paper_2607_02501_amd import eb
    from paper_2607_02501_amd import workloads as W

    dev = torch.device("cuda:0")
    cap = torch.cuda.Stream()
    dt = {"f16": torch.float16, "bf16": torch.bfloat16}
    lines = ["| format | x | k | n | m | GEMV us | MFMA us | faster |", "|---|---|---|---|---|---|---|---|"]
    cross = []
    for qt, xs, k, n in SHAPES:
        wbytes = n * k * (18 if qt == "q4_0" else 34) // 32
        copies = max(4, min(24, (600 << 20) // wbytes))
        qws = []
        for c in range(copies):
            w = W.normal((n, k), 7000 + c, dev, W.WEIGHT_STD)
            qws.append(eb.quantize(w, qt))
            del w
        first_mfma = None
        for m in MS:
            x = W.normal((m, k), 17, dev).to(dt[xs])
            y = torch.empty((m, n), device=dev)
            ops = eb.make_ops([(q, x, y) for q in qws])
            res = {}
            for path in ("gemv", "mfma"):
                if path == "gemv" and not _gemv_ok(m, k):
                    continue
                # warm up on the capture stream, so a split-K plan finds its
                # workspace there, then time graph replays of one launch per op
                with torch.cuda.stream(cap):
                    for _ in range(2):
                        for q in qws:
                            eb.qlinear(q, x, path=path, out=y)
                torch.cuda.synchronize()
                g = torch.cuda.CUDAGraph()
                with torch.cuda.graph(g, stream=cap):
                    for q in qws:
                        eb.qlinear(q, x, path=path, out=y)
                g.replay()
                torch.cuda.synchronize()
                s0, s1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                s0.record()
                for _ in range(args.reps):
                    g.replay()
                s1.record()
                torch.cuda.synchronize()
                res[path] = s0.elapsed_time(s1) * 1e3 / (args.reps * len(qws))
                del g
            gv, mf = res.get("gemv"), res.get("mfma")
            faster = "gemv" if gv is not None and gv <= mf else "mfma"
            if faster == "mfma" and first_mfma is None:
                first_mfma = m
            lines.append(f"| {qt} | {xs} | {k} | {n} | {m} | {gv:.2f} | {mf:.2f} | {faster} |" if gv is not None
                         else f"| {qt} | {xs} | {k} | {n} | {m} | - | {mf:.2f} | mfma |")
            print(lines[-1], flush=True)
        cross.append((qt, xs, k, n, first_mfma))
        del qws
        torch.cuda.empty_cache()
    lines.append("")
    lines.append("| format | x | k | n | smallest m where MFMA is faster |")
    lines.append("|---|---|---|---|---|")
    for qt, xs, k, n, m in cross:
        lines.append(f"| {qt} | {xs} | {k} | {n} | {m} |")
    text = "\n".join(lines) + "\n"
    print(text)
    if args.out:
        with open(args.out, "w") as f:
            f.write(text)


def _gemv_ok(m, k):
    mt = 1 if m <= 1 else 2 if m <= 2 else 4 if m <= 4 else 8
    return m <= 8 and mt * k <= 65536


if __name__ == "__main__":
    sys.exit(main())
