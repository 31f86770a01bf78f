#!/usr/bin/env python3
"""Training-step throughput of the dynamic-control-flow path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload lm2048]

A step is one whole forward + backward pass of the workload through the C
ABI (every kernel of the path), on inputs already resident in HBM.  The
default workload is the 2-layer LSTM with input 2048, hidden 2048, batch
256, length 256, bf16 with float32 accumulation, per-step projection to 2048
and MSE loss (synthetic seeded inputs).  Prints one JSON line.

Timing: W untimed warmup steps, then K steps between two events on the
stream the library launches on, bracketed by device synchronisation.  A
second pass of K steps with library tracing on gives each kernel's average
launch duration (HIP events around every launch); the kernel with the
largest total time is reported in "roofline".  The float64 oracle is timed
on the host on a bounded sample of the same workload ("cpu_baseline").
"""
from __future__ import annotations

import argparse
import glob
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 MFMA
PEAK_F32_TFLOPS = 157.3       # MI355X fp32 matrix
PEAK_HBM_GBS = 8000.0         # MI355X HBM3E

WORKLOADS = {
    "lm2048": dict(desc="2-layer LSTM, input 2048, hidden 2048, batch 256, length 256, bf16 (fp32 accumulate), "
                        "projection 2048 + MSE", unit="sequences/s"),
    "ptb": dict(desc="2-layer LSTM LM, vocab 10000 (Zipf 1.1), embed/hidden 650, batch 20, 35 steps, bf16, "
                     "softmax cross-entropy", unit="sequences/s"),
    "varlen": dict(desc="1-layer LSTM, input 512, hidden 1024, batch 128, lengths U[1,200], bf16, "
                        "mean of final h", unit="sequences/s"),
    "treelstm": dict(desc="binary TreeLSTM, embed 300, hidden 150, 25 trees of 5-50 leaves, fp32, "
                          "5-class softmax at roots", unit="trees/s"),
    "tiny": dict(desc="1-layer LSTM, input 32, hidden 64, batch 4, length 16, fp32, sum of squares of final h",
                 unit="sequences/s"),
    "treernn": dict(desc="binary TreeRNN, word vectors and hidden 300, 25 trees of 5-50 leaves, fp32, "
                         "5-class softmax at roots", unit="trees/s"),
    "childsum": dict(desc="Child-Sum TreeLSTM, embed 300, hidden 150, 25 random trees of 5-50 nodes, a word at "
                          "every node, fp32, 5-class softmax at roots", unit="trees/s"),
}


# The sources that define and launch the persistent recurrence kernels, whose
# HBM counters profiles/ records: a change to any of them voids the record.
TRAFFIC_SOURCES = ("device.hpp", "lstm.hip", "lstm_persist.hpp")


def source_digest() -> str:
    h = hashlib.sha256()
    for name in TRAFFIC_SOURCES:
        with open(os.path.join(ROOT, "paper_1812_01329_amd", "csrc", name), "rb") as f:
            h.update(name.encode())
            h.update(f.read())
    return h.hexdigest()[:16]


def load_traffic(label: str, workload: str):
    """HBM traffic per launch of `label` from a committed counter summary,
    or None when absent or taken on different kernel sources."""
    digest = source_digest()
    for p in sorted(glob.glob(os.path.join(ROOT, "profiles", "*.md"))):
        for line in open(p):
            m = re.match(r"traffic-record: (.*)$", line.strip())
            if not m:
                continue
            rec = dict(kv.split("=", 1) for kv in m.group(1).split())
            if rec.get("label") == label and rec.get("workload") == workload and rec.get("source") == digest:
                return float(rec["bytes_per_launch"])
    return None


def cpu_baseline(w, n_rows: int):
    """Time the oracle on the first n_rows sequences of the workload."""
    import numpy as np
    from oracle import steps as oracle_steps
    from paper_1812_01329_amd import workloads as wl
    try:
        from threadpoolctl import threadpool_info
        info = threadpool_info()
        cores = max([i.get("num_threads", 1) for i in info if i.get("user_api") == "blas"] or [1])
        blas = ",".join(sorted({i.get("internal_api", "?") for i in info if i.get("user_api") == "blas"}))
    except Exception:  # pragma: no cover - threadpoolctl is optional
        cores, blas = len(os.sched_getaffinity(0)), "?"
    if hasattr(w, "trees"):
        t0 = time.perf_counter()
        if isinstance(w, wl.TreeRNNWorkload):
            oracle_steps.treernn_step(w)
        elif isinstance(w, wl.ChildSumWorkload):
            oracle_steps.childsum_step(w)
        else:
            oracle_steps.tree_step(w)
        dt = time.perf_counter() - t0
        n = w.trees.num_trees
        sample = f"all {n} trees of the batch, float64 numpy oracle, fwd+bwd"
    else:
        rows = np.arange(min(n_rows, w.B))
        t0 = time.perf_counter()
        oracle_steps.lstm_step(w, batch_rows=rows)
        dt = time.perf_counter() - t0
        n = len(rows)
        sample = (f"{n} of {w.B} sequences of the same batch (full length, all layers, loss head), "
                  f"float64 numpy oracle, fwd+bwd")
    return {"value": n / dt, "unit": WORKLOADS_UNIT, "cores": int(cores), "kind": "oracle", "sample": sample,
            "seconds": round(dt, 3), "blas": blas, "host_cpus": len(os.sched_getaffinity(0))}


WORKLOADS_UNIT = "sequences/s"


def main():
    global WORKLOADS_UNIT
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="lm2048", choices=sorted(WORKLOADS))
    ap.add_argument("--cpu-rows", type=int, default=4, help="sequences in the oracle sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-trace", action="store_true")
    ap.add_argument("--with-update", action="store_true",
                    help="end every step with the SGD update with global-norm clipping (lr 0.1, max norm 5)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only copy a 1 GiB buffer three times (reference for HBM byte counters) and exit")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}, WORLD_SIZE {world}); "
              "the path shards by data parallelism and is benchmarked on a single MI355X.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    from paper_1812_01329_amd import janus as J
    from paper_1812_01329_amd import workloads as wl
    from paper_1812_01329_amd.train_step import make_step

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    if args.copy_calibration:
        # a plain device copy of known size: the HBM byte counters of one such
        # copy read 1 GiB fetched and 1 GiB written when they count bytes
        src = torch.empty(1 << 29, dtype=torch.bfloat16, device="cuda").fill_(1.0)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": src.numel() * src.element_size()}))
        return
    spec = WORKLOADS[args.workload]
    WORKLOADS_UNIT = spec["unit"]
    w = wl.FULL[args.workload]()
    print(f"[bench] workload {args.workload}: {spec['desc']}", file=sys.stderr, flush=True)
    step = make_step(w, update=(0.1, 5.0) if args.with_update else None)
    units = w.trees.num_trees if hasattr(w, "trees") else w.B

    for _ in range(args.warmup):
        step.run()
    torch.cuda.synchronize()
    print(f"[bench] warmup done ({args.warmup} steps)", file=sys.stderr, flush=True)
    stream = torch.cuda.current_stream()
    start = torch.cuda.Event(enable_timing=True)
    stop = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    start.record(stream)
    for _ in range(args.steps):
        step.run()
    stop.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = start.elapsed_time(stop) / args.steps
    value = units / (ms / 1e3)
    print(f"[bench] timed {args.steps} steps: {ms:.3f} ms/step (wall {wall / args.steps * 1e3:.3f})",
          file=sys.stderr, flush=True)

    roofline, kernels = None, None
    if not args.no_trace:
        J.janus_trace_begin()
        for _ in range(args.steps):
            step.run()
        stats = J.janus_trace_end()
        torch.cuda.synchronize()
        total = sum(s["total_ms"] for s in stats) / args.steps
        stats.sort(key=lambda s: -s["total_ms"])
        kernels = {s["label"]: {"launches_per_step": s["launches"] // args.steps,
                                "ms_per_step": round(s["total_ms"] / args.steps, 4),
                                "avg_us": round(1e3 * s["total_ms"] / s["launches"], 3),
                                "tflops": round(s["flops"] / (s["total_ms"] * 1e-3) / 1e12, 2) if s["flops"] else None,
                                "gbs": round(s["bytes"] / (s["total_ms"] * 1e-3) / 1e9, 1)}
                   for s in stats if s in stats[:8] or s["label"].startswith("sgd_")}
        top = stats[0]
        avg_s = top["total_ms"] / top["launches"] * 1e-3
        bf16 = top["label"].endswith("bf16") or w.dtype == wl.BF16
        if top["flops"] > 0:
            per_launch = top["flops"] / top["launches"]
            achieved = per_launch / avg_s / 1e12
            peak = PEAK_BF16_TFLOPS if bf16 else PEAK_F32_TFLOPS
            bound, unit = "mfma", "TFLOP/s"
        else:
            per_launch = top["bytes"] / top["launches"]
            achieved = per_launch / avg_s / 1e9
            peak, bound, unit = PEAK_HBM_GBS, "hbm", "GB/s"
        traffic = load_traffic(top["label"], args.workload)
        roofline = {"bound": bound, "achieved": round(achieved, 2), "peak": peak, "unit": unit,
                    "frac": round(achieved / peak, 4), "traffic": traffic, "kernel": top["label"],
                    "launches_per_step": top["launches"] // args.steps,
                    "avg_launch_us": round(avg_s * 1e6, 3),
                    "work_per_launch": per_launch,
                    # algorithmic bytes of the same kernel (each value read or written once) per second
                    "algorithmic_gbs": round(top["bytes"] / top["launches"] / avg_s / 1e9, 1) if top["bytes"] else None,
                    "traced_ms_per_step": round(total, 3)}
        print(f"[bench] traced pass: {total:.3f} ms of kernel time per step; top kernel {top['label']}",
              file=sys.stderr, flush=True)

    # whole-step algorithmic rate against the peak of the step's dtype
    step_flops = None
    if not hasattr(w, "trees") and w.head == "mse":
        H, I, B, T, L, P = w.H, w.I, w.B, w.T, w.L, w.Wout.shape[0]
        fwd = sum(2 * T * B * 4 * H * ((I if l == 0 else H) + H) for l in range(L)) + 2 * T * B * H * P
        bwd = (2 * T * B * H * P * 2                                       # head dW, dh
               + sum(2 * T * B * 4 * H * H                                  # recurrent dh
                     + 2 * T * B * 4 * H * ((I if l == 0 else H) + H)       # dWx, dWh
                     + (2 * T * B * 4 * H * H if l > 0 else 0)              # dX into the layer below
                     for l in range(L)))
        step_flops = fwd + bwd

    cpu = None
    if not args.no_cpu_baseline:
        print("[bench] timing the oracle on the host", file=sys.stderr, flush=True)
        cpu = cpu_baseline(w, args.cpu_rows)

    out = {
        "metric": "training sequences(trees)/sec fwd+bwd on 1 MI355X; % of bf16 MFMA peak",
        "value": round(value, 2),
        "unit": spec["unit"],
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if getattr(w, "dtype", "f32") == wl.BF16 else "f32",
        "data": "synthetic",
        "config": {"workload": f"{args.workload}: {spec['desc']}", "units_per_step": units,
                   "update": "sgd, global-norm clip 5.0" if args.with_update else None},
        "roofline": roofline,
        "cpu_baseline": cpu,
    }
    if step_flops:
        out["step_tflops"] = round(step_flops / (ms * 1e-3) / 1e12, 2)
        out["step_frac_of_bf16_peak"] = round(step_flops / (ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4)
    if kernels:
        out["kernels"] = kernels
    print(json.dumps(out))


if __name__ == "__main__":
    main()
