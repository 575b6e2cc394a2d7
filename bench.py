#!/usr/bin/env python3
"""Benchmark of the 2D-block FP4 linear-layer hot path on one MI355X.

One step = one forward + backward pass of every linear layer of the workload:
quantize each activation X and weight W (round to nearest) and each output
gradient dY (stochastic rounding) once into both packed layouts, then run the
three GEMMs of every layer, Y = X W^T (bf16 out), dX = dY W (bf16 out) and
dW = dY^T X (fp32 out), reusing the quantized operands transposed.

Prints one JSON line.  ``value`` = algorithmic GEMM flops of the step / wall
time of the whole step (quantizers included) with all inputs resident in HBM.
The ``roofline`` object is for the dominant kernel (the FP4 GEMM), timed per
launch with HIP events on the stream the kernels run on; ``quantizer`` reports
the fused quantizer against the HBM roofline the same way; ``cpu_baseline`` is
the CPU oracle timed on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, HERE)

PEAK_FP4_TFLOPS = 10100.0      # MI355X dense MXFP4 MFMA
PEAK_FP8_TFLOPS = 5000.0       # MI355X dense FP8 MFMA
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E

WORKLOAD_TEXT = {
    "dense_7b": "7B-class dense linears fwd+bwd (QKV 4096->12288, O 4096->4096, gate/up "
                "4096->11008, down 11008->4096), tokens 16384, bf16 inputs, 32x32 2D-block FP4 "
                "(X, W round-to-nearest; dY stochastic), X with 1% Student-t outlier channels",
    "dense_1b": "1B-class dense MLP fwd+bwd (up 2048->5632, down 5632->2048), tokens 8192, "
                "bf16 inputs, 32x32 2D-block FP4 with stochastic rounding on X, W and dY",
}


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=10)
    p.add_argument("--warmup", type=int, default=3)
    p.add_argument("--workload", default="dense_7b", choices=sorted(WORKLOAD_TEXT))
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-sample-tokens", type=int, default=256)
    return p.parse_args()


def quant_bytes(t) -> float:
    """Algorithmic bytes of one quantization: input once, both 4-bit layouts, scales once."""
    n = t.numel()
    return n * t.element_size() + n * 0.5 * 2 + n / 1024.0


def source_hash(*names) -> str:
    h = hashlib.sha256()
    for n in names:
        with open(os.path.join(HERE, "paper_2607_24953_amd", "csrc", n), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def read_traffic(kernel: str, src_hash: str):
    """HBM bytes per launch measured with rocprofv3 counters, if taken on this kernel source."""
    path = os.path.join(HERE, "profiles", "traffic.json")
    try:
        with open(path) as f:
            rec = json.load(f).get(kernel)
    except (OSError, ValueError):
        return None
    if not rec or rec.get("source_hash") != src_hash:
        return None
    return rec


class Step:
    """Runs one fwd+bwd pass of the workload and records per-kernel HIP events."""

    def __init__(self, q2d, torch, w):
        self.q2d, self.torch, self.w = q2d, torch, w
        dev = next(iter(w.tensors.values())).device
        self.q = {k: q2d.QTensor(q2d.FP4_2D, t.shape[0], t.shape[1], dev) for k, t in w.tensors.items()}
        self.out = []
        for lin in w.linears:
            self.out.append((torch.empty((lin.tokens, lin.n_out), dtype=torch.bfloat16, device=dev),
                             torch.empty((lin.tokens, lin.k_in), dtype=torch.bfloat16, device=dev),
                             torch.empty((lin.n_out, lin.k_in), dtype=torch.float32, device=dev)))
        self.events = None

    def run(self, record: bool):
        q2d, torch, w = self.q2d, self.torch, self.w
        ev = [] if record else None

        def mark(kind, work):
            if record:
                e0 = torch.cuda.Event(enable_timing=True)
                e0.record()
                return (kind, work, e0)
            return None

        def done(m):
            if m is not None:
                e1 = torch.cuda.Event(enable_timing=True)
                e1.record()
                ev.append(m + (e1,))

        for i, (k, t) in enumerate(w.tensors.items()):
            m = mark(("quant", k), quant_bytes(t))
            q2d.q2d_quantize(t, w.rounding[k], w.seed, i, out=self.q[k])
            done(m)
        for lin, (Y, dX, dW) in zip(w.linears, self.out):
            qx, qw, qdy = self.q[lin.x], self.q[lin.w], self.q[lin.dy]
            f = 2.0 * lin.tokens * lin.n_out * lin.k_in
            m = mark(("gemm", lin.name + ".fwd"), f); q2d.q2d_gemm(qx, 0, qw, 0, out=Y); done(m)
            m = mark(("gemm", lin.name + ".dX"), f); q2d.q2d_gemm(qdy, 0, qw, 1, out=dX); done(m)
            m = mark(("gemm", lin.name + ".dW"), f); q2d.q2d_gemm(qdy, 1, qx, 1, out=dW); done(m)
        if record:
            self.events = (self.events or []) + ev


def cpu_baseline(w, tokens: int):
    """The oracle (C quantizer with OpenMP, float64 numpy GEMMs) on the first `tokens`
    rows of every activation and gradient of the workload, full weights."""
    import numpy as np
    import oracle
    threads = len(os.sched_getaffinity(0))
    oracle.build()
    flops = 0.0
    t0 = time.perf_counter()
    cache = {}
    for lin in w.linears:
        def q(name, rows=None):
            key = (name, rows)
            if key not in cache:
                t = w.tensors[name]
                t = (t[:rows] if rows else t).cpu()
                cache[key] = oracle.quantize_fp4_2d(t, w.rounding[name], w.seed, 0, threads=threads)
            return cache[key]
        qx, qw, qdy = q(lin.x, tokens), q(lin.w), q(lin.dy, tokens)
        out = oracle.linear(qx, qw, qdy)
        flops += 3 * 2.0 * tokens * lin.n_out * lin.k_in
        del out
    dt = time.perf_counter() - t0
    return {"value": flops / dt / 1e12, "unit": "TFLOP/s", "cores": threads, "kind": "oracle",
            "sample": "all %d linears of the workload on the first %d tokens (full weights): "
                      "C oracle quantization of X, W, dY + float64 numpy GEMMs; %.1f s wall, "
                      "%.3f TFLOP" % (len(w.linears), tokens, dt, flops / 1e12)}


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py: this build measures one GPU only; --gpus %d is not supported" % args.gpus,
              file=sys.stderr)
        sys.exit(2)
    import torch
    import synth
    import paper_2607_24953_amd as q2d

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    w = synth.WORKLOADS[args.workload](device=dev)
    step = Step(q2d, torch, w)
    for _ in range(args.warmup):
        step.run(record=False)
    torch.cuda.synchronize()

    # timed region 1: wall clock of K whole steps
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step.run(record=False)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_per_step = wall * 1e3 / args.steps

    # timed region 2: the same K steps with HIP events around every launch
    for _ in range(args.steps):
        step.run(record=True)
    torch.cuda.synchronize()
    t_gemm = t_quant = 0.0
    f_gemm = b_quant = 0.0
    n_gemm = 0
    detail = {}
    for (kind, name), work, e0, e1 in step.events:
        ms = e0.elapsed_time(e1)
        d = detail.setdefault(name, [0.0, 0.0, 0])
        d[0] += ms; d[1] += work; d[2] += 1
        if kind == "gemm":
            t_gemm += ms; f_gemm += work; n_gemm += 1
        else:
            t_quant += ms; b_quant += work
    per_kernel = {}
    for name, (ms, work, n) in detail.items():
        rate = work / (ms * 1e-3) / (1e12 if "." in name else 1e9)
        per_kernel[name] = {"ms": round(ms / n, 4), ("TFLOP/s" if "." in name else "GB/s"): round(rate, 1)}
    gemm_tflops = f_gemm / (t_gemm * 1e-3) / 1e12
    quant_gbs = b_quant / (t_quant * 1e-3) / 1e9
    flops_step = float(w.gemm_flops)
    value = flops_step / (ms_per_step * 1e-3) / 1e12

    gemm_hash = source_hash("gemm.hip", "device_common.hpp")
    quant_hash = source_hash("quantize_fp4.hip", "device_common.hpp")
    tr_g = read_traffic("gemm_fp4", gemm_hash)
    tr_q = read_traffic("quantize_fp4", quant_hash)

    rec = {
        "metric": "FP4 fwd+bwd linear TFLOP/s (7B shapes) + quantizer GB/s, % of roofline",
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "fp4_e2m1 (fp32 accumulate)",
        "data": "synthetic (seeded normals, bf16; no datasets or trained weights)",
        "config": {"workload": WORKLOAD_TEXT[args.workload], "name": args.workload,
                   "tokens": w.linears[0].tokens, "linears": len(w.linears),
                   "gemms_per_step": 3 * len(w.linears), "gemm_tflop_per_step": flops_step / 1e12,
                   "quantizations_per_step": len(w.tensors), "block": 32},
        "roofline": {"bound": "mfma", "kernel": "gemm_kernel<FP4>", "achieved": round(gemm_tflops, 2),
                     "peak": PEAK_FP4_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(gemm_tflops / PEAK_FP4_TFLOPS, 4),
                     "traffic": tr_g["bytes_per_launch"] if tr_g else None,
                     "launches_timed": n_gemm, "avg_launch_ms": round(t_gemm / max(n_gemm, 1), 5)},
        "quantizer": {"bound": "hbm", "kernel": "fp4_quantize_kernel", "achieved": round(quant_gbs, 1),
                      "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": round(quant_gbs / PEAK_HBM_GBS, 4),
                      "traffic": tr_q["bytes_per_launch"] if tr_q else None,
                      "ms_per_step": round(t_quant / args.steps, 4)},
        "gemm_ms_per_step": round(t_gemm / args.steps, 4),
        "per_kernel": per_kernel,
    }
    if not args.no_cpu_baseline:
        rec["cpu_baseline"] = cpu_baseline(w, args.cpu_sample_tokens)
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
