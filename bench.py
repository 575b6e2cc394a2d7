#!/usr/bin/env python3
"""Benchmark of the 2D-block FP4 linear-layer hot path on one MI355X.

One step = one forward + backward pass of every linear layer of the workload:
quantize each activation X and weight W and each output gradient dY once into
both packed layouts, then run the three GEMMs of every layer, Y = X W^T (bf16
out), dX = dY W (bf16 out) and dW = dY^T X (fp32 out), reusing the quantized
operands transposed.  The 7B-class dense workload is the headline; the MoE
expert FFN (grouped quantizer and grouped GEMMs), the mixed MXFP8 / FP4 7B
block and the 7B linears with 1D-block activations (the paper's placement) are
measured in the same run under ``other_workloads``.

Prints one JSON line.  ``value`` = algorithmic GEMM flops of the step / wall
time of the whole step (quantizers included) with all inputs resident in HBM.
The ``roofline`` object is for the dominant kernel (the FP4 GEMM), timed per
launch with HIP events on the stream the kernels run on; ``quantizer`` reports
the fused quantizer against the HBM roofline the same way; ``cpu_baseline`` is
the CPU oracle timed on a bounded sample of the same workload.

``--copy-calibration BYTES`` only runs a plain device copy of that size (the
reference that scales the HBM byte counters of a profile).
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
    "tiny": "Tiny linear fwd+bwd: W 256x256 ~N(0,0.02), X 128x256 ~N(0,1), dY 128x256 ~N(0,1e-3), "
            "float32 inputs, 32x32 2D-block FP4 with stochastic rounding (seed 0) on X, W and dY; "
            "fwd, dX and dW GEMMs",
    "dense_1b": "1B-class dense MLP fwd+bwd (up 2048->5632, down 5632->2048), tokens 8192, "
                "bf16 inputs, 32x32 2D-block FP4 with stochastic rounding on X, W and dY",
    "moe_30b": "30B-class MoE expert FFN fwd+bwd: 16384 tokens, top-8 of 128 experts "
               "(Zipf 1.1 routing, 131072 token slots), hidden 2048, expert FFN 768 (gate+up "
               "2048->1536, down 768->2048); grouped 32x32 2D-block FP4 (X, W round-to-nearest; "
               "dY stochastic)",
    "dense_7b_1d": "7B-class dense linears fwd+bwd (shapes and tensors of dense_7b) with the paper's "
                   "quantization placement: activations X in 1D FP4 (1x32 blocks for the forward "
                   "GEMM, 32x1 for the weight gradient), W and dY in 32x32 2D-block FP4 (X, W "
                   "round-to-nearest; dY stochastic)",
    "dense_7b_b64": "7B-class dense linears fwd+bwd (shapes and tensors of dense_7b) with 64x64 "
                    "2D-block FP4 for X, W and dY (the larger block of the block-size trade-off; "
                    "X, W round-to-nearest; dY stochastic)",
    "dense_7b_yq_fused": "7B-class dense linears fwd+bwd (shapes and tensors of dense_7b) with every forward "
                         "output Y (round to nearest) and every data gradient dX (stochastic rounding) "
                         "delivered in 32x32 2D-block FP4 for the next GEMM, quantized in the producing "
                         "GEMM's epilogue",
    "dense_7b_yq_separate": "the dense_7b_yq_fused step with Y and dX written in bf16 by their GEMMs and "
                            "quantized by separate quantizer launches",
    "mixed_7b": "7B-class block fwd+bwd, tokens 16384: Q/K projections in MXFP8 (E4M3, 1x32) "
                "and V, O, gate, up, down in 32x32 2D-block FP4 with stochastic rounding; "
                "bf16 inputs with outlier channels",
}

# what each kind of launch is measured against
KIND_PEAK = {"gemm_fp4": ("mfma", PEAK_FP4_TFLOPS, "TFLOP/s"),
             "gemm_fp4_yq": ("mfma", PEAK_FP4_TFLOPS, "TFLOP/s"),
             "gemm_fp4_dxq": ("mfma", PEAK_FP4_TFLOPS, "TFLOP/s"),
             "gemm_fp4_grouped": ("mfma", PEAK_FP4_TFLOPS, "TFLOP/s"),
             # ragged-K weight gradients: per expert a short K and a float32 output
             # of E x N x K_in, so the output writes bound them
             "gemm_fp4_grouped_k": ("hbm", PEAK_HBM_GBS, "GB/s"),
             "gemm_fp8": ("mfma", PEAK_FP8_TFLOPS, "TFLOP/s"),
             "quant_fp4": ("hbm", PEAK_HBM_GBS, "GB/s"),
             "quant_fp4_grouped": ("hbm", PEAK_HBM_GBS, "GB/s"),
             "quant_fp4_1d": ("hbm", PEAK_HBM_GBS, "GB/s"),
             "quant_mxfp8": ("hbm", PEAK_HBM_GBS, "GB/s")}
KIND_KERNEL = {"gemm_fp4": "gemm_fp4_persistent_kernel", "gemm_fp4_grouped": "gemm_fp4_persistent_kernel (grouped)",
               "gemm_fp4_grouped_k": "gemm_fp4_persistent_kernel (grouped, ragged K)",
               "gemm_fp4_yq": "gemm_fp4_persistent_kernel (FP4-quantizing epilogue)",
               "gemm_fp4_dxq": "gemm_fp4_persistent_kernel (FP4-quantizing epilogue, stochastic rounding)",
               "gemm_fp8": "gemm_fp8_256_kernel", "quant_fp4": "fp4_quantize_kernel",
               "quant_fp4_grouped": "fp4_quantize_kernel (grouped)",
               "quant_fp4_1d": "fp4_quantize_kernel (1D blocks)",
               "quant_mxfp8": "mxfp8_quantize_kernel"}


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=10)
    p.add_argument("--warmup", type=int, default=3)
    p.add_argument("--workload", default="dense_7b", choices=sorted(WORKLOAD_TEXT))
    p.add_argument("--also", default="dense_1b,tiny,moe_30b,mixed_7b,dense_7b_1d,dense_7b_b64,dense_7b_yq_fused,"
                                     "dense_7b_yq_separate",
                   help="further workloads measured in the same run (comma list, or 'none')")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--eager", action="store_true",
                   help="time the steps as eager launches instead of replays of one captured HIP graph")
    p.add_argument("--cpu-sample-tokens", type=int, default=256)
    p.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES")
    p.add_argument("--hot-loop", default="", choices=["", "gemm", "gemm_fp8", "quant", "quant_sr"],
                   help="run one kernel of the 7B QKV shape in a loop for --seconds (for sampling "
                        "power and clocks from outside) and print its rate")
    p.add_argument("--seconds", type=float, default=8.0)
    p.add_argument("--summarize-profiles", default="", metavar="DIR",
                   help="write profiles/ summaries from the rocprofv3 outputs in DIR")
    return p.parse_args()


def hot_loop(torch, kind: str, seconds: float):
    """One kernel of the 7B QKV projection (16384 x 4096 activations, 12288 x 4096
    weight) in a loop: the forward FP4 or MXFP8 GEMM, or the FP4 quantizer of X (round
    to nearest or stochastic).  Progress goes to stderr, the rate to stdout as one JSON line."""
    import synth
    import paper_2607_24953_amd as q2d
    dev = "cuda:0"
    X = synth.normal((16384, 4096), 1.0, 7001, torch.bfloat16, dev)
    W = synth.normal((12288, 4096), 0.02, 7002, torch.bfloat16, dev)
    qx = q2d.q2d_quantize(X, "rtn", 0, 0)
    qw = q2d.q2d_quantize(W, "rtn", 0, 1)
    Y = torch.empty(16384, 12288, dtype=torch.bfloat16, device=dev)
    if kind == "gemm_fp8":
        qx = q2d.mxfp8_quantize(X)
        qw = q2d.mxfp8_quantize(W)
    calls = {"gemm": lambda: q2d.q2d_gemm(qx, 0, qw, 0, out=Y),
             "gemm_fp8": lambda: q2d.q2d_gemm(qx, 0, qw, 0, out=Y),
             "quant": lambda: q2d.q2d_quantize(X, "rtn", 0, 0, out=qx),
             "quant_sr": lambda: q2d.q2d_quantize(X, "sr", 0, 0, out=qx)}
    call = calls[kind]
    for _ in range(3):
        call()
    torch.cuda.synchronize()
    print("hot loop %s: start" % kind, file=sys.stderr, flush=True)
    t0 = time.perf_counter()
    n = 0
    while time.perf_counter() - t0 < seconds:
        for _ in range(20):
            call()
        torch.cuda.synchronize()
        n += 20
    dt = (time.perf_counter() - t0) / n
    if kind.startswith("gemm"):
        rate, unit = 2.0 * 16384 * 12288 * 4096 / dt / 1e12, "TFLOP/s"
    else:
        rate, unit = 16384 * 4096 * 3.001 / dt / 1e9, "GB/s"
    print(json.dumps({"hot_loop": kind, "launches": n, "ms_per_launch": round(dt * 1e3, 4),
                      "rate": round(rate, 1), "unit": unit}), flush=True)


def copy_calibration(torch, nbytes: int, reps: int = 3):
    """A plain copy of nbytes (read nbytes, write nbytes) repeated `reps` times."""
    src = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes": nbytes, "reps": reps}), flush=True)


def quant_bytes(t, fmt="fp4") -> float:
    """Algorithmic bytes of one quantization: the input once, both code layouts, scales.
    FP4: two 4-bit layouts and one E8M0 byte per 32x32 block; 1D FP4: two 4-bit layouts
    and one E8M0 byte per 32 elements in each; MXFP8: two 8-bit layouts and one E8M0
    byte per 32 elements in each layout."""
    n = t.numel()
    if fmt == "mxfp8":
        return n * t.element_size() + 2.0 * n + 2.0 * n / 32.0
    if fmt == "fp4_1d":
        return n * t.element_size() + n * 0.5 * 2 + 2.0 * n / 32.0
    return n * t.element_size() + n * 0.5 * 2 + n / 1024.0


def gemm_bytes(a_elems, b_elems, c_bytes, fmt="fp4", a1d=False, b1d=False) -> float:
    """Algorithmic HBM bytes of one GEMM: both quantized operands once (codes and
    scales) and the output once (a1d / b1d: that FP4 operand has 1x32 blocks)."""
    if fmt == "mxfp8":
        return (a_elems + b_elems) * (1.0 + 1.0 / 32.0) + c_bytes
    return (a_elems * (0.5 + (1.0 / 32.0 if a1d else 1.0 / 1024.0)) +
            b_elems * (0.5 + (1.0 / 32.0 if b1d else 1.0 / 1024.0)) + c_bytes)


KIND_SOURCES = {"gemm_fp4": "gemm.hip", "gemm_fp4_grouped": "gemm.hip", "gemm_fp4_grouped_k": "gemm.hip", "gemm_fp8": "gemm.hip", "gemm_fp4_yq": "gemm.hip",
                "gemm_fp4_dxq": "gemm.hip",
                "quant_fp4": "quantize_fp4.hip", "quant_fp4_grouped": "quantize_fp4.hip",
                "quant_fp4_1d": "quantize_fp4.hip", "quant_mxfp8": "quantize_mxfp8.hip"}


def kind_hash(kind: str) -> str:
    return source_hash(KIND_SOURCES[kind], "device_common.hpp", "kernels.hpp")


def kind_of(kernel_name: str):
    """Launch kind of a libq2d kernel from its (demangled) name, None for other kernels."""
    import re
    m = re.search(r"gemm_fp4_persistent_kernel<([^>]*)>", kernel_name)
    if m:
        # template arguments: bf16 output, accumulate, grouped mode, 1D operands, quantized
        # output, stochastic rounding of it
        a = [t.strip() for t in m.group(1).split(",")]
        if len(a) > 5 and a[5] == "true":
            return "gemm_fp4_dxq"
        if len(a) > 4 and a[4] == "true":
            return "gemm_fp4_yq"
        return {"0": "gemm_fp4", "1": "gemm_fp4_grouped"}.get(a[2], "gemm_fp4_grouped_k")
    if "gemm_fp8_256_kernel" in kernel_name:
        return "gemm_fp8"
    m = re.search(r"gemm_kernel<(\d)", kernel_name)
    if m:
        return "gemm_fp4" if m.group(1) == "0" else "gemm_fp8"
    m = re.search(r"fp4_quantize_kernel<([^>]*)>", kernel_name)
    if m:
        # template arguments: element type, VEC, SR, ALIGNED8, GROUPED, column waves, 1D
        a = [t.strip() for t in m.group(1).split(",")]
        if a[6] == "true":
            return "quant_fp4_1d"
        return "quant_fp4_grouped" if a[4] == "true" else "quant_fp4"
    if "mxfp8_quantize_kernel" in kernel_name:
        return "quant_mxfp8"
    return None


def source_hash(*names) -> str:
    """Hash of the code of the named kernel sources: comments and whitespace are
    dropped first, so that an edit of a comment does not count as a change of
    the kernel the counters were taken on."""
    import re
    h = hashlib.sha256()
    for n in names:
        with open(os.path.join(HERE, "paper_2607_24953_amd", "csrc", n), encoding="utf-8") as f:
            text = f.read()
        text = re.sub(r"//[^\n]*|/\*.*?\*/", "", text, flags=re.S)
        h.update(re.sub(r"\s+", "", text).encode())
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


def attach_traffic(workload: str, kinds: dict):
    """Measured HBM bytes per launch of each kind (null unless measured on these sources)."""
    for kind, obj in kinds.items():
        tr = read_traffic("%s/%s" % (workload, kind), kind_hash(kind))
        obj["traffic"] = tr["bytes_per_launch"] if tr else None


class Step:
    """One fwd+bwd pass of a workload as a list of launches (kind, name, work, call);
    work is algorithmic flops (GEMMs) or bytes (quantizers)."""

    def __init__(self, q2d, torch, w):
        self.q2d, self.torch, self.w = q2d, torch, w
        self.dev = next(iter(w.tensors.values())).device
        self.ops = []
        self.events = []
        if w.name == "moe_30b":
            self._moe()
        else:
            self._dense()

    def _dense(self):
        q2d, torch, w, dev = self.q2d, self.torch, self.w, self.dev
        qt = {}
        fmt_of = lambda lin, name: lin.x_fmt if (name == lin.x and lin.x_fmt) else lin.fmt
        for lin in w.linears:
            for name in (lin.x, lin.w, lin.dy):
                fmt = fmt_of(lin, name)
                key = (name, fmt)
                if key in qt:
                    continue
                t = w.tensors[name]
                if fmt == "fp4_1d":
                    qt[key] = q2d.QTensor(q2d.FP4_1D, t.shape[0], t.shape[1], dev)
                    off = len(qt)
                    b = quant_bytes(t, "fp4_1d")
                    self.ops.append(("quant_fp4_1d", name + ".1d", b, b,
                                     lambda t=t, o=qt[key], m=w.rounding[name], off=off:
                                     q2d.q2d_quantize_1d(t, m, w.seed, off, out=o)))
                elif fmt == "mxfp8":
                    qt[key] = q2d.QTensor(q2d.MXFP8, t.shape[0], t.shape[1], dev)
                    b = quant_bytes(t, "mxfp8")
                    self.ops.append(("quant_mxfp8", name + ".mxfp8", b, b,
                                     lambda t=t, o=qt[key]: q2d.mxfp8_quantize(t, out=o)))
                else:
                    qt[key] = q2d.QTensor(q2d.FP4_2D, t.shape[0], t.shape[1], dev, w.block)
                    off = len(qt)
                    b = quant_bytes(t)
                    self.ops.append(("quant_fp4", name, b, b,
                                     lambda t=t, o=qt[key], m=w.rounding[name], off=off:
                                     q2d.q2d_quantize(t, m, w.seed, off, out=o, block=w.block)))
        for lin in w.linears:
            x1d = fmt_of(lin, lin.x) == "fp4_1d"
            qx, qw, qdy = qt[(lin.x, fmt_of(lin, lin.x))], qt[(lin.w, lin.fmt)], qt[(lin.dy, lin.fmt)]
            Y = torch.empty((lin.tokens, lin.n_out), dtype=torch.bfloat16, device=dev)
            dX = torch.empty((lin.tokens, lin.k_in), dtype=torch.bfloat16, device=dev)
            dW = torch.empty((lin.n_out, lin.k_in), dtype=torch.float32, device=dev)
            f = 2.0 * lin.tokens * lin.n_out * lin.k_in
            kind = "gemm_fp8" if lin.fmt == "mxfp8" else "gemm_fp4"
            T, N, K = lin.tokens, lin.n_out, lin.k_in
            y_out = w.extra.get("y_out")
            for nm, a, ta, b, tb, out, mnk, a1, b1 in (("fwd", qx, 0, qw, 0, Y, (T, N, K), x1d, False),
                                                       ("dX", qdy, 0, qw, 1, dX, (T, K, N), False, False),
                                                       ("dW", qdy, 1, qx, 1, dW, (N, K, T), False, x1d)):
                M_, N_, K_ = mnk
                if nm == "fwd" and y_out == "fused":
                    # Y leaves the epilogue as both FP4 layouts and the scale grids
                    qy = q2d.QTensor(q2d.FP4_2D, T, N, dev)
                    ab = gemm_bytes(M_ * K_, N_ * K_, M_ * N_ * (1.0 + 2.0 / 1024.0), lin.fmt, a1, b1)
                    self.ops.append(("gemm_fp4_yq", "%s.%s" % (lin.name, nm), f, ab,
                                     lambda a=a, b=b, qy=qy: q2d.q2d_gemm_quantized(a, 0, b, 0, "rtn", out=qy)))
                    continue
                if nm == "dX" and y_out == "fused":
                    # dX leaves stochastically rounded, keyed by its own storage index
                    qdx = q2d.QTensor(q2d.FP4_2D, T, K, dev)
                    ab = gemm_bytes(M_ * K_, N_ * K_, M_ * N_ * (1.0 + 2.0 / 1024.0), lin.fmt, a1, b1)
                    off = 100 + len(self.ops)
                    self.ops.append(("gemm_fp4_dxq", "%s.%s" % (lin.name, nm), f, ab,
                                     lambda a=a, b=b, q=qdx, off=off:
                                     q2d.q2d_gemm_quantized(a, 0, b, 1, "sr", out=q, seed=w.seed, offset=off)))
                    continue
                ab = gemm_bytes(M_ * K_, N_ * K_, out.numel() * out.element_size(), lin.fmt, a1, b1)
                self.ops.append((kind, "%s.%s" % (lin.name, nm), f, ab,
                                 lambda a=a, ta=ta, b=b, tb=tb, out=out:
                                 q2d.q2d_gemm(a, ta, b, tb, out=out)))
                if nm == "fwd" and y_out == "separate":
                    qy = q2d.QTensor(q2d.FP4_2D, T, N, dev)
                    qb = quant_bytes(Y)
                    self.ops.append(("quant_fp4", "%s.Y" % lin.name, qb, qb,
                                     lambda Y=Y, qy=qy: q2d.q2d_quantize(Y, "rtn", out=qy)))
                if nm == "dX" and y_out == "separate":
                    qdx = q2d.QTensor(q2d.FP4_2D, T, K, dev)
                    qb = quant_bytes(dX)
                    off = 100 + len(self.ops)
                    self.ops.append(("quant_fp4", "%s.dX_q" % lin.name, qb, qb,
                                     lambda dX=dX, q=qdx, off=off: q2d.q2d_quantize(dX, "sr", w.seed, off, out=q)))
        self.flops = float(w.gemm_flops)

    def _moe(self):
        q2d, torch, w, dev = self.q2d, self.torch, self.w, self.dev
        x = w.extra
        off = torch.tensor(x["offsets"], dtype=torch.int64, device=dev)
        E, S, Hd, F = x["experts"], x["slots"], x["hidden"], x["ffn"]
        qt = {}
        for i, name in enumerate(("X", "H", "dY_gu", "dY_d")):
            t = w.tensors[name]
            qt[name] = q2d.QTensor(q2d.FP4_2D, S, t.shape[1], dev, nseg=E)
            self.ops.append(("quant_fp4_grouped", name, quant_bytes(t), quant_bytes(t),
                             lambda t=t, o=qt[name], m=w.rounding[name], i=i:
                             q2d.q2d_grouped_quantize(t, off, m, w.seed, i, out=o)))
        for i, name in enumerate(("W_gu", "W_d")):
            t = w.tensors[name]
            qt[name] = q2d.QTensor(q2d.FP4_2D, t.shape[0], t.shape[1], dev)
            self.ops.append(("quant_fp4", name, quant_bytes(t), quant_bytes(t),
                             lambda t=t, o=qt[name], m=w.rounding[name], i=i:
                             q2d.q2d_quantize(t, m, w.seed, 4 + i, out=o)))
        bf, f32 = torch.bfloat16, torch.float32
        gemms = [("gate_up.fwd", "X", 0, "W_gu", 0, (S, 2 * F), bf, 2.0 * S * 2 * F * Hd),
                 ("down.fwd", "H", 0, "W_d", 0, (S, Hd), bf, 2.0 * S * Hd * F),
                 ("down.dX", "dY_d", 0, "W_d", 1, (S, F), bf, 2.0 * S * Hd * F),
                 ("gate_up.dX", "dY_gu", 0, "W_gu", 1, (S, Hd), bf, 2.0 * S * 2 * F * Hd),
                 ("gate_up.dW", "dY_gu", 1, "X", 1, (E * 2 * F, Hd), f32, 2.0 * S * 2 * F * Hd),
                 ("down.dW", "dY_d", 1, "H", 1, (E * Hd, F), f32, 2.0 * S * Hd * F)]
        self.flops = 0.0
        for nm, a, ta, b, tb, shape, dt, f in gemms:
            out = torch.empty(shape, dtype=dt, device=dev)
            ab = gemm_bytes(w.tensors[a].numel(), w.tensors[b].numel(),
                            out.numel() * out.element_size(), "fp4")
            ragged_k = ta == 1 and tb == 1
            self.ops.append(("gemm_fp4_grouped_k" if ragged_k else "gemm_fp4_grouped", nm, ab if ragged_k else f, ab,
                             lambda a=qt[a], ta=ta, b=qt[b], tb=tb, out=out:
                             q2d.q2d_grouped_gemm(a, ta, b, tb, off, out=out)))
            self.flops += f
        assert abs(self.flops - x["flops"]) < 1.0

    def run(self, record: bool):
        torch = self.torch
        for kind, name, work, abytes, call in self.ops:
            if record:
                e0 = torch.cuda.Event(enable_timing=True)
                e1 = torch.cuda.Event(enable_timing=True)
                e0.record()
                call()
                e1.record()
                self.events.append((kind, name, work, abytes, e0, e1))
            else:
                call()


def capture(step, torch):
    """The step's launches as one HIP graph (torch's graph capture on a side stream,
    after a warm-up there); the library allocates nothing and issues no memset, so
    a replay runs exactly the step's kernels without their host launch costs."""
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        step.run(record=False)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step.run(record=False)
    g.replay()
    torch.cuda.synchronize()
    return g


def measure(step, torch, steps: int, warmup: int, graph: bool = True) -> dict:
    """Wall time of `steps` whole steps (replays of the step's HIP graph, or eager
    launches), then the same steps launched eagerly with HIP events around every
    launch (on torch's current stream, the stream the launches go to)."""
    for _ in range(warmup):
        step.run(record=False)
    torch.cuda.synchronize()
    g = capture(step, torch) if graph else None
    t0 = time.perf_counter()
    for _ in range(steps):
        if g is not None:
            g.replay()
        else:
            step.run(record=False)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    del g
    step.events = []
    for _ in range(steps):
        step.run(record=True)
    torch.cuda.synchronize()
    kinds, names = {}, {}
    for kind, name, work, abytes, e0, e1 in step.events:
        ms = e0.elapsed_time(e1)
        k = kinds.setdefault(kind, [0.0, 0.0, 0, 0.0])
        k[0] += ms; k[1] += work; k[2] += 1; k[3] += abytes
        n = names.setdefault(name, [kind, 0.0, 0.0, 0])
        n[1] += ms; n[2] += work; n[3] += 1
    ms_per_step = wall * 1e3 / steps
    res = {"ms_per_step": ms_per_step, "value": step.flops / (ms_per_step * 1e-3) / 1e12,
           "quant_gb_per_step": sum(o[3] for o in step.ops if o[0].startswith("quant")) / 1e9,
           "kinds": {}, "per_kernel": {},
           # one dispatch per op: warm-up, (graph: side-stream warm-up and one untimed
           # replay,) timed steps, event-timed steps
           "launches": len(step.ops) * (warmup + 2 * steps + (2 if graph else 0))}
    for kind, (ms, work, n, abytes) in kinds.items():
        bound, peak, unit = KIND_PEAK[kind]
        scale = 1e12 if unit == "TFLOP/s" else 1e9
        ach = work / (ms * 1e-3) / scale
        res["kinds"][kind] = {"bound": bound, "kernel": KIND_KERNEL[kind], "achieved": round(ach, 2),
                              "peak": peak, "unit": unit, "frac": round(ach / peak, 4),
                              "launches_timed": n, "avg_launch_ms": round(ms / n, 5),
                              "work_per_launch": work / n, "algorithmic_bytes_per_launch": abytes / n,
                              "ms_per_step": round(ms / steps, 4)}
        if bound == "mfma":
            # both ceilings of a launch: its flops at the MFMA peak and its algorithmic
            # bytes (operands once, output once) at the HBM peak; a short-K GEMM whose
            # bf16 output outweighs its flops sits on the HBM side of the ridge
            t_mfma = work / n / (peak * 1e12)
            t_hbm = abytes / n / (PEAK_HBM_GBS * 1e9)
            res["kinds"][kind]["ideal_ms"] = {"mfma": round(t_mfma * 1e3, 5), "hbm": round(t_hbm * 1e3, 5)}
            res["kinds"][kind]["ridge_side"] = "hbm" if t_hbm > t_mfma else "mfma"
            res["kinds"][kind]["frac_of_roofline"] = round(max(t_mfma, t_hbm) / (ms / n * 1e-3), 4)
    for name, (kind, ms, work, n) in names.items():
        unit = KIND_PEAK[kind][2]
        rate = work / (ms * 1e-3) / (1e12 if unit == "TFLOP/s" else 1e9)
        res["per_kernel"][name] = {"ms": round(ms / n, 4), unit: round(rate, 1)}
    return res


def cpu_baseline(w, tokens: int):
    """The oracle (C quantizer with OpenMP, float64 numpy GEMMs) on the first `tokens`
    rows of every activation and gradient of the workload, full weights (dense FP4
    workloads only)."""
    import oracle
    if not w.linears or any(l.fmt != "fp4" for l in w.linears):
        return None
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


PROFILE_WORKLOADS = ("dense_7b", "dense_1b", "moe_30b", "mixed_7b", "dense_7b_1d", "dense_7b_b64",
                     "dense_7b_yq_fused")
PROFILE_FILES = {
    "dense_1b": [("fp4_kernels.dense_1b.md", ("gemm_fp4", "quant_fp4"))],
    "tiny": [("fp4_kernels.tiny.md", ("gemm_fp4", "quant_fp4"))],
    "dense_7b": [("gemm_fp4_persistent_kernel.dense_7b.md", ("gemm_fp4",)),
                 ("fp4_quantize_kernel.dense_7b.md", ("quant_fp4",))],
    "moe_30b": [("grouped_fp4_kernels.moe_30b.md", ("gemm_fp4_grouped", "gemm_fp4_grouped_k", "quant_fp4_grouped",
                                                    "quant_fp4"))],
    "dense_7b_1d": [("fp4_1d_kernels.dense_7b_1d.md", ("quant_fp4_1d", "gemm_fp4", "quant_fp4"))],
    "mixed_7b": [("mxfp8_kernels.mixed_7b.md", ("gemm_fp8", "quant_mxfp8", "gemm_fp4", "quant_fp4"))],
    "dense_7b_b64": [("block64_kernels.dense_7b_b64.md", ("quant_fp4", "gemm_fp4"))],
    "dense_7b_yq_fused": [("gemm_fp4_yq.dense_7b_yq_fused.md", ("gemm_fp4_yq", "gemm_fp4_dxq", "gemm_fp4",
                                                                 "quant_fp4"))],
    "dense_7b_yq_separate": [("gemm_fp4_yq.dense_7b_yq_separate.md", ("gemm_fp4", "quant_fp4"))],
}
PROFILE_COMMANDS = """cd /tmp && export TMPDIR=/tmp; R=/root/repo; O=${PROFILE_OUT:-$R/profile_runs}; mkdir -p $O
rocprofv3 --kernel-trace --stats --output-format csv -d $O/trace -o bench -- python3 $R/bench.py > $O/bench_trace.log 2>&1
for c in FETCH_SIZE WRITE_SIZE; do
  rocprofv3 --pmc $c --output-format csv -d $O/copy_$c -o copy -- python3 $R/bench.py --copy-calibration 1073741824 > $O/copy_$c.log 2>&1
  for wl in dense_7b dense_1b moe_30b mixed_7b dense_7b_1d dense_7b_b64 dense_7b_yq_fused; do
    rocprofv3 --pmc $c --output-format csv -d $O/${wl}_$c -o $wl -- python3 $R/bench.py --workload $wl --also none --steps 1 --warmup 0 --no-cpu-baseline > $O/${wl}_$c.log 2>&1
  done
done
rocprofv3 --pmc MfmaUtil LdsUtil LDSBankConflict LdsBankConflict --output-format csv -d $O/dense_7b_util -o dense_7b -- python3 $R/bench.py --workload dense_7b --also none --steps 1 --warmup 0 --no-cpu-baseline > $O/dense_7b_util.log 2>&1
rocprofv3 --pmc TCC_HIT_sum TCC_MISS_sum --output-format csv -d $O/dense_7b_l2 -o dense_7b -- python3 $R/bench.py --workload dense_7b --also none --steps 1 --warmup 0 --no-cpu-baseline > $O/dense_7b_l2.log 2>&1
rocprofv3 --pmc VALUBusy SALUBusy --output-format csv -d $O/dense_7b_valu -o dense_7b -- python3 $R/bench.py --workload dense_7b --also none --steps 1 --warmup 0 --no-cpu-baseline > $O/dense_7b_valu.log 2>&1
python3 $R/bench.py --summarize-profiles $O"""



def _json_line(path):
    with open(path) as f:
        for line in f:
            if line.startswith("{"):
                return json.loads(line)
    raise ValueError("no JSON line in " + path)


def _csv(dirname, suffix):
    import csv
    import glob
    paths = glob.glob(os.path.join(dirname, "*" + suffix))
    if len(paths) != 1:
        raise ValueError("expected one *%s in %s" % (suffix, dirname))
    with open(paths[0]) as f:
        return list(csv.DictReader(f))


def _counter_means(dirname, counter):
    """Mean KiB of `counter` per dispatch for every libq2d kind (and the copy kernel)."""
    acc = {}
    for r in _csv(dirname, "_counter_collection.csv"):
        if r["Counter_Name"] != counter:
            continue
        name = r["Kernel_Name"]
        kind = "copy" if "copyBuffer" in name else kind_of(name)
        if kind:
            a = acc.setdefault(kind, [0.0, 0])
            a[0] += float(r["Counter_Value"]); a[1] += 1
    return {k: (v[0] / v[1], v[1]) for k, v in acc.items()}


def _per_dispatch(dirname):
    """{dispatch id: (kind, duration ns, {counter: value})} of a counter-collection run."""
    out = {}
    for r in _csv(dirname, "_counter_collection.csv"):
        kind = kind_of(r["Kernel_Name"])
        if kind is None:
            continue
        dur = int(r["End_Timestamp"]) - int(r["Start_Timestamp"])
        k, _, cs = out.setdefault(int(r["Dispatch_Id"]), (kind, dur, {}))
        cs[r["Counter_Name"]] = cs.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    return out


UTIL_COUNTERS = ("MfmaUtil", "LdsUtil", "LDSBankConflict", "LdsBankConflict", "TCC_HIT_sum", "TCC_MISS_sum",
                 "VALUBusy", "SALUBusy")


def utilisation(d: str) -> dict:
    """Per kind of the dense 7B step, from the counter runs of PROFILE_COMMANDS:
    rocprofv3's MfmaUtil (% of SIMD cycles with the MFMA unit busy), LdsUtil,
    LDSBankConflict (% of GPU time LDS stalls on bank conflicts) and LdsBankConflict
    (conflicts per access), each averaged over dispatches weighted by duration, and
    the L2 hit rate TCC_HIT / (TCC_HIT + TCC_MISS)."""
    acc = {}
    for sub in ("dense_7b_util", "dense_7b_l2", "dense_7b_valu"):
        path = os.path.join(d, sub)
        if not os.path.isdir(path):
            continue
        for kind, dur, cs in _per_dispatch(path).values():
            a = acc.setdefault(kind, {c: [0.0, 0.0] for c in UTIL_COUNTERS})
            for c, v in cs.items():
                if c in a:
                    a[c][0] += v * (dur if not c.startswith("TCC") else 1.0)
                    a[c][1] += dur if not c.startswith("TCC") else 1.0
    out = {}
    for kind, a in acc.items():
        mean = {c: (v / w if w else None) for c, (v, w) in a.items()}
        hit, miss = a["TCC_HIT_sum"][0], a["TCC_MISS_sum"][0]
        out[kind] = {"mfma_util_pct": None if mean["MfmaUtil"] is None else round(mean["MfmaUtil"], 2),
                     "lds_util_pct": None if mean["LdsUtil"] is None else round(mean["LdsUtil"], 2),
                     "lds_bank_conflict_pct_time": None if mean["LDSBankConflict"] is None
                     else round(mean["LDSBankConflict"], 2),
                     "lds_bank_conflicts_per_access": None if mean["LdsBankConflict"] is None
                     else round(mean["LdsBankConflict"], 4),
                     "l2_hit_rate": round(hit / (hit + miss), 4) if hit + miss else None,
                     "valu_busy_pct": None if mean["VALUBusy"] is None else round(mean["VALUBusy"], 2),
                     "salu_busy_pct": None if mean["SALUBusy"] is None else round(mean["SALUBusy"], 2)}
    return out


def phase_owners(n_rows: int, phases) -> list:
    """Workload of each libq2d dispatch of a trace, in dispatch order: the workloads
    run one after the other and each reports how many dispatches it made."""
    total = sum(n for _, n in phases)
    if n_rows != total:
        raise ValueError("trace holds %d libq2d dispatches, the run reports %d" % (n_rows, total))
    return [wl for wl, n in phases for _ in range(n)]


def summarize_profiles(d: str, out_dir: str):
    """Turn the rocprofv3 outputs of PROFILE_COMMANDS into the text summaries of
    `out_dir`: per-kernel duration statistics next to the benchmark's own HIP-event
    averages, and HBM bytes per launch from FETCH_SIZE / WRITE_SIZE scaled by what
    the same counters read for a plain copy of known size."""
    cal = {}
    for c in ("FETCH_SIZE", "WRITE_SIZE"):
        nbytes = _json_line(os.path.join(d, "copy_%s.log" % c))["copy_calibration_bytes"]
        kib, n = _counter_means(os.path.join(d, "copy_" + c), c)["copy"]
        cal[c] = {"copy_bytes": nbytes, "counter_kib": kib, "factor": nbytes / (kib * 1024.0)}
    traffic = {"_calibration": cal}
    for wl in PROFILE_WORKLOADS:
        bj = _json_line(os.path.join(d, "%s_FETCH_SIZE.log" % wl))
        fetch = _counter_means(os.path.join(d, wl + "_FETCH_SIZE"), "FETCH_SIZE")
        write = _counter_means(os.path.join(d, wl + "_WRITE_SIZE"), "WRITE_SIZE")
        for kind in fetch:
            if kind == "copy" or kind not in write or kind not in bj["kinds"]:
                continue
            fb = fetch[kind][0] * 1024.0 * cal["FETCH_SIZE"]["factor"]
            wb = write[kind][0] * 1024.0 * cal["WRITE_SIZE"]["factor"]
            alg = bj["kinds"][kind]["algorithmic_bytes_per_launch"]
            traffic["%s/%s" % (wl, kind)] = {
                "bytes_per_launch": round(fb + wb), "fetch_bytes_per_launch": round(fb),
                "write_bytes_per_launch": round(wb), "algorithmic_bytes_per_launch": round(alg),
                "traffic_over_algorithmic": round((fb + wb) / alg, 3), "launches": fetch[kind][1],
                "source_hash": bj["source_hashes"][kind]}
    util = utilisation(d)
    if util:
        traffic["_utilisation_dense_7b"] = util
    with open(os.path.join(out_dir, "traffic.json"), "w") as f:
        json.dump(traffic, f, indent=1, sort_keys=True)
        f.write("\n")

    # kernel trace of the default benchmark run: the workloads run in order, each
    # making a known number of libq2d dispatches, which splits the trace by workload
    bt = _json_line(os.path.join(d, "bench_trace.log"))
    events = {bt["config"]["name"]: bt["kinds"]}
    phases = [(bt["config"]["name"], bt["launches"])]
    for wl, o in bt.get("other_workloads", {}).items():
        events[wl] = o["kinds"]
        phases.append((wl, o["launches"]))
    rows = _csv(os.path.join(d, "trace"), "_kernel_trace.csv")
    rows.sort(key=lambda r: int(r["Dispatch_Id"]))
    rows = [r for r in rows if kind_of(r["Kernel_Name"]) is not None]
    owner = phase_owners(len(rows), phases)
    durs = {}
    for r, phase in zip(rows, owner):
        kind = kind_of(r["Kernel_Name"])
        a = durs.setdefault((phase, kind), [0.0, 0])
        a[0] += (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-6; a[1] += 1
    stats = _csv(os.path.join(d, "trace"), "_kernel_stats.csv")
    for wl, files in PROFILE_FILES.items():
        for fname, kinds in files:
            out = ["# %s: %s" % (fname[:-3], ", ".join(kinds)), "",
                   "Workload: %s." % wl, "", "Commands (rocprofv3, ROCm 7.2, one MI355X):", "",
                   "```", PROFILE_COMMANDS, "```", "",
                   "## Kernel duration: rocprofv3 kernel trace vs the benchmark's HIP events", "",
                   "| kind | launches (trace, this workload) | avg ms (trace) | avg ms (HIP events) | achieved | frac of peak |",
                   "|---|---|---|---|---|---|"]
            for kind in kinds:
                ms, n = durs.get((wl, kind), (0.0, 0))
                ev = events.get(wl, {}).get(kind)
                if not n or not ev:
                    continue
                out.append("| %s | %d | %.4f | %.4f | %.1f %s | %.3f |" % (
                    kind, n, ms / n, ev["avg_launch_ms"], ev["achieved"], ev["unit"], ev["frac"]))
            out += ["", "## HBM traffic per launch (FETCH_SIZE x %.3f + WRITE_SIZE x %.3f, copy-calibrated)"
                    % (cal["FETCH_SIZE"]["factor"], cal["WRITE_SIZE"]["factor"]), "",
                    "| kind | measured bytes | algorithmic bytes | ratio |", "|---|---|---|---|"]
            for kind in kinds:
                t = traffic.get("%s/%s" % (wl, kind))
                if t:
                    out.append("| %s | %d | %d | %.3f |" % (kind, t["bytes_per_launch"],
                                                         t["algorithmic_bytes_per_launch"],
                                                         t["traffic_over_algorithmic"]))
            if wl == "dense_7b" and util:
                out += ["", "## MFMA, VALU and LDS utilisation, L2 hit rate (counter runs of this workload)", "",
                        "rocprofv3 derived counters per dispatch, averaged weighted by duration: MfmaUtil, "
                        "VALUBusy and SALUBusy (% of GPU time the vector / scalar ALUs issue), LdsUtil, "
                        "LDSBankConflict (% of GPU time LDS stalls on bank conflicts), LdsBankConflict "
                        "(conflicts per access); L2 hit rate = TCC_HIT / (TCC_HIT + TCC_MISS).",
                        "", "| kind | MfmaUtil % | VALUBusy % | SALUBusy % | LdsUtil % | LDSBankConflict % | "
                        "LdsBankConflict / access | L2 hit rate |", "|---|---|---|---|---|---|---|---|"]
                for kind in kinds:
                    u = util.get(kind)
                    if u:
                        out.append("| %s | %s | %s | %s | %s | %s | %s | %s |" % (
                            kind, u["mfma_util_pct"], u.get("valu_busy_pct"), u.get("salu_busy_pct"),
                            u["lds_util_pct"], u["lds_bank_conflict_pct_time"],
                            u["lds_bank_conflicts_per_access"], u["l2_hit_rate"]))
            out += ["", "## rocprofv3 --stats rows of these kernels (whole benchmark run, all workloads)", "",
                    "| kernel | calls | avg us | min us | max us |", "|---|---|---|---|---|"]
            for r in stats:
                if kind_of(r["Name"]) in kinds:
                    nm = r["Name"].replace("void q2d::(anonymous namespace)::", "").split("(")[0]
                    out.append("| %s | %s | %.1f | %.1f | %.1f |" % (
                        nm, r["Calls"], float(r["AverageNs"]) / 1e3, float(r["MinNs"]) / 1e3,
                        float(r["MaxNs"]) / 1e3))
            with open(os.path.join(out_dir, fname), "w") as f:
                f.write("\n".join(out) + "\n")


def main():
    args = parse()
    if args.summarize_profiles:
        summarize_profiles(args.summarize_profiles, os.path.join(HERE, "profiles"))
        return
    if args.gpus != 1:
        print("bench.py: this build measures one GPU only; --gpus %d is not supported" % args.gpus,
              file=sys.stderr)
        sys.exit(2)
    import torch
    if args.copy_calibration:
        copy_calibration(torch, args.copy_calibration)
        return
    if args.hot_loop:
        hot_loop(torch, args.hot_loop, args.seconds)
        return
    import synth
    import paper_2607_24953_amd as q2d

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    w = synth.WORKLOADS[args.workload](device=dev)
    step = Step(q2d, torch, w)
    res = measure(step, torch, args.steps, args.warmup, graph=not args.eager)
    print("bench: %s measured" % args.workload, file=sys.stderr, flush=True)
    kinds = res["kinds"]
    gemm_kind = max((k for k in kinds if k.startswith("gemm")), key=lambda k: kinds[k]["ms_per_step"])
    quant_kind = max((k for k in kinds if k.startswith("quant")), key=lambda k: kinds[k]["ms_per_step"])

    attach_traffic(args.workload, kinds)
    roof = dict(kinds[gemm_kind])
    quant = dict(kinds[quant_kind])

    rec = {
        "metric": "FP4 fwd+bwd linear TFLOP/s (7B shapes) + quantizer GB/s, % of roofline",
        "value": round(res["value"], 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(res["ms_per_step"], 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "fp4_e2m1 (fp32 accumulate)" if args.workload != "mixed_7b"
                 else "fp4_e2m1 + fp8_e4m3 (fp32 accumulate)",
        "data": "synthetic (seeded normals, bf16; no datasets or trained weights)",
        "config": {"workload": WORKLOAD_TEXT[args.workload], "name": args.workload,
                   "gemms_per_step": sum(1 for o in step.ops if o[0].startswith("gemm")),
                   "gemm_tflop_per_step": step.flops / 1e12,
                   "quantizer_gb_per_step": round(res["quant_gb_per_step"], 6),
                   "quantizations_per_step": sum(1 for o in step.ops if o[0].startswith("quant")),
                   "block": w.block,
                   "timed_as": "eager launches" if args.eager else "replays of one captured HIP graph per step"},
        "roofline": roof,
        "quantizer": quant,
        "kinds": kinds,
        "per_kernel": res["per_kernel"],
        "launches": res["launches"],
        "source_hashes": {k: kind_hash(k) for k in kinds},
    }
    others = [a for a in args.also.split(",") if a and a != "none" and a != args.workload]
    if others:
        del step, w
        torch.cuda.empty_cache()
        rec["other_workloads"] = {}
        for name in others:
            wo = synth.WORKLOADS[name](device=dev)
            so = Step(q2d, torch, wo)
            ro = measure(so, torch, args.steps, args.warmup, graph=not args.eager)
            print("bench: %s measured" % name, file=sys.stderr, flush=True)
            attach_traffic(name, ro["kinds"])
            rec["other_workloads"][name] = {
                "workload": WORKLOAD_TEXT[name], "TFLOP/s": round(ro["value"], 2),
                "ms_per_step": round(ro["ms_per_step"], 4), "gemm_tflop_per_step": so.flops / 1e12,
                "quantizer_gb_per_step": round(ro["quant_gb_per_step"], 6),
                "kinds": ro["kinds"], "per_kernel": ro["per_kernel"], "launches": ro["launches"]}
            del so, wo
            torch.cuda.empty_cache()
    if not args.no_cpu_baseline:
        rec["cpu_baseline"] = cpu_baseline(synth.WORKLOADS[args.workload](device=dev),
                                           args.cpu_sample_tokens)
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
