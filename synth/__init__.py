"""Seeded synthetic inputs shared by the tests, the benchmark and the smoke check.

This module only draws random tensors with the shapes and value distributions of
the linear-layer operands of the paper's training runs (OLMo-1B, OLMo-7B, a
Qwen-30B-class MoE; Sec. 4.1 and Table 5).  It holds none of the quantization
method's arithmetic, so both the CPU oracle and the HIP path can consume its
output without sharing any code with each other.

Recipe (stated once here, repeated in the design notes):
  * every tensor has its own seed, ``1000 * workload_id + tensor_index``;
  * values are float32 normals multiplied by the stated standard deviation and
    then cast to bfloat16 with round-to-nearest-even (the Tiny workload stays
    float32);
  * activations X of the 7B-class workloads carry outlier channels: 1 % of the
    input channels (``round(0.01 * K_in)``, picked by ``randperm``) are replaced
    by 20 x Student-t(nu=3) samples (t = z / sqrt(chi2_3 / 3));
  * MoE routing: expert weights p_r proportional to r**-1.1 over ranks
    r = 1..E, ranks permuted by the seed, every token picks 8 distinct experts
    by Gumbel-top-8; the per-expert counts define the row segments.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np
import torch

__all__ = [
    "normal", "add_outlier_channels", "moe_counts", "segment_offsets",
    "Workload", "student_t", "regression_task", "sparse_regression_task", "tiny", "dense_1b", "dense_7b", "dense_7b_1d", "dense_7b_b64", "dense_7b_yq", "moe_30b", "mixed_7b", "WORKLOADS",
]


def _gen(seed: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    return g


def normal(shape, std: float, seed: int, dtype=torch.bfloat16, device="cpu") -> torch.Tensor:
    """N(0, std^2) samples drawn in float32 and cast to ``dtype`` (RNE for bf16)."""
    g = _gen(seed, device)
    x = torch.randn(tuple(shape), generator=g, device=device, dtype=torch.float32)
    if std != 1.0:
        x.mul_(std)
    return x.to(dtype)


def add_outlier_channels(x: torch.Tensor, seed: int, frac: float = 0.01,
                         scale: float = 20.0, nu: int = 3) -> torch.Tensor:
    """Replace ``round(frac * cols)`` columns of ``x`` with ``scale`` x Student-t(nu)."""
    rows, cols = x.shape
    n = int(round(frac * cols))
    if n == 0:
        return x
    g = _gen(seed, x.device)
    idx = torch.randperm(cols, generator=g, device=x.device)[:n]
    z = torch.randn((rows, n), generator=g, device=x.device, dtype=torch.float32)
    chi2 = torch.zeros((rows, n), device=x.device, dtype=torch.float32)
    for _ in range(nu):
        w = torch.randn((rows, n), generator=g, device=x.device, dtype=torch.float32)
        chi2.add_(w * w)
    t = z / torch.sqrt(chi2 / nu)
    x[:, idx] = (scale * t).to(x.dtype)
    return x


def student_t(shape, nu: int, seed: int, device="cpu") -> torch.Tensor:
    """Float32 Student-t(nu) samples: z / sqrt(chi2_nu / nu) from seeded normals."""
    g = _gen(seed, device)
    z = torch.randn(tuple(shape), generator=g, device=device, dtype=torch.float32)
    chi2 = torch.zeros(tuple(shape), device=device, dtype=torch.float32)
    for _ in range(nu):
        w = torch.randn(tuple(shape), generator=g, device=device, dtype=torch.float32)
        chi2.add_(w * w)
    return z / torch.sqrt(chi2 / nu)


def regression_task(tokens: int, k_in: int, n_out: int, noise: float, nu: int, seed: int, device="cpu"):
    """Teacher-student linear regression: X ~ N(0, 1) [tokens, k_in], teacher
    W* ~ N(0, 1/k_in) [n_out, k_in], targets X W*^T + noise * Student-t(nu)
    (heavy-tailed residuals, so the output gradients of a 32 x 32 block span a
    wide range).  Returns float32 (X, W*, Y)."""
    X = normal((tokens, k_in), 1.0, seed, torch.float32, device)
    W = normal((n_out, k_in), 1.0 / float(k_in) ** 0.5, seed + 1, torch.float32, device)
    Y = X @ W.t()
    if noise:
        Y = Y + noise * student_t((tokens, n_out), nu, seed + 2, device)
    return X, W, Y


def sparse_regression_task(tokens: int, k_in: int, n_out: int, nnz: int, lo: float, hi: float,
                           background: float, seed: int, device="cpu"):
    """Teacher-student linear regression on sparse large features: every row of
    X has `nnz` entries of magnitude uniform in [lo, hi) with random signs at
    random positions, the rest N(0, background^2); teacher W* ~ N(0, 1/k_in);
    targets X W*^T (no noise).  Returns float32 (X, W*, Y)."""
    g = _gen(seed, device)
    X = background * torch.randn((tokens, k_in), generator=g, device=device, dtype=torch.float32)
    pos = torch.rand((tokens, k_in), generator=g, device=device).argsort(dim=1)[:, :nnz]
    mag = lo + (hi - lo) * torch.rand((tokens, nnz), generator=g, device=device)
    sgn = torch.where(torch.rand((tokens, nnz), generator=g, device=device) < 0.5, -1.0, 1.0)
    X.scatter_(1, pos, mag * sgn)
    W = normal((n_out, k_in), 1.0 / float(k_in) ** 0.5, seed + 1, torch.float32, device)
    return X, W, X @ W.t()


def moe_counts(tokens: int = 16384, experts: int = 128, topk: int = 8,
               s: float = 1.1, seed: int = 0) -> np.ndarray:
    """Per-expert token counts from Zipf(s)-weighted Gumbel-top-k routing."""
    rng = np.random.Generator(np.random.PCG64(seed))
    ranks = rng.permutation(experts) + 1
    logp = -s * np.log(ranks.astype(np.float64))
    gumbel = -np.log(-np.log(rng.random((tokens, experts))))
    choice = np.argpartition(-(logp[None, :] + gumbel), topk - 1, axis=1)[:, :topk]
    counts = np.bincount(choice.ravel(), minlength=experts).astype(np.int64)
    assert counts.sum() == tokens * topk
    return counts


def segment_offsets(counts) -> np.ndarray:
    """Row offsets (len E+1) of expert segments stored back to back."""
    off = np.zeros(len(counts) + 1, dtype=np.int64)
    off[1:] = np.cumsum(np.asarray(counts, dtype=np.int64))
    return off


@dataclass
class Linear:
    """Operands of one linear layer Y = X W^T with N_out x K_in weight W."""
    name: str
    x: str
    w: str
    dy: str
    tokens: int
    n_out: int
    k_in: int
    fmt: str = "fp4"          # "fp4" (2D-block FP4) or "mxfp8"
    x_fmt: str = ""           # format of X when it differs: "fp4_1d" (1D-block FP4)

    @property
    def flops(self) -> int:
        # forward, data gradient and weight gradient GEMMs, 2*M*N*K each
        return 3 * 2 * self.tokens * self.n_out * self.k_in


@dataclass
class Workload:
    name: str
    tensors: dict = field(default_factory=dict)     # name -> torch.Tensor
    linears: list = field(default_factory=list)     # list[Linear]
    rounding: dict = field(default_factory=dict)    # tensor name -> "rtn" | "sr"
    seed: int = 0                                   # Philox seed for SR
    extra: dict = field(default_factory=dict)
    block: int = 32                                 # 2D block edge (32, or 64)

    @property
    def gemm_flops(self) -> int:
        return sum(l.flops for l in self.linears)


def tiny(device="cpu") -> Workload:
    """W 256x256 ~N(0,0.02), X 128x256 ~N(0,1), dY 128x256 ~N(0,1e-3), float32."""
    t = {
        "W": normal((256, 256), 0.02, 1000, torch.float32, device),
        "X": normal((128, 256), 1.0, 1001, torch.float32, device),
        "dY": normal((128, 256), 1e-3, 1002, torch.float32, device),
    }
    lin = [Linear("tiny", "X", "W", "dY", 128, 256, 256)]
    return Workload("tiny", t, lin, {k: "sr" for k in t}, seed=0)


def dense_1b(device="cpu") -> Workload:
    """1B-class MLP: tokens 8192, hidden 2048, FFN 5632, bf16, SR on every operand."""
    T, H, F = 8192, 2048, 5632
    t = {
        "X": normal((T, H), 1.0, 2000, device=device),
        "H": normal((T, F), 1.0, 2001, device=device),
        "W_up": normal((F, H), 0.02, 2002, device=device),
        "W_down": normal((H, F), 0.02, 2003, device=device),
        "dY_up": normal((T, F), 1e-3, 2004, device=device),
        "dY_down": normal((T, H), 1e-3, 2005, device=device),
    }
    lin = [Linear("up", "X", "W_up", "dY_up", T, F, H),
           Linear("down", "H", "W_down", "dY_down", T, H, F)]
    return Workload("dense_1b", t, lin, {k: "sr" for k in t}, seed=2)


def _dense_7b_tensors(cfg: int, device, names_w, names_dy):
    T, H, F = 16384, 4096, 11008
    t = {}
    t["X_qkv"] = normal((T, H), 1.0, 1000 * cfg + 0, device=device)
    t["X_o"] = normal((T, H), 1.0, 1000 * cfg + 1, device=device)
    t["X_gu"] = normal((T, H), 1.0, 1000 * cfg + 2, device=device)
    t["X_down"] = normal((T, F), 1.0, 1000 * cfg + 3, device=device)
    for i, key in enumerate(("X_qkv", "X_o", "X_gu", "X_down")):
        add_outlier_channels(t[key], 1000 * cfg + 50 + i)
    shapes_w = {"W_qkv": (3 * H, H), "W_q": (H, H), "W_k": (H, H), "W_v": (H, H),
                "W_o": (H, H), "W_gate": (F, H), "W_up": (F, H), "W_down": (H, F)}
    shapes_dy = {"dY_qkv": (T, 3 * H), "dY_q": (T, H), "dY_k": (T, H), "dY_v": (T, H),
                 "dY_o": (T, H), "dY_gate": (T, F), "dY_up": (T, F), "dY_down": (T, H)}
    for i, key in enumerate(names_w):
        t[key] = normal(shapes_w[key], 0.02, 1000 * cfg + 10 + i, device=device)
    for i, key in enumerate(names_dy):
        t[key] = normal(shapes_dy[key], 1e-3, 1000 * cfg + 30 + i, device=device)
    return t


def dense_7b(device="cpu") -> Workload:
    """7B-class linears: QKV, O, gate, up, down at tokens 16384, hidden 4096, FFN 11008.

    X and W are rounded to nearest, dY stochastically (forward vs backward rounding)."""
    T, H, F = 16384, 4096, 11008
    t = _dense_7b_tensors(3, device, ("W_qkv", "W_o", "W_gate", "W_up", "W_down"),
                          ("dY_qkv", "dY_o", "dY_gate", "dY_up", "dY_down"))
    lin = [Linear("qkv", "X_qkv", "W_qkv", "dY_qkv", T, 3 * H, H),
           Linear("o", "X_o", "W_o", "dY_o", T, H, H),
           Linear("gate", "X_gu", "W_gate", "dY_gate", T, F, H),
           Linear("up", "X_gu", "W_up", "dY_up", T, F, H),
           Linear("down", "X_down", "W_down", "dY_down", T, H, F)]
    rnd = {k: ("sr" if k.startswith("dY") else "rtn") for k in t}
    return Workload("dense_7b", t, lin, rnd, seed=3)


def dense_7b_1d(device="cpu") -> Workload:
    """The dense_7b tensors and linears with the paper's activation placement: X in
    1D-block FP4 (1x32 along K_in for the forward GEMM, 32x1 along tokens for the
    weight gradient), W and dY in 2D blocks."""
    w = dense_7b(device)
    for lin in w.linears:
        lin.x_fmt = "fp4_1d"
    w.name = "dense_7b_1d"
    return w


def dense_7b_b64(device="cpu") -> Workload:
    """The dense_7b tensors and linears with 64 x 64 blocks for X, W and dY (the larger
    block of the block-size trade-off, Table 4)."""
    w = dense_7b(device)
    w.block = 64
    w.name = "dense_7b_b64"
    return w


def dense_7b_yq(device="cpu", fused: bool = True) -> Workload:
    """The dense_7b tensors and linears with every forward output Y (round to
    nearest) and every data gradient dX (stochastic rounding) delivered in
    2D-block FP4 for the next GEMM: quantized in the producing GEMM's epilogue
    (fused) or by a separate quantization of the bf16 result."""
    w = dense_7b(device)
    w.extra["y_out"] = "fused" if fused else "separate"
    w.name = "dense_7b_yq_fused" if fused else "dense_7b_yq_separate"
    return w


def mixed_7b(device="cpu") -> Workload:
    """7B block with Q/K projections in MXFP8 and V, O, gate, up, down in 2D-block FP4 (SR)."""
    T, H, F = 16384, 4096, 11008
    t = _dense_7b_tensors(5, device,
                          ("W_q", "W_k", "W_v", "W_o", "W_gate", "W_up", "W_down"),
                          ("dY_q", "dY_k", "dY_v", "dY_o", "dY_gate", "dY_up", "dY_down"))
    lin = [Linear("q", "X_qkv", "W_q", "dY_q", T, H, H, fmt="mxfp8"),
           Linear("k", "X_qkv", "W_k", "dY_k", T, H, H, fmt="mxfp8"),
           Linear("v", "X_qkv", "W_v", "dY_v", T, H, H),
           Linear("o", "X_o", "W_o", "dY_o", T, H, H),
           Linear("gate", "X_gu", "W_gate", "dY_gate", T, F, H),
           Linear("up", "X_gu", "W_up", "dY_up", T, F, H),
           Linear("down", "X_down", "W_down", "dY_down", T, H, F)]
    return Workload("mixed_7b", t, lin, {k: "sr" for k in t}, seed=5)


def moe_30b(device="cpu", tokens: int = 16384, experts: int = 128, topk: int = 8,
            hidden: int = 2048, ffn: int = 768) -> Workload:
    """30B-class MoE expert FFN: 128 experts of FFN 768, top-8 Zipf(1.1) routing.

    Grouped tensors hold the token slots of all experts back to back (segment
    offsets in ``extra['offsets']``); expert weights are stacked along rows."""
    counts = moe_counts(tokens, experts, topk, 1.1, seed=0)
    off = segment_offsets(counts)
    S = int(off[-1])
    t = {
        "X": normal((S, hidden), 1.0, 4000, device=device),
        "W_gu": normal((experts * 2 * ffn, hidden), 0.02, 4001, device=device),
        "H": normal((S, ffn), 1.0, 4002, device=device),
        "W_d": normal((experts * hidden, ffn), 0.02, 4003, device=device),
        "dY_gu": normal((S, 2 * ffn), 1e-3, 4004, device=device),
        "dY_d": normal((S, hidden), 1e-3, 4005, device=device),
    }
    rnd = {k: ("sr" if k.startswith("dY") else "rtn") for k in t}
    w = Workload("moe_30b", t, [], rnd, seed=4)
    w.extra = {"counts": counts, "offsets": off, "experts": experts, "hidden": hidden,
               "ffn": ffn, "slots": S}
    w.extra["flops"] = 3 * 2 * S * (2 * ffn * hidden + hidden * ffn)
    return w


WORKLOADS = {"tiny": tiny, "dense_1b": dense_1b, "dense_7b": dense_7b, "dense_7b_1d": dense_7b_1d,
             "dense_7b_b64": dense_7b_b64, "moe_30b": moe_30b, "mixed_7b": mixed_7b,
             "dense_7b_yq_fused": lambda device="cpu": dense_7b_yq(device, True),
             "dense_7b_yq_separate": lambda device="cpu": dense_7b_yq(device, False)}
