"""Forward/backward consistency of a quantized tensor (Sec. 2, "Scale
inconsistency under transposition" and "Bias induced by scale inconsistency";
Fig. 1 (c) and (d)).

A linear layer's forward GEMM reads one stored copy of each operand and the
backward GEMMs read the other.  ``transposition_consistency`` quantizes a
tensor, dequantizes both copies with ``q2d_dequantize`` (values and per-element
scale exponents, in the matrix's own orientation) and reports

* the scale-difference map e_fwd - e_bwd (in powers of two) and how much of the
  tensor it covers (Fig. 1 (c));
* the effective deviation |X_fwd - X_bwd| between the two quantized copies,
  relative to the tensor (Fig. 1 (d)).

2D blocks give exactly zero for both; 1D blocks (1x32 forward, 32x1 backward)
and MXFP8 do not.  ``python -m paper_2607_24953_amd.consistency`` prints the
report for the 7B-class synthetic tensors (activations with outlier channels,
weights, output gradients).
"""
from __future__ import annotations

import json
import sys

import torch

from . import mxfp8_quantize, q2d_dequantize, q2d_quantize, q2d_quantize_1d

FORMATS = ("fp4_2d", "fp4_2d_b64", "fp4_1d", "mxfp8")


def quantize(x: torch.Tensor, fmt: str, mode: str = "rtn", seed: int = 0, offset: int = 0):
    if fmt == "fp4_2d":
        return q2d_quantize(x, mode, seed, offset)
    if fmt == "fp4_2d_b64":
        return q2d_quantize(x, mode, seed, offset, block=64)
    if fmt == "fp4_1d":
        return q2d_quantize_1d(x, mode, seed, offset)
    if fmt == "mxfp8":
        return mxfp8_quantize(x)
    raise ValueError("unknown format " + fmt)


def transposition_consistency(x: torch.Tensor, fmt: str = "fp4_2d", mode: str = "rtn", seed: int = 0,
                              offset: int = 0, window: int = 64) -> dict:
    """Statistics of the two stored copies of ``x`` quantized in ``fmt`` (see the
    module docstring); ``window`` x ``window`` corners of both maps are returned as
    CPU tensors under "maps"."""
    q = quantize(x, fmt, mode, seed, offset)
    v0, e0 = q2d_dequantize(q, 0, torch.float32, exps=True)
    v1, e1 = q2d_dequantize(q, 1, torch.float32, exps=True)
    finite = (e0 != -128) & (e1 != -128)
    de = torch.where(finite, e0.to(torch.int16) - e1.to(torch.int16), torch.zeros_like(e0, dtype=torch.int16))
    dv = torch.where(finite, v0 - v1, torch.zeros_like(v0))
    xf = torch.where(finite, x.float(), torch.zeros_like(v0))
    xn = float(torch.linalg.vector_norm(xf.double()))
    n = x.numel()
    out = {
        "format": fmt, "shape": list(x.shape), "mode": mode,
        "scale_mismatch_fraction": float((de != 0).sum()) / n,
        "scale_diff_mean_abs": float(de.abs().double().mean()),
        "scale_diff_max_abs": int(de.abs().max()),
        "values_differ_fraction": float((dv != 0).sum()) / n,
        "deviation_rel_frobenius": float(torch.linalg.vector_norm(dv.double())) / (xn if xn > 0 else 1.0),
        "deviation_max_abs": float(dv.abs().max()),
        "quant_error_fwd_rel_frobenius":
            float(torch.linalg.vector_norm((torch.where(finite, v0, xf) - xf).double())) / (xn if xn > 0 else 1.0),
        "maps": {"scale_diff": de[:window, :window].cpu(), "deviation": dv[:window, :window].abs().cpu()},
    }
    del q, v0, v1, e0, e1
    return out


def main(argv=None) -> int:
    import os
    sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    import synth
    dev = torch.device("cuda:0")
    T, H = 16384, 4096
    tensors = {
        "X (activation, 1% outlier channels)":
            synth.add_outlier_channels(synth.normal((T, H), 1.0, 4001, torch.bfloat16, device=dev), 4002),
        "W (weight, N(0, 0.02))": synth.normal((3 * H, H), 0.02, 4003, torch.bfloat16, device=dev),
        "dY (output gradient, N(0, 1e-3))": synth.normal((T, 3 * H), 1e-3, 4004, torch.bfloat16, device=dev),
    }
    for name, t in tensors.items():
        for fmt in FORMATS:
            r = transposition_consistency(t, fmt)
            r.pop("maps")
            r["tensor"] = name
            print(json.dumps(r), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
