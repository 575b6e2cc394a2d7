"""PyTorch autograd form of the quantized linear layer (Sec. 3; App. C, App. E).

``Q2DLinear`` is a bias-free linear layer y = x W^T whose forward and backward
GEMMs run on quantized operands through ``q2d_linear_fwd`` / ``q2d_linear_bwd``:

* forward: X and W are quantized (round to nearest by default, the forward
  placement of App. E), Y = Q(X) Q(W)^T;
* backward: dY is quantized (stochastic rounding by default, App. E) and
  dX = Q(dY) Q(W), dW = Q(dY)^T Q(X) reuse the forward's quantized copies
  transposed (the 2D blocks keep their scales; Sec. 3);
* the straight-through estimator (Sec. 3) treats the quantizer as the identity:
  the gradients above are returned for x and W as they are.

Each call draws fresh stochastic-rounding streams: the layer's seed with
offsets 3n, 3n+1, 3n+2 for X, W and dY of its n-th forward call.  A layer built
without a seed takes the next value of a process-wide counter, so the layers of
a model draw independent streams (App. E asks for unbiased, independent
rounding; one seed shared by every layer would give the n-th gradients of all
layers the same random bits at the same storage indices).  The weight
(the master copy, usually float32) is cast to the input's dtype (float32 or
bfloat16) before quantization; Y and dX have the input's dtype, dW is computed
in float32 and cast to the weight's dtype.

Options mirror the paper's ablations: ``mode_*`` "rtn" / "sr" choose the
rounding per operand, the "-floor" variants the scale rule that the
truncation-free ablation goes back to; ``activations="1d"`` quantizes X in 1D
blocks (App. C, "Activations"); ``block=64`` uses 64 x 64 blocks (Table 4).
"""
from __future__ import annotations

import itertools
import math

import torch

from . import FP4_1D, FP4_2D, Q2DError, q2d_linear_bwd, q2d_linear_fwd

_DTYPES = (torch.float32, torch.bfloat16)


class _Q2DLinearFunction(torch.autograd.Function):
    @staticmethod
    def forward(ctx, x, weight, layer):
        K = x.shape[-1]
        if K != weight.shape[1]:
            raise Q2DError("input features %d != weight columns %d" % (K, weight.shape[1]))
        lead = x.shape[:-1]
        dt = x.dtype if x.dtype in _DTYPES else torch.float32
        x2 = x.reshape(-1, K).to(dt).contiguous()
        w = weight.detach().to(dt).contiguous()
        n = layer._calls
        layer._calls += 1
        Y, qX, qW = q2d_linear_fwd(x2, w, layer.mode_x, layer.mode_w, layer.seed, 3 * n, 3 * n + 1,
                                   y_dtype=dt, fmt_x=FP4_1D if layer.activations == "1d" else FP4_2D,
                                   block=layer.block)
        ctx.qX, ctx.qW = qX, qW
        ctx.layer, ctx.offset_dy = layer, 3 * n + 2
        ctx.x_shape, ctx.x_dtype, ctx.w_dtype, ctx.dt = x.shape, x.dtype, weight.dtype, dt
        return Y.reshape(*lead, weight.shape[0])

    @staticmethod
    def backward(ctx, dY):
        layer = ctx.layer
        N = dY.shape[-1]
        dY2 = dY.reshape(-1, N).to(ctx.dt).contiguous()
        dX, dW, _ = q2d_linear_bwd(dY2, ctx.qX, ctx.qW, layer.mode_dy, layer.seed, ctx.offset_dy,
                                   dx_dtype=ctx.dt, dw_dtype=torch.float32, block=layer.block)
        ctx.qX = ctx.qW = None
        return dX.reshape(ctx.x_shape).to(ctx.x_dtype), dW.to(ctx.w_dtype), None


# seeds of layers built without one (distinct per layer within a process)
_SEEDS = itertools.count(0x5EED0001)


class Q2DLinear(torch.nn.Module):
    """Bias-free linear layer on 2D-block FP4 GEMMs (see the module docstring)."""

    def __init__(self, in_features: int, out_features: int, *, mode_x: str = "rtn", mode_w: str = "rtn",
                 mode_dy: str = "sr", activations: str = "2d", block: int = 32, seed: int | None = None,
                 device=None, dtype=torch.float32):
        super().__init__()
        if activations not in ("2d", "1d"):
            raise ValueError("activations must be '2d' or '1d'")
        if seed is None:
            seed = next(_SEEDS)
        self.in_features, self.out_features = in_features, out_features
        self.mode_x, self.mode_w, self.mode_dy = mode_x, mode_w, mode_dy
        self.activations, self.block, self.seed = activations, block, seed
        self.weight = torch.nn.Parameter(torch.empty((out_features, in_features), device=device, dtype=dtype))
        self._calls = 0
        self.reset_parameters()

    def reset_parameters(self):
        torch.nn.init.kaiming_uniform_(self.weight, a=math.sqrt(5))

    def forward(self, x: torch.Tensor) -> torch.Tensor:
        return _Q2DLinearFunction.apply(x, self.weight, self)

    def extra_repr(self) -> str:
        return "in=%d, out=%d, x=%s, w=%s, dy=%s, activations=%s, block=%d, seed=%#x" % (
            self.in_features, self.out_features, self.mode_x, self.mode_w, self.mode_dy,
            self.activations, self.block, self.seed)
