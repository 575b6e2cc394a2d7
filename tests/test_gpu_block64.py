"""GPU parity of 64 x 64 blocks (the larger block of the block-size trade-off,
Table 4) against the oracle.

Quantization: every byte of the four buffers (the scale grids stay 32-granular,
each 64 x 64 block's byte in its four entries) equal to the oracle's, for
ragged shapes (64-blocks cut by the matrix edge and by the 128-row tiles of the
kernel), both dtypes, both rounding modes, transposed and strided views, a
non-finite value in one 32 x 32 quarter of a block, and full-size 7B-class
tensors.

GEMMs: block-64 operands, alone and mixed with block-32 and 1D ones, on the
small-problem and the persistent kernel, and the linear layer with 64 x 64
blocks, against the float64 oracle GEMM (relative Frobenius error <= 1e-5 for
float32 output).
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from helpers import assert_same_bytes, gpu_buffers, poison, rel_frob

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
TOL = 1e-5


@pytest.fixture(scope="module")
def q2d():
    import paper_2607_24953_amd as q
    return q


def run_case(q2d, x_dev, mode, seed=0, offset=0, label="", x_cpu=None):
    q = q2d.QTensor(q2d.FP4_2D, x_dev.shape[0], x_dev.shape[1], x_dev.device, 64)
    poison(q)
    q2d.q2d_quantize(x_dev, mode, seed, offset, out=q, block=64)
    got = gpu_buffers(q)
    if x_cpu is None:
        assert x_dev.is_contiguous()
        x_cpu = x_dev.cpu()
    assert x_cpu.stride() == x_dev.stride()
    want = oracle.quantize_fp4_2d(x_cpu, mode, seed, offset, block=64)
    assert_same_bytes(got, want, label)


SHAPES = [(128, 256), (64, 64), (100, 70), (33, 129), (1, 5), (257, 31), (300, 1000),
          (192, 320), (129, 4097)]


@pytest.mark.parametrize("shape", SHAPES)
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("mode", ["rtn", "sr"])
def test_quantize_block64(q2d, shape, dtype, mode):
    x = synth.normal(shape, 1.0, 300 + shape[0], dtype, device=DEV)
    synth.add_outlier_channels(x, 8, frac=0.02)
    run_case(q2d, x, mode, 77, 3, "%s %s %s" % (shape, dtype, mode))


@pytest.mark.parametrize("mode", ["rtn", "sr"])
def test_quantize_block64_views(q2d, mode):
    base = synth.normal((200, 300), 1.0, 61, torch.bfloat16)
    bd = base.to(DEV)
    run_case(q2d, bd.t(), mode, 4, 5, "transposed view", x_cpu=base.t())
    run_case(q2d, bd[:, ::2], mode, 4, 5, "column-strided view", x_cpu=base[:, ::2])
    run_case(q2d, bd[10:150, 7:290], mode, 4, 5, "offset view", x_cpu=base[10:150, 7:290])


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_special_values_block64(q2d, dtype):
    """A NaN or infinity in one 32 x 32 quarter marks the whole 64 x 64 block (all four
    scale entries 0xFF, all its codes 0); zero and tiny blocks."""
    x = synth.normal((192, 256), 1.0, 62, torch.float32)
    x[3, 40] = float("nan")            # block (0, 0), quarter (0, 1)
    x[100, 7] = float("inf")           # block (1, 0), quarter (3, 0)
    x[70, 200] = -float("inf")         # block (1, 3), quarter (2, 6)
    x[128:192, 128:192] = 0.0
    x[128:192, 0:64] = 1e-30
    xd = x.to(dtype).to(DEV)
    for mode in ("rtn", "sr"):
        run_case(q2d, xd, mode, 1, 2, "special %s" % mode)


def test_full_size_7b_block64(q2d):
    """The 7B-class QKV input and FFN weight at full size, all bytes."""
    x = synth.add_outlier_channels(synth.normal((16384, 4096), 1.0, 3011, torch.bfloat16), 3012)
    print("block64 X 16384x4096", flush=True)
    run_case(q2d, x.to(DEV), "rtn", 0, 0, "7B X block 64")
    w = synth.normal((11008, 4096), 0.02, 3013, torch.bfloat16)
    print("block64 W 11008x4096", flush=True)
    run_case(q2d, w.to(DEV), "sr", 5, 1, "7B W block 64")
    del x, w
    torch.cuda.empty_cache()


# ------------------------------------------------------------------ GEMMs

def _quant(q2d, x, fmt, mode, seed=0, offset=0):
    if fmt == "fp4_1d":
        q = q2d.q2d_quantize_1d(x, mode, seed, offset)
        o = oracle.quantize_fp4_1d(x.cpu(), mode, seed, offset)
    else:
        blk = 64 if fmt == "fp4_64" else 32
        q = q2d.q2d_quantize(x, mode, seed, offset, block=blk)
        o = oracle.quantize_fp4_2d(x.cpu(), mode, seed, offset, block=blk)
    assert_same_bytes(gpu_buffers(q), o, "operand %s" % fmt)
    return q, o


GEMM_CASES = [
    # (M, N, K, ta, tb, fmt_a, fmt_b) on the small kernel and the persistent kernel
    (300, 200, 160, 0, 0, "fp4_64", "fp4_64"),
    (257, 129, 96, 1, 1, "fp4_64", "fp4"),
    (128, 256, 256, 0, 1, "fp4_1d", "fp4_64"),
    (2100, 4000, 384, 0, 0, "fp4_64", "fp4_64"),
    (4096, 2048, 640, 1, 1, "fp4_64", "fp4_64"),
    (4200, 4100, 256, 1, 0, "fp4", "fp4_64"),
    (2048, 4224, 512, 0, 0, "fp4_1d", "fp4_64"),
]


@pytest.mark.parametrize("M,N,K,ta,tb,fa,fb", GEMM_CASES)
def test_gemm_with_block64_operands(q2d, M, N, K, ta, tb, fa, fb):
    A = synth.normal((K, M) if ta else (M, K), 1.0, M + 3 * K, torch.bfloat16, device=DEV)
    B = synth.normal((K, N) if tb else (N, K), 0.02, N + 5 * K, torch.bfloat16, device=DEV)
    qa, oa = _quant(q2d, A, fa, "rtn")
    qb, ob = _quant(q2d, B, fb, "sr", 7, 1)
    ofa = "fp4_1d" if fa == "fp4_1d" else "fp4"
    ofb = "fp4_1d" if fb == "fp4_1d" else "fp4"
    ref = oracle.gemm(oracle.operand(oa, bool(ta), ofa), oracle.operand(ob, bool(tb), ofb))
    c32 = q2d.q2d_gemm(qa, ta, qb, tb, out_dtype=torch.float32)
    assert rel_frob(c32.cpu().numpy(), ref) <= TOL


@pytest.mark.parametrize("T,N,K", [(192, 320, 256), (4096, 2048, 1024)])
def test_linear_block64(q2d, T, N, K):
    """Y = X W^T, dX = dY W, dW = dY^T X with every operand in 64 x 64 blocks."""
    X = synth.normal((T, K), 1.0, 71, torch.bfloat16, device=DEV)
    W = synth.normal((N, K), 0.02, 72, torch.bfloat16, device=DEV)
    dY = synth.normal((T, N), 1e-3, 73, torch.bfloat16, device=DEV)
    Y, qX, qW = q2d.q2d_linear_fwd(X, W, "rtn", "rtn", 0, 0, 1, torch.float32, block=64)
    dX, dW, qdY = q2d.q2d_linear_bwd(dY, qX, qW, "sr", 0, 2, torch.float32, torch.float32, block=64)
    ox = oracle.quantize_fp4_2d(X.cpu(), "rtn", 0, 0, block=64)
    ow = oracle.quantize_fp4_2d(W.cpu(), "rtn", 0, 1, block=64)
    ody = oracle.quantize_fp4_2d(dY.cpu(), "sr", 0, 2, block=64)
    assert qX.desc.block == qW.desc.block == qdY.desc.block == 64
    for name, gq, oq in (("X", qX, ox), ("W", qW, ow), ("dY", qdY, ody)):
        assert_same_bytes(gpu_buffers(gq), oq, name)
    ref = oracle.linear(ox, ow, ody)
    assert rel_frob(Y.cpu().numpy(), ref["Y"]) <= TOL
    assert rel_frob(dX.cpu().numpy(), ref["dX"]) <= TOL
    assert rel_frob(dW.cpu().numpy(), ref["dW"]) <= TOL
