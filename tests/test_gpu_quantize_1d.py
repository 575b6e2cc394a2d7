"""GPU parity of the 1D FP4 activation path (Sec. 3, "Application to linear
layers"; App. C, "Activations") against the oracle.

Quantization: every byte of both copies (1x32 rowwise codes and scales, 32x1
colwise codes and scales) equal to the oracle's, for ragged shapes, both
dtypes, both rounding modes, transposed and strided views, non-finite and zero
blocks, every finite bfloat16 value under every block exponent it can meet,
float32 midpoints and subnormals, and the 7B-class activation at full size.

GEMMs: 1D operands mixed with 2D ones (forward: A = X rowwise; weight
gradient: B = X colwise) on the small-problem and the persistent kernel, and
the linear layer with 1D activations, against the float64 oracle GEMM
(relative Frobenius error <= 1e-5 for float32 output).
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from helpers import assert_same_bytes, check_bf16, gpu_buffers, poison, rel_frob

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
TOL = 1e-5


@pytest.fixture(scope="module")
def q2d():
    import paper_2607_24953_amd as q
    return q


def run_case(q2d, x_dev, mode, seed=0, offset=0, label="", x_cpu=None):
    q = q2d.QTensor(q2d.FP4_1D, x_dev.shape[0], x_dev.shape[1], x_dev.device)
    poison(q)
    q2d.q2d_quantize_1d(x_dev, mode, seed, offset, out=q)
    got = gpu_buffers(q)
    if x_cpu is None:
        assert x_dev.is_contiguous()
        x_cpu = x_dev.cpu()
    assert x_cpu.stride() == x_dev.stride()
    want = oracle.quantize_fp4_1d(x_cpu, mode, seed, offset)
    assert_same_bytes(got, want, label)


SHAPES = [(128, 256), (100, 70), (33, 129), (1, 5), (257, 31), (300, 1000), (129, 4097)]


@pytest.mark.parametrize("shape", SHAPES)
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("mode", ["rtn", "sr"])
def test_quantize_1d(q2d, shape, dtype, mode):
    x = synth.normal(shape, 1.5, shape[0] * 7 + shape[1], dtype, device=DEV)
    run_case(q2d, x, mode, 3, 11, "%s %s %s" % (shape, dtype, mode))


@pytest.mark.parametrize("mode", ["rtn", "sr"])
def test_quantize_1d_views(q2d, mode):
    base = synth.normal((200, 300), 1.0, 41, torch.bfloat16)
    bd = base.to(DEV)
    run_case(q2d, bd.t(), mode, 4, 5, "transposed view", x_cpu=base.t())
    run_case(q2d, bd[:, ::2], mode, 4, 5, "column-strided view", x_cpu=base[:, ::2])
    run_case(q2d, bd[10:150, 7:290], mode, 4, 5, "offset view", x_cpu=base[10:150, 7:290])


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_special_values_1d(q2d, dtype):
    x = synth.normal((96, 160), 1.0, 42, torch.float32)
    x[3, 40] = float("nan")
    x[50, 7] = float("inf")
    x[70, 100] = -float("inf")
    x[64:96, 128:160] = 0.0
    x[0:32, 0:32] = 1e-30
    xd = x.to(dtype).to(DEV)
    for mode in ("rtn", "sr"):
        run_case(q2d, xd, mode, 1, 2, "special %s" % mode)


def _every_value_rows(exponents):
    """Rows of 32: 31 finite bfloat16 values with |x| <= 6 * 2^e and a 6 * 2^e entry
    (so the 1x32 block scale is exactly 2^e); per exponent the rows list every
    such value once, with both signs."""
    pos = (np.arange(0x7F80, dtype=np.uint32) << 16).view(np.float32)
    rows = []
    for e in exponents:
        top = np.float32(6.0 * 2.0 ** e)
        vals = pos[pos <= top]
        vals = np.concatenate([vals, -vals])
        n = -(-len(vals) // 31)
        blk = np.zeros((n, 32), dtype=np.float32)
        flat = np.zeros(n * 31, dtype=np.float32)
        flat[:len(vals)] = vals
        blk[:, :31] = flat.reshape(n, 31)
        blk[:, 31] = top
        rows.append(blk)
    return torch.from_numpy(np.concatenate(rows, axis=0)).to(torch.bfloat16)


@pytest.mark.parametrize("exps", [list(range(-24, 25)), [-127, -126, -125, -100, -60, 60, 100, 124, 125]])
def test_every_value_under_every_scale_1d(q2d, exps):
    x = _every_value_rows(exps)                  # rowwise blocks: the rows above
    xt = x.t().contiguous()                      # colwise blocks: the same values down columns
    for mode in ("rtn", "sr"):
        run_case(q2d, x.to(DEV), mode, 5, 6, "every value rowwise %s" % mode)
        run_case(q2d, xt.to(DEV), mode, 5, 6, "every value colwise %s" % mode)
    run_case(q2d, x.float().to(DEV), "rtn", 0, 0, "every value fp32 rtn")


def test_fp32_midpoints_and_subnormals_1d(q2d):
    mids = np.array([0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0], np.float32)
    cand = np.concatenate([mids, np.nextafter(mids, np.float32(0)), np.nextafter(mids, np.float32(9))])
    rows = []
    for e in (-130, -127, -126, -20, -1, 0, 1, 7, 50, 120):
        scale = np.float32(2.0 ** e)
        for sgn in (1, -1):
            r = np.zeros(64, np.float32)
            r[:len(cand)] = sgn * cand * scale
            r[31] = np.float32(6.0) * scale
            r[63] = np.float32(6.0) * scale
            rows.append(r)
    sub = (np.arange(1, 65, dtype=np.uint32) * 7919).view(np.float32)
    rows.append(sub)
    rows.append(-sub)
    x = torch.from_numpy(np.stack(rows))
    for mode in ("rtn", "sr"):
        run_case(q2d, x.to(DEV), mode, 9, 1, "fp32 midpoints rowwise %s" % mode)
        run_case(q2d, x.t().contiguous().to(DEV), mode, 9, 1, "fp32 midpoints colwise %s" % mode)


def test_full_size_7b_activation(q2d):
    """The 7B-class QKV input (16384 x 4096 bf16, 1 % outlier channels), all bytes."""
    x = synth.add_outlier_channels(synth.normal((16384, 4096), 1.0, 3001, torch.bfloat16), 3002)
    run_case(q2d, x.to(DEV), "rtn", 0, 0, "7B X 1D")


# ------------------------------------------------------------------ GEMMs

def _quant(q2d, x, fmt, mode, seed=0, offset=0):
    if fmt == "fp4_1d":
        q = q2d.q2d_quantize_1d(x, mode, seed, offset)
        o = oracle.quantize_fp4_1d(x.cpu(), mode, seed, offset)
    else:
        q = q2d.q2d_quantize(x, mode, seed, offset)
        o = oracle.quantize_fp4_2d(x.cpu(), mode, seed, offset)
    assert_same_bytes(gpu_buffers(q), o, "operand %s" % fmt)
    return q, o


GEMM_CASES = [
    # (M, N, K, ta, tb, fmt_a, fmt_b): forward (A = X rowwise 1D), weight gradient
    # (B = X colwise 1D), both 1D, on the small kernel and the persistent kernel
    (300, 200, 160, 0, 0, "fp4_1d", "fp4"),
    (257, 129, 96, 1, 1, "fp4", "fp4_1d"),
    (128, 256, 256, 0, 0, "fp4_1d", "fp4_1d"),
    (2100, 4000, 384, 0, 0, "fp4_1d", "fp4"),
    (4096, 2048, 640, 1, 1, "fp4", "fp4_1d"),
    (4200, 4100, 256, 0, 1, "fp4_1d", "fp4"),
    (2048, 4224, 512, 0, 0, "fp4_1d", "fp4_1d"),
]


@pytest.mark.parametrize("M,N,K,ta,tb,fa,fb", GEMM_CASES)
def test_gemm_with_1d_operands(q2d, M, N, K, ta, tb, fa, fb):
    A = synth.normal((K, M) if ta else (M, K), 1.0, M + 3 * K, torch.bfloat16, device=DEV)
    B = synth.normal((K, N) if tb else (N, K), 0.02, N + 5 * K, torch.bfloat16, device=DEV)
    qa, oa = _quant(q2d, A, fa, "rtn")
    qb, ob = _quant(q2d, B, fb, "sr", 7, 1)
    ref = oracle.gemm(oracle.operand(oa, bool(ta), fa), oracle.operand(ob, bool(tb), fb))
    c32 = q2d.q2d_gemm(qa, ta, qb, tb, out_dtype=torch.float32)
    assert rel_frob(c32.cpu().numpy(), ref) <= TOL
    # bf16 output: on the persistent kernel, interleaved output columns (a 1D B
    # operand's row words follow its permuted rows)
    check_bf16(q2d.q2d_gemm(qa, ta, qb, tb, out_dtype=torch.bfloat16), ref)


@pytest.mark.parametrize("T,N,K", [(256, 384, 512), (4096, 2048, 1024)])
def test_linear_with_1d_activations(q2d, T, N, K):
    """Y = X W^T, dX = dY W, dW = dY^T X with X in 1D blocks (rowwise copy forward,
    colwise copy for dW), W and dY in 2D blocks (App. C)."""
    X = synth.normal((T, K), 1.0, 51, torch.bfloat16, device=DEV)
    W = synth.normal((N, K), 0.02, 52, torch.bfloat16, device=DEV)
    dY = synth.normal((T, N), 1e-3, 53, torch.bfloat16, device=DEV)
    Y, qX, qW = q2d.q2d_linear_fwd(X, W, "rtn", "rtn", 0, 0, 1, torch.float32, fmt_x=q2d.FP4_1D)
    dX, dW, qdY = q2d.q2d_linear_bwd(dY, qX, qW, "sr", 0, 2, torch.float32, torch.float32)
    ox = oracle.quantize_fp4_1d(X.cpu(), "rtn", 0, 0)
    ow = oracle.quantize_fp4_2d(W.cpu(), "rtn", 0, 1)
    ody = oracle.quantize_fp4_2d(dY.cpu(), "sr", 0, 2)
    assert_same_bytes(gpu_buffers(qX), ox, "qX")
    assert_same_bytes(gpu_buffers(qdY), ody, "qdY")
    ref = oracle.linear(ox, ow, ody, fmt_x="fp4_1d")
    assert rel_frob(Y.cpu().numpy(), ref["Y"]) <= TOL
    assert rel_frob(dX.cpu().numpy(), ref["dX"]) <= TOL
    assert rel_frob(dW.cpu().numpy(), ref["dW"]) <= TOL
