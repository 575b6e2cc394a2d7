"""GPU parity of the MXFP8 quantizer (query/key path, Sec. 3.2) against the oracle.

Every byte of the rowwise (1 x 32) and colwise (32 x 1, stored transposed)
copies and their E8M0 scales equals ``oracle.quantize_mxfp8``: ragged shapes,
bf16 and fp32 inputs, strided and transposed views, special values (zeros,
signed zeros, NaN, infinities, subnormals, the top of the range), and every
finite bfloat16 value under each block exponent it can meet (E4M3
round-to-nearest-even exhaustively).
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from helpers import assert_same_bytes, gpu_buffers, poison

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


@pytest.fixture(scope="module")
def q2d():
    import paper_2607_24953_amd as q
    return q


def run_case(q2d, x_dev, label, x_cpu=None):
    q = q2d.QTensor(q2d.MXFP8, x_dev.shape[0], x_dev.shape[1], x_dev.device)
    poison(q)
    q2d.mxfp8_quantize(x_dev, out=q)
    got = gpu_buffers(q)
    if x_cpu is None:
        assert x_dev.is_contiguous()
        x_cpu = x_dev.cpu()
    want = oracle.quantize_mxfp8(x_cpu)
    assert_same_bytes(got, want, label)


@pytest.mark.parametrize("shape", [(128, 256), (100, 70), (33, 129), (1, 5), (257, 31), (640, 384),
                                   (129, 4097), (1000, 4096)])
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_mxfp8_shapes(q2d, shape, dtype):
    x = synth.normal(shape, 1.0, shape[0] * 7 + shape[1], dtype, device=DEV)
    synth.add_outlier_channels(x, 4, frac=0.02)
    run_case(q2d, x, "mxfp8 %s %s" % (shape, dtype))


def test_mxfp8_views(q2d):
    base = synth.normal((300, 520), 1.0, 3, torch.bfloat16, device=DEV)
    base_cpu = base.cpu()
    run_case(q2d, base[:, 8:264], "row-strided", x_cpu=base_cpu[:, 8:264])
    run_case(q2d, base.t(), "transposed", x_cpu=base_cpu.t())
    run_case(q2d, base[::2, ::3], "strided", x_cpu=base_cpu[::2, ::3])


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_mxfp8_special_values(q2d, dtype):
    x = synth.normal((160, 200), 1.0, 13, torch.float32)
    x[0:32, 0:32] = 0.0
    x[32:64, 0:32] = -0.0
    x[3, 40] = float("nan")
    x[40, 70] = float("inf")
    x[70, 100] = -float("inf")
    x[100:132, 0:32] *= 1e-40
    x[100:132, 32:64] *= 1e36
    x[140, 140] = 3.0e38
    x[150, 190] = 1e-30
    run_case(q2d, x.to(dtype).to(DEV), "mxfp8 special %s" % dtype)


def _every_value_matrix(exponents):
    """Strips of 32 rows, one per exponent e: every row holds 31 finite bfloat16
    values with |x| <= 448 * 2^e and the value 448 * 2^e itself (so every 1 x 32
    row block has scale exactly 2^e); together the rows list every such value
    with both signs."""
    pos = (np.arange(0x7F80, dtype=np.uint32) << 16).view(np.float32)
    strips = []
    for e in exponents:
        top = np.float32(448.0 * 2.0 ** e)
        vals = pos[pos <= top]
        vals = np.concatenate([vals, -vals])
        nrow = -(-len(vals) // 31)
        nrow = -(-nrow // 32) * 32
        rows = np.zeros((nrow, 32), dtype=np.float32)
        flat = rows[:, :31].reshape(-1)
        flat[:len(vals)] = vals
        rows[:, :31] = flat.reshape(nrow, 31)
        rows[:, 31] = top
        # 32 rows per band, bands side by side
        strips.append(rows.reshape(nrow // 32, 32, 32).transpose(1, 0, 2).reshape(32, -1))
    width = max(s_.shape[1] for s_ in strips)
    out = np.zeros((32 * len(strips), width), dtype=np.float32)
    for k, s_ in enumerate(strips):
        out[32 * k:32 * (k + 1), :s_.shape[1]] = s_
    return torch.from_numpy(out).to(torch.bfloat16)


@pytest.mark.parametrize("exps", [list(range(-20, 21)), [-127, -126, -125, -100, 100, 118, 119]])
def test_mxfp8_every_value_under_every_scale(q2d, exps):
    x = _every_value_matrix(exps)
    run_case(q2d, x.to(DEV), "mxfp8 every value bf16")
    run_case(q2d, x.float().to(DEV), "mxfp8 every value fp32")
    run_case(q2d, x.t().contiguous().to(DEV), "mxfp8 every value, columns")
