"""GPU parity of the floor scale rule (the rule that the truncation-free
ablation goes back to: Sec. 4.2, the ablation figure; App. G) against the
oracle: every byte of the four buffers for round to nearest and stochastic
rounding, bf16 and fp32, ragged shapes, 32x32 and 64x64 blocks, views, the
grouped form, every bf16 value under extreme and ordinary block exponents
(with the saturating maximum), and a GEMM on floor-rule operands.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from helpers import assert_same_bytes, gpu_buffers, poison, rel_frob

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


@pytest.fixture(scope="module")
def q2d():
    import paper_2607_24953_amd as q
    return q


def run_case(q2d, x_dev, mode, seed=0, offset=0, block=32, label="", x_cpu=None):
    q = q2d.QTensor(q2d.FP4_2D, x_dev.shape[0], x_dev.shape[1], x_dev.device, block)
    poison(q)
    q2d.q2d_quantize(x_dev, mode, seed, offset, out=q, block=block)
    got = gpu_buffers(q)
    if x_cpu is None:
        x_cpu = x_dev.cpu()
    want = oracle.quantize_fp4_2d(x_cpu, mode, seed, offset, block=block)
    assert_same_bytes(got, want, label)
    return q, want


SHAPES = [(128, 256), (100, 70), (33, 129), (257, 31), (300, 1000)]


@pytest.mark.parametrize("shape", SHAPES)
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("mode", ["rtn-floor", "sr-floor"])
@pytest.mark.parametrize("block", [32, 64])
def test_floor_rule_quantize(q2d, shape, dtype, mode, block):
    x = synth.normal(shape, 1.0, 700 + shape[1], dtype, device=DEV)
    synth.add_outlier_channels(x, 10, frac=0.03)
    run_case(q2d, x, mode, 6, 2, block, "%s %s %s b%d" % (shape, dtype, mode, block))


@pytest.mark.parametrize("mode", ["rtn-floor", "sr-floor"])
def test_floor_rule_views(q2d, mode):
    base = synth.normal((200, 300), 1.0, 71, torch.bfloat16)
    bd = base.to(DEV)
    run_case(q2d, bd.t(), mode, 1, 1, label="transposed view", x_cpu=base.t())
    run_case(q2d, bd[:, ::2], mode, 1, 1, label="column-strided view", x_cpu=base[:, ::2])


def _every_value_matrix(exponents):
    """32-row blocks of every finite bf16 value below 8 * 2^e (both signs), so every
    block's floor exponent is e and the values in (6 * 2^e, 8 * 2^e) saturate."""
    pos = (np.arange(0x7F80, dtype=np.uint32) << 16).view(np.float32)
    cols = []
    for e in exponents:
        top = np.float32(2.0 ** (e + 2) * 1.9921875)     # largest bf16 below 8 * 2^e
        vals = pos[pos <= top]
        vals = np.concatenate([vals, -vals])
        n = -(-len(vals) // (32 * 32)) * 32
        flat = np.zeros(32 * n, dtype=np.float32)
        flat[:len(vals)] = vals
        blk = flat.reshape(32, n)
        blk[0, ::32] = top
        cols.append(blk)
    return torch.from_numpy(np.concatenate(cols, axis=1)).to(torch.bfloat16)


@pytest.mark.parametrize("exps", [list(range(-12, 13)), [-127, -126, -125, -100, 60, 100, 124, 125]])
def test_floor_rule_every_value(q2d, exps):
    x = _every_value_matrix(exps)
    for mode in ("rtn-floor", "sr-floor"):
        run_case(q2d, x.to(DEV), mode, 3, 9, label="every value %s" % mode)
        run_case(q2d, x.t().contiguous().to(DEV), mode, 3, 9, label="every value transposed %s" % mode)
    run_case(q2d, x.float().to(DEV), "rtn-floor", label="every value fp32")


@pytest.mark.parametrize("mode", ["rtn-floor", "sr-floor"])
def test_floor_rule_grouped(q2d, mode):
    off = synth.segment_offsets([0, 1, 31, 33, 127, 130, 256])
    S = int(off[-1])
    x = synth.normal((S, 160), 1.0, 72, torch.bfloat16, device=DEV)
    synth.add_outlier_channels(x, 11, frac=0.05)
    q = q2d.q2d_grouped_quantize(x, torch.tensor(off, device=DEV), mode, 5, 3)
    torch.cuda.synchronize()
    o = oracle.quantize_fp4_grouped(x.cpu(), off, mode, 5, 3)
    P = int(o["padded_rows"][-1])
    got = {"codes": q.codes[:P].cpu().numpy(), "scales": q.scales[:P // 32].cpu().numpy(),
           "codes_t": q.codes_t[:, :P // 2].cpu().numpy(), "scales_t": q.scales_t[:, :P // 32].cpu().numpy()}
    assert_same_bytes(got, o, "grouped %s" % mode)


def test_floor_rule_gemm_and_1d_rejected(q2d):
    A = synth.normal((2100, 384), 1.0, 73, torch.bfloat16, device=DEV)
    B = synth.normal((4000, 384), 0.02, 74, torch.bfloat16, device=DEV)
    qa, oa = run_case(q2d, A, "rtn-floor")
    qb, ob = run_case(q2d, B, "sr-floor", 2, 2)
    c = q2d.q2d_gemm(qa, 0, qb, 0, out_dtype=torch.float32)
    ref = oracle.gemm(oracle.operand(oa, False), oracle.operand(ob, False))
    assert rel_frob(c.cpu().numpy(), ref) <= 1e-5
    with pytest.raises(q2d.Q2DError):
        q2d.q2d_quantize_1d(A, "rtn-floor")
