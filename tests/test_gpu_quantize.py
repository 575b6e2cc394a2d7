"""GPU parity of the fused 2D-block FP4 quantizer against the CPU oracle.

Bit-exact on every byte of the four output buffers (codes, codes_t, scales,
scales_t, padding included; buffers are poisoned before each call), for round to
nearest and stochastic rounding, float32 and bfloat16 inputs, ragged shapes that
span several 128 x 128 tiles, views (transposed, sliced, strided, misaligned),
special values, and the full-size tensors of the 1B and 7B linear workloads.
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


def run_case(q2d, x_dev, mode, seed=0, offset=0, label="", x_cpu=None):
    """x_cpu: the same view taken on a host copy of the base tensor, so that the
    storage strides (and hence the random-stream indices) match the device view."""
    q = q2d.QTensor(q2d.FP4_2D, x_dev.shape[0], x_dev.shape[1], x_dev.device)
    poison(q)
    q2d.q2d_quantize(x_dev, mode, seed, offset, out=q)
    got = gpu_buffers(q)
    if x_cpu is None:
        assert x_dev.is_contiguous()
        x_cpu = x_dev.cpu()
    assert x_cpu.stride() == x_dev.stride()
    want = oracle.quantize_fp4_2d(x_cpu, mode, seed, offset)
    assert_same_bytes(got, want, label)


SHAPES = [(128, 256), (256, 256), (100, 70), (33, 129), (1, 5), (257, 31), (300, 1000),
          (640, 384), (129, 4097)]


@pytest.mark.parametrize("shape", SHAPES)
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("mode", ["rtn", "sr"])
def test_quantize_shapes(q2d, shape, dtype, mode):
    x = synth.normal(shape, 1.0, 100 + shape[0], dtype, device=DEV)
    synth.add_outlier_channels(x, 7, frac=0.02)
    run_case(q2d, x, mode, seed=1234, offset=shape[1], label="%s %s %s" % (shape, dtype, mode))


@pytest.mark.parametrize("seed,offset", [(0, 0), (2**32 - 1, 2**32 + 5), (2**63 + 11, 2**40)])
def test_quantize_seed_offset(q2d, seed, offset):
    x = synth.normal((192, 320), 0.02, 5, torch.bfloat16, device=DEV)
    run_case(q2d, x, "sr", seed, offset)


@pytest.mark.parametrize("mode", ["rtn", "sr"])
def test_quantize_views(q2d, mode):
    base = synth.normal((300, 520), 1.0, 9, torch.bfloat16, device=DEV)
    hb = base.cpu()
    views = [("transposed view", lambda t: t.t()),
             ("column slice (row stride 520)", lambda t: t[:, :400]),
             ("offset slice", lambda t: t[5:200, 8:300]),
             ("strided both", lambda t: t[::2, ::3]),
             ("transposed slice", lambda t: t[3:250, 16:400].t())]
    for label, fn in views:
        run_case(q2d, fn(base), mode, 3, 4, label, x_cpu=fn(hb))
    odd = synth.normal((77, 100), 1.0, 10, torch.bfloat16, device=DEV)   # 200-byte rows
    run_case(q2d, odd, mode, 3, 4, "unaligned rows")
    f = synth.normal((70, 90), 1.0, 11, torch.float32, device=DEV)
    run_case(q2d, f.t(), mode, 3, 4, "fp32 transposed", x_cpu=f.cpu().t())


def test_transposed_view_equals_swapped_layouts(q2d):
    w = synth.normal((384, 256), 0.02, 12, torch.bfloat16, device=DEV)
    a = gpu_buffers(q2d.q2d_quantize(w, "sr", 8, 9))
    b = gpu_buffers(q2d.q2d_quantize(w.t(), "sr", 8, 9))
    assert np.array_equal(a["codes"], b["codes_t"]) and np.array_equal(a["codes_t"], b["codes"])
    assert np.array_equal(a["scales"], b["scales_t"]) and np.array_equal(a["scales_t"], b["scales"])


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_special_values(q2d, dtype):
    x = synth.normal((160, 200), 1.0, 13, torch.float32)
    x[0:32, 0:32] = 0.0                       # zero block
    x[32:64, 0:32] = -0.0                     # negative zeros keep their sign bit
    x[3, 40] = float("nan")
    x[40, 70] = float("inf")
    x[70, 100] = -float("inf")
    x[100:132, 0:32] *= 1e-40                 # float32 subnormals
    x[100:132, 32:64] *= 1e36                 # near the top of the range
    x[140, 140] = 3.0e38
    x[64:96, 64:96] = torch.tensor(6.0) * torch.sign(x[64:96, 64:96])   # v = 6 exactly
    x[150, 190] = 1e-30                        # lone tiny value in an otherwise normal block
    xd = x.to(dtype).to(DEV)
    for mode in ("rtn", "sr"):
        run_case(q2d, xd, mode, 1, 2, "special %s" % mode)


def test_exhaustive_bf16_values(q2d):
    """Every finite bfloat16 bit pattern, placed so that blocks span all exponents."""
    bits = torch.arange(0, 1 << 16, dtype=torch.int32).to(torch.int16)
    x = bits.view(torch.bfloat16).reshape(256, 256).clone()
    x[torch.isnan(x) | torch.isinf(x)] = 0
    xd = x.to(DEV)
    for mode in ("rtn", "sr"):
        run_case(q2d, xd, mode, 77, 1, "all bf16 %s" % mode)
        run_case(q2d, xd.t(), mode, 77, 1, "all bf16 transposed %s" % mode, x_cpu=x.t())


def _every_value_matrix(exponents):
    """32-row strips, one per exponent e: 32 x 32 blocks that each hold a 6 * 2^e
    entry (so the block scale is exactly 2^e) and 1023 other finite bfloat16
    values with |x| <= 6 * 2^e; together they list every such value once,
    with both signs."""
    pos = (np.arange(0x7F80, dtype=np.uint32) << 16).view(np.float32)
    strips = []
    for e in exponents:
        top = np.float32(6.0 * 2.0 ** e)
        vals = pos[pos <= top]
        vals = np.concatenate([vals, -vals])
        nb = -(-len(vals) // 1023)
        blocks = np.zeros((nb, 1024), dtype=np.float32)
        flat = blocks.reshape(-1)
        for b in range(nb):
            chunk = vals[b * 1023:(b + 1) * 1023]
            blocks[b, :len(chunk)] = chunk
            blocks[b, 1023] = top
        strips.append(blocks.reshape(nb, 32, 32).transpose(1, 0, 2).reshape(32, nb * 32))
    width = max(s_.shape[1] for s_ in strips)
    out = np.zeros((32 * len(strips), width), dtype=np.float32)
    for k, s_ in enumerate(strips):
        out[32 * k:32 * (k + 1), :s_.shape[1]] = s_
    return torch.from_numpy(out).to(torch.bfloat16)


@pytest.mark.parametrize("exps", [list(range(-24, 25)), [-127, -126, -125, -100, -60, 60, 100, 124, 125]])
def test_every_value_under_every_scale(q2d, exps):
    """Round to nearest (and SR) of every finite bfloat16 value under each exponent it can meet."""
    x = _every_value_matrix(exps)
    xd = x.to(DEV)
    for mode in ("rtn", "sr"):
        run_case(q2d, xd, mode, 5, 6, "every value %s" % mode)
    run_case(q2d, xd.float(), "rtn", 0, 0, "every value fp32 rtn")


def test_fp32_midpoints_and_subnormals(q2d):
    """float32 inputs at E2M1 midpoints +- 1 ulp and float32 subnormals, per block scale."""
    mids = np.array([0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0], np.float32)
    cand = np.concatenate([mids, np.nextafter(mids, np.float32(0)), np.nextafter(mids, np.float32(9))])
    rows = []
    for e in (-130, -127, -126, -20, -1, 0, 1, 7, 50, 120):
        scale = np.float32(2.0 ** e) if e > -150 else np.float32(0)
        blk = np.zeros(1024, np.float32)
        blk[:len(cand)] = cand * scale
        blk[len(cand):2 * len(cand)] = -cand * scale
        blk[1023] = np.float32(6.0) * scale
        rows.append(blk.reshape(32, 32))
    sub = np.zeros(1024, np.float32)
    sub[:512] = (np.arange(1, 513, dtype=np.uint32) * 7919).view(np.float32)     # subnormals
    sub[512:1023] = -sub[:511]
    rows.append(sub.reshape(32, 32))
    x = torch.from_numpy(np.concatenate(rows, axis=1))
    for mode in ("rtn", "sr"):
        run_case(q2d, x.to(DEV), mode, 9, 1, "fp32 midpoints %s" % mode)


def test_deterministic(q2d):
    x = synth.normal((512, 768), 1.0, 15, torch.bfloat16, device=DEV)
    a = gpu_buffers(q2d.q2d_quantize(x, "sr", 5, 6))
    b = gpu_buffers(q2d.q2d_quantize(x, "sr", 5, 6))
    for k in a:
        assert np.array_equal(a[k], b[k])


@pytest.mark.parametrize("name", ["dense_1b", "dense_7b"])
def test_full_size_workloads(q2d, name):
    """Every quantized tensor of the workload at full size, all bytes compared."""
    w = synth.WORKLOADS[name](device=DEV)
    for k, x in w.tensors.items():
        mode = w.rounding[k]
        print("quantize %s %s %s %s" % (name, k, tuple(x.shape), mode), flush=True)
        q = q2d.q2d_quantize(x, mode, w.seed, 17)
        got = gpu_buffers(q)
        want = oracle.quantize_fp4_2d(x.cpu(), mode, w.seed, 17)
        assert_same_bytes(got, want, "%s %s" % (name, k))
        del q, got, want
    del w
    torch.cuda.empty_cache()
