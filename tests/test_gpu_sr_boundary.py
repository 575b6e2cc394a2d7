"""Stochastic rounding of the GPU quantizers at the exact threshold (App. E:
E[round(x)] = x rests on rounding up iff floor(2^16 d / Delta) + r16 >= 2^16).

Every element of a float32 input sits at F = 2^16 - r16 or 2^16 - r16 - 1 for
its own Philox draw (tests/sr_boundary.py), so the hardware conversion's seed
(r16 << 16 for the first element of a pair, r16 << 15 for the second) is
checked at the one place where it can differ from the contract, on both
nibbles of every byte, even and odd rows and columns, every grid interval
(including the subnormal E2M1 interval [0, 0.5]) and both signs.  Every byte of
the four outputs must equal the oracle's, which the CPU tests pin to the
threshold itself."""
import numpy as np
import pytest
import torch

import oracle
from helpers import assert_same_bytes, gpu_buffers, grouped_written, poison
from sr_boundary import boundary_input, unpack

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


@pytest.fixture(scope="module")
def q2d():
    import paper_2607_24953_amd as q
    return q


@pytest.mark.parametrize("R,C", [(96, 160), (300, 260), (33, 1024)])
@pytest.mark.parametrize("seed,offset", [(0, 0), (0xDEADBEEF12345678, 2 ** 32 + 3)])
def test_2d_threshold(q2d, R, C, seed, offset):
    rng = np.random.default_rng(R * C + (seed & 0xFF))
    x, want = boundary_input(R, C, seed, offset, rng)
    xt = torch.from_numpy(x)
    o = oracle.quantize_fp4_2d(xt, "sr", seed, offset)
    assert np.array_equal(unpack(o["codes"], R, C), want)
    q = q2d.QTensor(q2d.FP4_2D, R, C, DEV)
    poison(q)
    q2d.q2d_quantize(xt.to(DEV), "sr", seed, offset, out=q)
    assert_same_bytes(gpu_buffers(q), o, "sr threshold %dx%d" % (R, C))
    # the transposed view draws the same bits (storage-index keyed)
    ov = oracle.quantize_fp4_2d(xt.t(), "sr", seed, offset)
    qv = q2d.q2d_quantize(xt.to(DEV).t(), "sr", seed, offset)
    assert_same_bytes(gpu_buffers(qv), ov, "transposed view")


def test_2d_threshold_block64(q2d):
    rng = np.random.default_rng(64)
    x, want = boundary_input(192, 320, 5, 9, rng, exps=(4,))
    xt = torch.from_numpy(x)
    o = oracle.quantize_fp4_2d(xt, "sr", 5, 9, block=64)
    assert np.array_equal(unpack(o["codes"], 192, 320), want)
    q = q2d.q2d_quantize(xt.to(DEV), "sr", 5, 9, block=64)
    assert_same_bytes(gpu_buffers(q), o, "block 64")


def test_1d_threshold(q2d):
    rng = np.random.default_rng(1)
    x, want = boundary_input(160, 224, 3, 4, rng)
    xt = torch.from_numpy(x)
    o = oracle.quantize_fp4_1d(xt, "sr", 3, 4)
    assert np.array_equal(unpack(o["codes"], 160, 224), want)
    q = q2d.q2d_quantize_1d(xt.to(DEV), "sr", 3, 4)
    assert_same_bytes(gpu_buffers(q), o, "1d")


def test_grouped_threshold(q2d):
    rng = np.random.default_rng(2)
    x, want = boundary_input(352, 128, 8, 1, rng)
    offs = [0, 64, 64, 160, 352]                 # 32-aligned segments (one empty)
    xt = torch.from_numpy(x)
    o = oracle.quantize_fp4_grouped(xt, offs, "sr", 8, 1)
    q = q2d.q2d_grouped_quantize(xt.to(DEV), torch.tensor(offs, dtype=torch.int64, device=DEV), "sr", 8, 1)
    want = {k: o[k] for k in ("codes", "codes_t", "scales", "scales_t")}
    assert_same_bytes(grouped_written(q, int(o["padded_rows"][-1])), want, "grouped")
