"""Pins of the oracle's 1D FP4 quantizer (activations; Sec. 3 "Application to
linear layers"; App. C "Activations").

* Special cases that reduce it to the pinned 2D-block quantizer: when the 32
  rows of every 32 x 32 block are equal, each 1 x 32 row block has the 2D
  block's maximum, so the rowwise copy equals the 2D codes and scales; the
  same for columns and the colwise copy.
* The colwise copy of X is the rowwise copy of X^T (a transposed view draws
  the same stochastic bits, a materialised copy gives the same nearest codes).
* A hand-derived block (scale and round-to-nearest ties worked out by hand).
* The forward/backward inconsistency of 1D layouts that the 2D blocks remove
  (Sec. 2, "Scale inconsistency under transposition"): the two 1D copies of a
  matrix with an outlier dequantize to different values; the two 2D copies
  never do.
* Element-wise definition against block maxima computed with numpy, and the
  round-to-nearest error bound (Sec. 3.1).
"""
import numpy as np
import pytest
import torch

import oracle
import synth

B = 32


def _unpack(packed, n):
    u = np.empty((packed.shape[0], packed.shape[1] * 2), dtype=np.uint8)
    u[:, 0::2] = packed & 15
    u[:, 1::2] = packed >> 4
    return u[:, :n]


@pytest.mark.parametrize("shape", [(96, 160), (70, 100), (33, 65)])
@pytest.mark.parametrize("mode", ["rtn", "sr"])
def test_rowwise_reduces_to_2d_on_row_replicated_blocks(shape, mode):
    R, C = shape
    base = synth.normal((-(-R // B), C), 1.3, 21, torch.bfloat16)
    x = base[torch.arange(R) // B].contiguous()          # the 32 rows of each block are equal
    q1 = oracle.quantize_fp4_1d(x, mode, seed=3, offset=4)
    q2 = oracle.quantize_fp4_2d(x, mode, seed=3, offset=4)
    np.testing.assert_array_equal(q1["codes"], q2["codes"])
    np.testing.assert_array_equal(oracle.scale_grid_1d(q1["scales"], R), q2["scales"][np.arange(R) // B])


@pytest.mark.parametrize("shape", [(96, 160), (70, 100), (65, 33)])
@pytest.mark.parametrize("mode", ["rtn", "sr"])
def test_colwise_reduces_to_2d_on_column_replicated_blocks(shape, mode):
    R, C = shape
    base = synth.normal((R, -(-C // B)), 0.9, 22, torch.bfloat16)
    x = base[:, torch.arange(C) // B].contiguous()       # the 32 columns of each block are equal
    q1 = oracle.quantize_fp4_1d(x, mode, seed=8, offset=1)
    q2 = oracle.quantize_fp4_2d(x, mode, seed=8, offset=1)
    np.testing.assert_array_equal(q1["codes_t"], q2["codes_t"])
    np.testing.assert_array_equal(oracle.scale_grid_1d(q1["scales_t"], C), q2["scales_t"][np.arange(C) // B])


@pytest.mark.parametrize("mode", ["rtn", "sr"])
def test_colwise_is_rowwise_of_transposed_view(mode):
    x = synth.normal((100, 70), 1.0, 23, torch.bfloat16)
    q = oracle.quantize_fp4_1d(x, mode, seed=9, offset=2)
    qt = oracle.quantize_fp4_1d(x.t(), mode, seed=9, offset=2)   # view: same storage indices
    for a, b in (("codes", "codes_t"), ("scales", "scales_t"), ("codes_t", "codes"), ("scales_t", "scales")):
        np.testing.assert_array_equal(qt[a], q[b])


def test_materialised_transpose_rtn():
    x = synth.normal((90, 130), 1.0, 24, torch.float32)
    q = oracle.quantize_fp4_1d(x, "rtn")
    qt = oracle.quantize_fp4_1d(x.t().contiguous(), "rtn")
    np.testing.assert_array_equal(qt["codes"], q["codes_t"])
    np.testing.assert_array_equal(qt["scales"], q["scales_t"])


def test_hand_derived_block():
    # row block [7, 0.75, -2.5, 1.25, 0, ...]: M = 7; 6 * 2^0 < 7 <= 6 * 2^1, so e = 1
    # (byte 128).  x / 2 = 3.5 -> tie of 3 (index 5) and 4 (index 6): even index 6;
    # 0.375 -> above the 0.25 midpoint: 0.5 (index 1); -1.25 -> tie of 1 (2) and
    # 1.5 (3): even index 2, negative: 8 | 2; 0.625 -> below the 0.75 midpoint: 0.5.
    # Column 0 holds 7 and zeros: its 32 x 1 block has the same scale and code.
    x = np.zeros((32, 32), dtype=np.float32)
    x[0, :4] = [7.0, 0.75, -2.5, 1.25]
    q = oracle.quantize_fp4_1d(x, "rtn")
    sg, sgt = oracle.scale_grid_1d(q["scales"], 32), oracle.scale_grid_1d(q["scales_t"], 32)
    assert sg[0, 0] == 128 and q["scales"][0, 0] == 128    # byte 0 of word (0, row 0)
    assert list(_unpack(q["codes"], 32)[0, :5]) == [6, 1, 10, 1, 0]
    assert sg[1, 0] == 0                                   # all-zero row block: byte 0x00
    assert sgt[0, 0] == 128 and _unpack(q["codes_t"], 32)[0, 0] == 6
    # column 1 is 0.75 alone: 6 * 2^-3 < 0.75 <= 6 * 2^-2, e = -3, 0.75 / 2^-3 = 6 (index 7)
    assert sgt[1, 0] == 124 and q["scales_t"][0, 4] == 124 and _unpack(q["codes_t"], 32)[1, 0] == 7


def test_forward_backward_inconsistency_of_1d_blocks():
    x = synth.normal((64, 64), 1.0, 25, torch.float32)
    x[5, 7] = 200.0                                        # an outlier
    q1 = oracle.quantize_fp4_1d(x, "rtn")
    fwd = oracle.operand(q1, False, "fp4_1d")               # the forward GEMM's copy
    bwd = oracle.operand(q1, True, "fp4_1d").T              # the weight-gradient GEMM's copy
    differ = fwd != bwd
    assert differ.sum() > 0
    # the outlier's row block flushes its neighbours in the forward copy only
    assert np.count_nonzero(fwd[5, :32]) < np.count_nonzero(bwd[5, :32])
    q2 = oracle.quantize_fp4_2d(x, "rtn")
    np.testing.assert_array_equal(oracle.operand(q2, False), oracle.operand(q2, True).T)


@pytest.mark.parametrize("shape", [(70, 100), (1, 33), (129, 1)])
@pytest.mark.parametrize("mode", ["rtn", "sr"])
def test_elementwise_definition(shape, mode):
    R, C = shape
    x = synth.normal(shape, 0.6, 26, torch.bfloat16)
    q = oracle.quantize_fp4_1d(x, mode, seed=2, offset=6)
    x64 = oracle.to_float64(x)
    idx = np.arange(R)[:, None] * x.stride(0) + np.arange(C)[None, :]
    r16 = np.vectorize(lambda i: oracle.sr_bits(int(i), 2, 6))(idx).astype(np.uint32) if mode == "sr" else None
    # rowwise: block maxima along columns
    nbc = -(-C // B)
    rmax = np.stack([np.abs(x64[:, j * B:(j + 1) * B]).max(axis=1) for j in range(nbc)], axis=1)
    er = np.vectorize(oracle.fp4_scale_exponent)(rmax).astype(np.int64)
    sg = oracle.scale_grid_1d(q["scales"], R)
    np.testing.assert_array_equal(sg[:, :nbc], (er + 127).astype(np.uint8))
    assert not sg[:, nbc:].any()
    want = oracle.fp4_codes(x64, er[:, np.arange(C) // B], mode == "sr", r16)
    np.testing.assert_array_equal(_unpack(q["codes"], C), want)
    # colwise: block maxima along rows
    nbr = -(-R // B)
    cmax = np.stack([np.abs(x64[i * B:(i + 1) * B, :]).max(axis=0) for i in range(nbr)], axis=0)
    ec = np.vectorize(oracle.fp4_scale_exponent)(cmax).astype(np.int64)
    np.testing.assert_array_equal(oracle.scale_grid_1d(q["scales_t"], C)[:, :nbr], (ec.T + 127).astype(np.uint8))
    wantc = oracle.fp4_codes(x64, ec[np.arange(R) // B, :], mode == "sr", r16)
    np.testing.assert_array_equal(_unpack(q["codes_t"], R), wantc.T)
    # round to nearest: |Q(x) - x| <= S * delta / 2 <= S (largest E2M1 spacing is 2)
    if mode == "rtn":
        d = np.abs(oracle.operand(q, False, "fp4_1d") - x64)
        assert np.all(d <= np.ldexp(1.0, er[:, np.arange(C) // B]))
