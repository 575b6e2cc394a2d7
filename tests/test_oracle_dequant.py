"""Pins of the oracle's dequantization and scale-exponent maps (the forward and
backward copies X_fwd, X_bwd of Sec. 2, "Bias induced by scale inconsistency";
the scale-difference and effective-deviation maps of Fig. 1).

* E4M3FN decoding of all 256 codes against torch's float8_e4m3fn conversion.
* Exponent maps against a brute-force search for the smallest e with
  Qp * 2^e >= block maximum (Qp = 6 for E2M1, 448 for E4M3) over numpy block
  maxima, for 2D blocks (32 and 64), both 1D copies and both MXFP8 copies.
* 2D blocks: the two copies dequantize to the same values and exponents
  (transposition invariance, Sec. 3); 1D blocks: the exponent maps differ
  exactly where the row block's and the column block's maxima give different
  exponents, and with round to nearest the values differ only there.
"""
import numpy as np
import pytest
import torch

import oracle
import synth


def _brute_exponent(M: np.ndarray, qp: float) -> np.ndarray:
    """Smallest integer e in [-127, 127] with qp * 2^e >= M (elementwise, by search)."""
    out = np.full(M.shape, 127, dtype=np.int64)
    for e in range(126, -128, -1):
        out = np.where(qp * np.ldexp(1.0, e) >= M, e, out)
    return out


def _maxima(a: np.ndarray, br: int, bc: int) -> np.ndarray:
    """Per-element maximum of |a| over the br x bc block holding it."""
    R, C = a.shape
    out = np.zeros_like(a)
    for i in range(0, R, br):
        for j in range(0, C, bc):
            out[i:i + br, j:j + bc] = np.abs(a[i:i + br, j:j + bc]).max()
    return out


def test_e4m3_decoding_matches_torch():
    codes = np.arange(256, dtype=np.uint8).reshape(8, 32)
    scales = np.full((8, 4), 127, dtype=np.uint8)          # e = 0
    got = oracle.dequant_mxfp8(np.pad(codes, ((0, 0), (0, 96))), scales, 8, 32)
    want = torch.from_numpy(codes.reshape(-1).copy()).view(torch.float8_e4m3fn).float().numpy().reshape(8, 32)
    assert np.array_equal(np.isnan(got), np.isnan(want))
    ok = ~np.isnan(want)
    assert np.array_equal(got[ok], want[ok].astype(np.float64))
    assert np.isnan(got).sum() == 2                         # 0x7F and 0xFF


@pytest.mark.parametrize("block", [32, 64])
@pytest.mark.parametrize("mode", ["rtn", "sr"])
def test_2d_copies_agree_and_exponents_follow_definition(block, mode):
    x = synth.add_outlier_channels(synth.normal((150, 200), 1.0, 81, torch.bfloat16), 82, frac=0.05)
    q = oracle.quantize_fp4_2d(x, mode, 3, 4, block=block)
    v0, v1 = oracle.dequantize(q, 0), oracle.dequantize(q, 1)
    e0, e1 = oracle.scale_exponents(q, 0), oracle.scale_exponents(q, 1)
    assert np.array_equal(v0, v1) and np.array_equal(e0, e1)
    x64 = oracle.to_float64(x)
    assert np.array_equal(e0, _brute_exponent(_maxima(x64, block, block), 6.0))


@pytest.mark.parametrize("mode", ["rtn", "sr"])
def test_1d_exponent_maps_and_mismatch(mode):
    x = synth.add_outlier_channels(synth.normal((100, 130), 1.0, 83, torch.bfloat16), 84, frac=0.05)
    x64 = oracle.to_float64(x)
    q = oracle.quantize_fp4_1d(x, mode, 5, 6)
    e0, e1 = oracle.scale_exponents(q, 0, "fp4_1d"), oracle.scale_exponents(q, 1, "fp4_1d")
    want0 = _brute_exponent(_maxima(x64, 1, 32), 6.0)      # 1 x 32 row blocks
    want1 = _brute_exponent(_maxima(x64, 32, 1), 6.0)      # 32 x 1 column blocks
    assert np.array_equal(e0, want0) and np.array_equal(e1, want1)
    assert (e0 != e1).any()
    if mode == "rtn":
        v0, v1 = oracle.dequantize(q, 0, "fp4_1d"), oracle.dequantize(q, 1, "fp4_1d")
        same = e0 == e1
        assert np.array_equal(v0[same], v1[same])
        assert (v0[~same] != v1[~same]).any()


def test_mxfp8_exponent_maps():
    x = synth.normal((70, 100), 1.0, 85, torch.bfloat16)
    x64 = oracle.to_float64(x)
    q = oracle.quantize_mxfp8(x)
    assert np.array_equal(oracle.scale_exponents(q, 0, "mxfp8"), _brute_exponent(_maxima(x64, 1, 32), 448.0))
    assert np.array_equal(oracle.scale_exponents(q, 1, "mxfp8"), _brute_exponent(_maxima(x64, 32, 1), 448.0))


def test_non_finite_block_exponent():
    x = np.zeros((64, 64), dtype=np.float32)
    x[5, 40] = np.nan
    q = oracle.quantize_fp4_2d(x, "rtn")
    e = oracle.scale_exponents(q, 0)
    assert (e[:32, 32:] == -128).all() and (e[:32, :32] == -127).all()
    assert np.isnan(oracle.dequantize(q, 1)[:32, 32:]).all()
