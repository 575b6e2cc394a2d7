"""Pins of the oracle's floor scale rule, the rule that the truncation-free
ablation goes back to (Sec. 4.2, the ablation figure; App. G, "Truncation-free
scaling").

* The exponent against a brute-force search for the largest integer e with
  4 * 2^e <= M (floor(log2 M) minus E2M1's largest exponent 2), clamped to -127,
  for every positive finite bfloat16 M and float32 edges.
* It is the truncation-free exponent or one less (less exactly when M's
  mantissa exceeds 1.5), so it never gives a larger scale.
* A hand-derived block: saturation of the maximum and round to nearest below it.
* Element-wise definition against numpy block maxima (codes saturate at 6).
* Clipping: under the truncation-free rule every |x| <= 6 S and round to
  nearest stays within S (half the largest E2M1 spacing) of x; under the floor
  rule the elements above 6 S are clipped to 6 S (a block maximum loses up to a
  quarter of its magnitude) and every other element keeps the same bound.
"""
import numpy as np
import pytest
import torch

import oracle
import synth


def _brute_floor(M: np.ndarray) -> np.ndarray:
    out = np.full(M.shape, -127, dtype=np.int64)
    for e in range(-127, 128):
        out = np.where(4.0 * np.ldexp(1.0, e) <= M, e, out)
    return out


def _unpack(packed, n):
    u = np.empty((packed.shape[0], packed.shape[1] * 2), dtype=np.uint8)
    u[:, 0::2] = packed & 15
    u[:, 1::2] = packed >> 4
    return u[:, :n]


def test_floor_exponent_every_bf16_maximum():
    M = (np.arange(1, 0x7F80, dtype=np.uint32) << 16).view(np.float32).astype(np.float64)
    got = np.array([oracle.fp4_floor_exponent(m) for m in M])
    assert np.array_equal(got, _brute_floor(M))
    tf = np.array([oracle.fp4_scale_exponent(m) for m in M])
    d = tf - got
    assert set(np.unique(d)) <= {0, 1}
    # one less exactly when the mantissa exceeds 1.5 (and above the clamp)
    mant, _ = np.frexp(M)                      # M = mant * 2^p, mant in [0.5, 1)
    big = (mant > 0.75) & (M >= 2.0 ** -125)
    assert np.array_equal(d == 1, big)


@pytest.mark.parametrize("M,e", [(0.0, -127), (np.float32(1e-45), -127), (2.0 ** -125, -127),
                                 (2.0 ** -124, -126), (3.9, -1), (4.0, 0), (7.99, 0), (8.0, 1),
                                 (3.0e38, 125)])
def test_floor_exponent_edges(M, e):
    assert oracle.fp4_floor_exponent(float(M)) == e


def test_hand_derived_block():
    # max 7: floor(log2 7) - 2 = 0 (byte 127); 7 saturates to 6 (index 7); 3.5 is a
    # tie of 3 (index 5) and 4 (index 6): even index 6; -0.3 -> 0.5 (index 1), negative.
    # The truncation-free rule gives e = 1 here (6 * 2^0 < 7): 7 / 2 = 3.5 -> 4 (index 6).
    x = np.zeros((32, 32), dtype=np.float32)
    x[0, :3] = [7.0, 3.5, -0.3]
    q = oracle.quantize_fp4_2d(x, "rtn-floor")
    assert q["scales"][0, 0] == 127
    assert list(_unpack(q["codes"], 32)[0, :3]) == [7, 6, 9]
    qt = oracle.quantize_fp4_2d(x, "rtn")
    assert qt["scales"][0, 0] == 128 and _unpack(qt["codes"], 32)[0, 0] == 6
    # max 3.9: e = -1 (byte 126); 3.9 / 0.5 = 7.8 saturates to 6, i.e. 3.0
    x[0, :3] = [3.9, 0.0, 0.0]
    q = oracle.quantize_fp4_2d(x, "rtn-floor")
    assert q["scales"][0, 0] == 126 and _unpack(q["codes"], 32)[0, 0] == 7
    assert oracle.dequantize(q, 0)[0, 0] == 3.0


@pytest.mark.parametrize("shape", [(96, 160), (70, 100), (33, 65)])
@pytest.mark.parametrize("mode", ["rtn-floor", "sr-floor"])
def test_floor_elementwise_definition(shape, mode):
    R, C = shape
    x = synth.add_outlier_channels(synth.normal(shape, 0.8, 91, torch.bfloat16), 92, frac=0.05)
    q = oracle.quantize_fp4_2d(x, mode, seed=4, offset=1)
    x64 = oracle.to_float64(x)
    nbr, nbc = -(-R // 32), -(-C // 32)
    bm = np.array([[np.abs(x64[i * 32:(i + 1) * 32, j * 32:(j + 1) * 32]).max() for j in range(nbc)]
                   for i in range(nbr)])
    e = _brute_floor(bm)
    np.testing.assert_array_equal(q["scales"][:, :nbc], (e + 127).astype(np.uint8))
    eb = e[np.arange(R)[:, None] // 32, np.arange(C)[None, :] // 32]
    sr = mode.startswith("sr")
    idx = np.arange(R)[:, None] * x.stride(0) + np.arange(C)[None, :]
    r16 = np.vectorize(lambda i: oracle.sr_bits(int(i), 4, 1))(idx).astype(np.uint32) if sr else None
    want = oracle.fp4_codes(x64, eb, sr, r16)
    np.testing.assert_array_equal(_unpack(q["codes"], C), want)
    np.testing.assert_array_equal(_unpack(q["codes_t"], R), want.T)


def test_clipping_under_each_rule():
    x = synth.normal((256, 256), 1.0, 93, torch.float32)
    x64 = oracle.to_float64(x)
    for mode, clipped in (("rtn", False), ("rtn-floor", True)):
        q = oracle.quantize_fp4_2d(x, mode)
        S = np.ldexp(1.0, oracle.scale_exponents(q, 0))
        v = oracle.dequantize(q, 0)
        over = np.abs(x64) > 6 * S
        assert over.any() == clipped
        assert np.all(np.abs(v - x64)[~over] <= S[~over])
        assert np.array_equal(v[over], np.sign(x64[over]) * 6 * S[over])
        assert np.all(np.abs(v[over]) >= 0.75 * np.abs(x64[over]))
