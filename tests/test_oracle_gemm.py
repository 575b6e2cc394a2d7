"""Pins of the oracle's GEMMs and MXFP8 layouts.

* With every block scale 2^0 the three GEMMs reduce to an exact integer matmul
  of 2 * E2M1 values (int64), which the float64 oracle must equal exactly.
* A tiny GEMM in exact Python rationals equals the float64 oracle to 1e-15.
* The linear layer's backward GEMMs reuse the forward's quantized operands in
  transposed form (Sec. 3; App. C, App. D): dX = dY W and dW = dY^T X with
  the very values of Q(W) and Q(X) used by Y = X W^T.
* MXFP8 rowwise / colwise copies: 1x32 blocks along each direction (Sec. 3.2).
"""
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle
import synth


def _unit_scale_input(R, C, seed):
    """Values on the E2M1 grid with every 32x32 block holding a 6 (so e = 0)."""
    rng = np.random.default_rng(seed)
    g = np.array([0, .5, 1, 1.5, 2, 3, 4, 6])
    x = g[rng.integers(0, 8, (R, C))] * rng.choice([-1, 1], (R, C))
    x[::32, ::32] = 6.0
    return torch.from_numpy(x.astype(np.float32))


def test_unit_scales_reduce_to_integer_matmul():
    X = _unit_scale_input(96, 160, 1)
    W = _unit_scale_input(64, 160, 2)
    dY = _unit_scale_input(96, 64, 3)
    qx, qw, qdy = (oracle.quantize_fp4_2d(t, "rtn") for t in (X, W, dY))
    for q in (qx, qw, qdy):
        assert np.all(q["scales"][:, :-(-q["cols"] // 32)] == 127)
    out = oracle.linear(qx, qw, qdy)
    xi = (2 * X.numpy()).astype(np.int64)
    wi = (2 * W.numpy()).astype(np.int64)
    dyi = (2 * dY.numpy()).astype(np.int64)
    assert np.array_equal(out["Y"] * 4, (xi @ wi.T).astype(np.float64))
    assert np.array_equal(out["dX"] * 4, (dyi @ wi).astype(np.float64))
    assert np.array_equal(out["dW"] * 4, (dyi.T @ xi).astype(np.float64))


def test_exact_rational_gemm_tiny():
    X = synth.normal((8, 64), 1.0, 1, torch.float32)
    W = synth.normal((6, 64), 0.02, 2, torch.float32)
    qx, qw = oracle.quantize_fp4_2d(X, "sr", seed=1), oracle.quantize_fp4_2d(W, "sr", seed=1, offset=1)
    a, b = oracle.operand(qx, False), oracle.operand(qw, False)
    got = oracle.gemm(a, b)
    ref = [[sum(Fraction(a[m, k]) * Fraction(b[n, k]) for k in range(64)) for n in range(6)]
           for m in range(8)]
    ref = np.array([[float(v) for v in row] for row in ref])
    assert np.linalg.norm(got - ref) <= 1e-15 * np.linalg.norm(ref)


def test_linear_reuses_operands_transposed():
    X = synth.normal((64, 96), 1.0, 5, torch.bfloat16)
    W = synth.normal((128, 96), 0.02, 6, torch.bfloat16)
    dY = synth.normal((64, 128), 1e-3, 7, torch.bfloat16)
    qx = oracle.quantize_fp4_2d(X, "rtn")
    qw = oracle.quantize_fp4_2d(W, "rtn")
    qdy = oracle.quantize_fp4_2d(dY, "sr", seed=9)
    out = oracle.linear(qx, qw, qdy)
    Xq, Wq, dYq = (oracle.operand(q, False) for q in (qx, qw, qdy))
    np.testing.assert_array_equal(out["Y"], Xq @ Wq.T)
    np.testing.assert_array_equal(out["dX"], dYq @ Wq)
    np.testing.assert_array_equal(out["dW"], dYq.T @ Xq)


@pytest.mark.parametrize("shape", [(64, 96), (70, 33), (1, 200)])
def test_mxfp8_rowwise_colwise(shape):
    x = synth.normal(shape, 1.0, 12, torch.bfloat16)
    synth.add_outlier_channels(x, 13, frac=0.05)
    q = oracle.quantize_mxfp8(x)
    x64 = oracle.to_float64(x)
    R, C = shape
    lay = oracle.mxfp8_layout(R, C)
    assert q["codes"].shape == lay["codes"] and q["codes_t"].shape == lay["codes_t"]
    for r in range(R):
        for J in range(-(-C // 32)):
            blk = x64[r, J * 32:(J + 1) * 32]
            e = oracle.fp8_scale_exponent(np.abs(blk).max())
            assert q["scales"][r, J] == e + 127
            np.testing.assert_array_equal(q["codes"][r, J * 32:J * 32 + len(blk)],
                                          oracle.e4m3_codes(blk, e))
    for c in range(C):
        for I in range(-(-R // 32)):
            blk = x64[I * 32:(I + 1) * 32, c]
            e = oracle.fp8_scale_exponent(np.abs(blk).max())
            assert q["scales_t"][c, I] == e + 127
            np.testing.assert_array_equal(q["codes_t"][c, I * 32:I * 32 + len(blk)],
                                          oracle.e4m3_codes(blk, e))
    assert not q["codes"][:, C:].any() and not q["codes_t"][:, R:].any()
    d = oracle.operand(q, False, "mxfp8")
    assert np.all(np.abs(d - x64) <= np.abs(x64) * 2.0 ** -4 + 2.0 ** -9 * 2.0 ** (
        q["scales"][:, np.arange(C) // 32].astype(np.float64) - 127))
