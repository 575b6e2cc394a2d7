"""Pins of the oracle's GEMM with a quantized result (a layer output that is the
next GEMM's operand; App. C).

* Unit-scale operands on the E2M1 grid make the float64 product exact and
  representable in float32; the quantized result then equals the quantizer
  applied to an integer-matrix product computed with int64 arithmetic.
* The result is transposition invariant: quantizing C^T gives the other
  orientation of quantizing C (the 2D-block property, Sec. 3).
"""
import numpy as np
import torch

import oracle

GRID = np.array([0, 0.5, 1, 1.5, 2, 3, 4, 6])


def _grid_matrix(rows, cols, seed):
    """Values on the E2M1 grid with a 6 in every 32 x 32 block (scale 2^0)."""
    rng = np.random.default_rng(seed)
    x = GRID[rng.integers(0, 8, (rows, cols))] * rng.choice([-1, 1], (rows, cols))
    x[::32, ::32] = 6.0
    return x.astype(np.float32)


def test_unit_scale_product_is_exact():
    a, b = _grid_matrix(96, 160, 1), _grid_matrix(70, 160, 2)
    qa, qb = oracle.quantize_fp4_2d(a, "rtn"), oracle.quantize_fp4_2d(b, "rtn")
    assert (qa["scales"][:, :5] == 127).all() and (qb["scales"][:, :5] == 127).all()
    A, B = oracle.operand(qa, False), oracle.operand(qb, False)
    assert np.array_equal(A, a) and np.array_equal(B, b)
    ci = (a * 2).astype(np.int64) @ (b * 2).astype(np.int64).T         # exact, in quarters
    q = oracle.gemm_quantized(A, B)
    want = oracle.quantize_fp4_2d((ci / 4.0).astype(np.float32), "rtn")
    for k in ("codes", "codes_t", "scales", "scales_t"):
        assert np.array_equal(q[k], want[k]), k


def test_transposed_result_swaps_orientations():
    rng = np.random.default_rng(3)
    a = rng.standard_normal((100, 96)).astype(np.float32)
    b = rng.standard_normal((130, 96)).astype(np.float32)
    A = oracle.operand(oracle.quantize_fp4_2d(a, "rtn"), False)
    B = oracle.operand(oracle.quantize_fp4_2d(b, "rtn"), False)
    q, qt = oracle.gemm_quantized(A, B), oracle.gemm_quantized(B, A)
    assert np.array_equal(q["codes"], qt["codes_t"]) and np.array_equal(q["codes_t"], qt["codes"])
    assert np.array_equal(q["scales"], qt["scales_t"]) and np.array_equal(q["scales_t"], qt["scales"])


def test_stochastic_unit_scale_product_is_exact():
    """SR of an exactly representable product (App. E) equals the SR quantizer
    applied to the integer-matrix product with the same stream."""
    a, b = _grid_matrix(96, 160, 4), _grid_matrix(72, 160, 5)
    A = oracle.operand(oracle.quantize_fp4_2d(a, "rtn"), False)
    B = oracle.operand(oracle.quantize_fp4_2d(b, "rtn"), False)
    ci = (a * 2).astype(np.int64) @ (b * 2).astype(np.int64).T
    q = oracle.gemm_quantized(A, B, "sr", 9, 2 ** 33 + 1)
    want = oracle.quantize_fp4_2d((ci / 4.0).astype(np.float32), "sr", 9, 2 ** 33 + 1)
    for k in ("codes", "codes_t", "scales", "scales_t"):
        assert np.array_equal(q[k], want[k]), k


def test_stochastic_result_is_unbiased_between_grid_neighbours():
    """Each SR value of the product is one of the two E2M1 neighbours of the
    exact value under its block scale, and the mean over 4000 offsets is the
    exact value within 5 standard errors plus the 2^-16 resolution of the draws
    (E[round(x)] = x, App. E)."""
    rng = np.random.default_rng(6)
    a = rng.standard_normal((32, 64)).astype(np.float32)
    b = rng.standard_normal((32, 64)).astype(np.float32)
    A = oracle.operand(oracle.quantize_fp4_2d(a, "rtn"), False)
    B = oracle.operand(oracle.quantize_fp4_2d(b, "rtn"), False)
    c = oracle.gemm(A, B).astype(np.float32).astype(np.float64)
    e = oracle.fp4_scale_exponent(float(np.abs(c).max()))
    s = 2.0 ** e
    mag = np.abs(c) / s
    k = np.searchsorted(GRID, mag, side="right") - 1
    lo_v = GRID[k] * s
    hi_v = GRID[np.minimum(k + 1, 7)] * s
    n = 4000
    acc = np.zeros_like(c)
    for off in range(n):
        v = oracle.dequantize(oracle.gemm_quantized(A, B, "sr", 3, off), 0)
        av = np.abs(v)
        assert np.all((av == lo_v) | (av == hi_v)), off
        assert np.all((v == 0) | (np.sign(v) == np.sign(c)))
        acc += v
    mean = acc / n
    delta = hi_v - lo_v
    p = np.where(delta > 0, (np.abs(c) - lo_v) / np.where(delta > 0, delta, 1), 0)
    se = delta * np.sqrt(p * (1 - p) / n)
    assert np.all(np.abs(mean - c) <= 5 * se + delta * 2.0 ** -16 + 1e-300)
