"""GPU pins of the E4M3 scaled-MFMA arithmetic that the MXFP8 GEMM's error
bound is derived from (the model and the bound: tests/fp8_mfma_model.py).

Operands are written byte by byte into MXFP8 descriptors and multiplied through
q2d_gemm (float32 output), so the pins hold for the library's own kernels:
  * the hand-derived cases: group boundaries, the 13-bit window, truncation of
    each product toward zero, the exponent the window follows, the order of
    group pairs and float32 rounding of the accumulator;
  * random single instructions (every finite E4M3 code, scales 2^-7..2^7)
    equal the model bit for bit, on the small-problem kernel and on the
    large-tile kernel;
  * long-K products stay within the derived bound, and adversarial groups
    (seven products just below the window) come within 0.85 of its first
    term, beyond the 2^-11 |A||B|^T that random data suggests.
"""
from fractions import Fraction

import numpy as np
import pytest
import torch

import fp8_mfma_model as fm

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


@pytest.fixture(scope="module")
def q2d():
    import paper_2607_24953_amd as q
    return q


def mx_operand(q2d, codes: np.ndarray, scales: np.ndarray):
    """An MXFP8 descriptor holding only the row-major copy: the given E4M3 codes
    [R, K] and E8M0 bytes [R, K/32]; the padding codes are zero."""
    R, K = codes.shape
    t = q2d.QTensor(q2d.MXFP8, R, K, DEV, orientations=(True, False))
    c = torch.zeros(t.codes.shape, dtype=torch.uint8)
    c[:, :K] = torch.from_numpy(codes)
    s = torch.full(t.scales.shape, 127, dtype=torch.uint8)
    s[:, :K // 32] = torch.from_numpy(scales.astype(np.uint8))
    t.codes.copy_(c)
    t.scales.copy_(s)
    return t


def gemm(q2d, A, sA, B, sB) -> np.ndarray:
    C = q2d.q2d_gemm(mx_operand(q2d, A, sA), 0, mx_operand(q2d, B, sB), 0, out_dtype=torch.float32)
    torch.cuda.synchronize()
    return C.cpu().numpy()


def random_operand(rng, R, K, lo=120, hi=135):
    c = rng.integers(0, 256, size=(R, K)).astype(np.uint8)
    c[(c & 0x7F) == 0x7F] = 0x38                 # no NaN codes
    return c, rng.integers(lo, hi, size=(R, K // 32))


@pytest.mark.parametrize("K", [64, 128])
def test_hand_derived_cases(q2d, K):
    cases = [c for c in fm.CASES if c[0] == K]
    R = 32
    A = np.zeros((R, K), np.uint8)
    B = np.zeros((R, K), np.uint8)
    sA = np.full((R, K // 32), 127)
    sB = np.full((R, K // 32), 127)
    for i, (_, terms, sa, _, _) in enumerate(cases):
        A[i], sA[i], B[i], sB[i] = fm.case_operands(K, terms, sa)
    C = gemm(q2d, A, sA, B, sB)
    for i, (_, terms, sa, want, why) in enumerate(cases):
        assert C[i, i] == np.float32(want), "%s: gpu %.17g, expected %.17g" % (why, C[i, i], want)


def test_single_instruction_bit_exact_small_kernel(q2d):
    rng = np.random.default_rng(21)
    A, sA = random_operand(rng, 64, 64)
    B, sB = random_operand(rng, 64, 64)
    C = gemm(q2d, A, sA, B, sB)
    for m in range(64):
        for n in range(64):
            assert Fraction(float(C[m, n])) == fm.dot(A[m], sA[m], B[n], sB[n]), (m, n)


def test_single_instruction_bit_exact_large_kernel(q2d):
    """4096 x 2048 outputs (128 tiles of 256 x 256: the large-tile kernel), one
    instruction each; 512 sampled outputs against the model."""
    rng = np.random.default_rng(22)
    A, sA = random_operand(rng, 4096, 64, 124, 131)
    B, sB = random_operand(rng, 2048, 64, 124, 131)
    C = gemm(q2d, A, sA, B, sB)
    for m, n in zip(rng.integers(0, 4096, 512), rng.integers(0, 2048, 512)):
        assert Fraction(float(C[m, n])) == fm.dot(A[m], sA[m], B[n], sB[n]), (m, n)


def _check_bound(C, A, sA, B, sB):
    qa = {"rows": A.shape[0], "cols": A.shape[1], "codes": A, "scales": sA.astype(np.uint8)}
    qb = {"rows": B.shape[0], "cols": B.shape[1], "codes": B, "scales": sB.astype(np.uint8)}
    av, am = fm.operand_fields(qa, False)
    bv, bm = fm.operand_fields(qb, False)
    exact = av @ bv.T                   # exact: every product and partial sum fits float64 here
    bound = fm.error_bound(av, am, bv, bm)
    err = np.abs(C.astype(np.float64) - exact)
    assert np.all(err <= bound), float((err / bound).max())
    return err, exact, np.abs(av) @ np.abs(bv).T, am @ bm.T


@pytest.mark.parametrize("K", [256, 4096])
def test_long_k_within_bound(q2d, K):
    rng = np.random.default_rng(K)
    # scales 126..128: the float64 products and partial sums of the check stay exact
    A, sA = random_operand(rng, 96, K, 126, 129)
    B, sB = random_operand(rng, 64, K, 126, 129)
    _check_bound(gemm(q2d, A, sA, B, sB), A, sA, B, sB)


@pytest.mark.parametrize("K", [64, 1024])
def test_adversarial_groups(q2d, K):
    """Each group of 8 holds one product 1 and seven of 1.75 * 2^-14, just below
    its window: all seven are cut, in every group of every instruction."""
    t = fm.e4m3_table()
    a = np.array([fm.encode(1.0 if k % 8 == 0 else 1.75 * 2.0 ** -7, t) for k in range(K)], np.uint8)
    b = np.array([fm.encode(1.0 if k % 8 == 0 else 2.0 ** -7, t) for k in range(K)], np.uint8)
    A = np.tile(a, (32, 1))
    B = np.tile(b, (32, 1))
    s = np.full((32, K // 32), 127)
    C = gemm(q2d, A, s, B, s)
    assert np.all(C == K // 8)
    err, exact, P, X = _check_bound(C, A, s, B, s)
    assert np.all(err > 2.0 ** -11 * P)
    assert np.all(err >= 0.85 * 7 * 2.0 ** -13 * X)
