"""GPU parity of q2d_gemm_quantized (the GEMM result quantized to 2D-block FP4
in the epilogue; App. C) against the oracle.

* Exact cases: operands on the E2M1 grid with a 6 in every block (unit
  scales) make the float32 accumulation exact, so every byte of the four
  output buffers must equal the oracle's quantization of the exact product:
  ragged shapes on one and several 256 x 256 tiles, all transpose flags, 1D
  operands, a result that overflows float32 (scale 0xFF, zero codes).
* General cases (normal inputs, mixed scales): the float32 accumulation may
  move a value across a rounding boundary, so the check is that the result is
  a valid quantization of a value within the accumulation error bound of the
  exact product -- every block's exponent is the truncation-free exponent of a
  maximum within the bound, every code the round-to-nearest code of a value
  within the bound under that exponent -- and that nearly every byte equals
  the oracle's; the two orientations agree exactly (transposition invariance).
* The full 7B forward shape (QKV, 16384 x 12288 x 4096) on sampled rows.
* Stochastic rounding (a data gradient dX that is the next layer's output
  gradient; App. E): the same exact cases bit for bit against the oracle's SR
  quantization of the product (element (r, c) keyed by storage index r N + c),
  general cases valid under each element's own draw, and the full 7B QKV data
  gradient shape on sampled rows.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from helpers import assert_same_bytes, gpu_buffers, poison

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
GRID = np.array([0, 0.5, 1, 1.5, 2, 3, 4, 6], dtype=np.float32)


@pytest.fixture(scope="module")
def q2d():
    import paper_2607_24953_amd as q
    return q


def _grid_matrix(rows, cols, seed, scale=1.0):
    """E2M1 grid values with a 6 in every 32 x 32 block and in every 1 x 32 and
    32 x 1 run (so the 2D and both 1D scales are all `scale`)."""
    rng = np.random.default_rng(seed)
    x = GRID[rng.integers(0, 8, (rows, cols))] * rng.choice(np.array([-1, 1], np.float32), (rows, cols))
    x[::32, :] = 6.0
    x[:, ::32] = 6.0
    return torch.from_numpy(x * np.float32(scale))


def _quant(q2d, x, fmt):
    """Device and oracle quantization (bytes checked equal)."""
    xd = x.to(DEV)
    if fmt == "fp4_1d":
        q, o = q2d.q2d_quantize_1d(xd, "rtn"), oracle.quantize_fp4_1d(x, "rtn")
    else:
        q, o = q2d.q2d_quantize(xd, "rtn"), oracle.quantize_fp4_2d(x, "rtn")
    assert_same_bytes(gpu_buffers(q), o, "operand %s" % fmt)
    return q, o


def _run(q2d, qa, ta, qb, tb, M, N, mode="rtn", seed=0, offset=0):
    out = q2d.QTensor(q2d.FP4_2D, M, N, DEV)
    poison(out)
    q2d.q2d_gemm_quantized(qa, ta, qb, tb, mode, out=out, seed=seed, offset=offset)
    got = gpu_buffers(out)
    got["rows"], got["cols"] = M, N
    return got


EXACT = [
    # M, N, K, ta, tb, fmt_a, fmt_b
    (128, 256, 256, 0, 0, "fp4", "fp4"),
    (300, 200, 160, 0, 1, "fp4", "fp4"),
    (257, 129, 96, 1, 1, "fp4", "fp4"),
    (1, 1, 32, 0, 0, "fp4", "fp4"),
    (33, 65, 64, 1, 0, "fp4", "fp4"),
    (2100, 4000, 384, 0, 0, "fp4", "fp4"),
    (4096, 2048, 640, 1, 1, "fp4", "fp4"),
    (1000, 700, 256, 0, 0, "fp4_1d", "fp4"),
    (600, 900, 320, 1, 1, "fp4", "fp4_1d"),
]


@pytest.mark.parametrize("M,N,K,ta,tb,fa,fb", EXACT)
def test_exact_products_bit_exact(q2d, M, N, K, ta, tb, fa, fb):
    a = _grid_matrix(K, M, M + K) if ta else _grid_matrix(M, K, M + K)
    b = _grid_matrix(K, N, N + 3 * K) if tb else _grid_matrix(N, K, N + 3 * K)
    qa, oa = _quant(q2d, a, fa)
    qb, ob = _quant(q2d, b, fb)
    A, B = oracle.operand(oa, bool(ta), fa), oracle.operand(ob, bool(tb), fb)
    got = _run(q2d, qa, ta, qb, tb, M, N)
    want = oracle.gemm_quantized(A, B)
    assert_same_bytes(got, want, "%dx%dx%d %s %s" % (M, N, K, fa, fb))


def test_overflowing_result(q2d):
    """Products of 6 * 2^100 blocks overflow float32: scale byte 0xFF, zero codes."""
    a = _grid_matrix(256, 128, 5, 2.0 ** 100)
    b = _grid_matrix(256, 128, 6, 2.0 ** 100)
    qa, oa = _quant(q2d, a, "fp4")
    qb, ob = _quant(q2d, b, "fp4")
    got = _run(q2d, qa, 0, qb, 0, 256, 256)
    want = oracle.gemm_quantized(oracle.operand(oa, False), oracle.operand(ob, False))
    assert (want["scales"] == 0xFF).any()
    assert_same_bytes(got, want, "overflow")


def _rtn_values(x, e):
    """Round-to-nearest E2M1 values of x under exponents e (the oracle's codec)."""
    codes = oracle.fp4_codes(x, e, False, None)
    mag = GRID[codes & 7].astype(np.float64)
    return np.where(codes & 8, -mag, mag) * np.ldexp(1.0, e)


def check_valid(got, A, B, label, min_exact=0.99):
    """got is a valid round-to-nearest quantization of a value within the float32
    accumulation bound of the exact product, and mostly byte-equal to the oracle."""
    M, N = A.shape[0], B.shape[0]
    K = A.shape[1]
    C = oracle.gemm(A, B)
    eps = (K / 64 + 2) * 2.0 ** -24 * (np.abs(A) @ np.abs(B).T)
    e = oracle.scale_exponents(got, 0)
    # both orientations carry the same values (transposition invariance)
    assert np.array_equal(e, oracle.scale_exponents(got, 1)), label
    v = oracle.dequantize(got, 0)
    assert np.array_equal(v, oracle.dequantize(got, 1)), label
    # block exponents
    nbr, nbc = -(-M // 32), -(-N // 32)
    pad = lambda t: np.pad(t, ((0, nbr * 32 - M), (0, nbc * 32 - N)))
    blk = lambda t: pad(t).reshape(nbr, 32, nbc, 32).max(axis=(1, 3))
    Mb, Eb = blk(np.abs(C)), blk(eps)
    tf = np.vectorize(oracle.fp4_scale_exponent)
    e_lo, e_hi = tf(np.maximum(Mb - Eb, 0.0)), tf(Mb + Eb)
    eb = e[::32, ::32]
    assert np.all((e_lo <= eb) & (eb <= e_hi)), label
    # codes: between the RTN values of C - eps and C + eps under the kernel's exponent
    lo, hi = _rtn_values(C - eps, e), _rtn_values(C + eps, e)
    bad = (v < lo) | (v > hi)
    assert not bad.any(), (label, int(bad.sum()), np.argwhere(bad)[:3])
    want = oracle.gemm_quantized(A, B)
    same = np.mean(oracle.dequantize(want, 0) == v)
    assert same >= min_exact, (label, same)


GENERAL = [
    (300, 200, 160, 0, 0, "fp4", "fp4"),
    (257, 129, 96, 1, 1, "fp4", "fp4"),
    (2100, 4000, 384, 0, 1, "fp4", "fp4"),
    (1024, 1536, 2048, 1, 1, "fp4", "fp4"),
    (1000, 700, 512, 0, 0, "fp4_1d", "fp4"),
]


@pytest.mark.parametrize("M,N,K,ta,tb,fa,fb", GENERAL)
def test_general_products_valid(q2d, M, N, K, ta, tb, fa, fb):
    a = synth.normal((K, M) if ta else (M, K), 1.0, 7 * M + K, torch.bfloat16)
    synth.add_outlier_channels(a, 8, frac=0.02)
    b = synth.normal((K, N) if tb else (N, K), 0.02, 9 * N + K, torch.bfloat16)
    qa, oa = _quant(q2d, a, fa)
    qb, ob = _quant(q2d, b, fb)
    A, B = oracle.operand(oa, bool(ta), fa), oracle.operand(ob, bool(tb), fb)
    got = _run(q2d, qa, ta, qb, tb, M, N)
    check_valid(got, A, B, "%dx%dx%d" % (M, N, K))


def test_full_7b_qkv_sampled(q2d):
    """QKV forward at full size (16384 x 12288 x 4096): every byte written, the two
    orientations equal, and 64 sampled 32-row bands against the oracle's product."""
    X = synth.add_outlier_channels(synth.normal((16384, 4096), 1.0, 3031, torch.bfloat16, device=DEV), 3032)
    W = synth.normal((12288, 4096), 0.02, 3033, torch.bfloat16, device=DEV)
    qx, qw = q2d.q2d_quantize(X, "rtn"), q2d.q2d_quantize(W, "rtn")
    out = q2d.QTensor(q2d.FP4_2D, 16384, 12288, DEV)
    poison(out)
    q2d.q2d_gemm_quantized(qx, 0, qw, 0, "rtn", out=out)
    torch.cuda.synchronize()
    v0 = q2d.q2d_dequantize(out, 0)
    v1 = q2d.q2d_dequantize(out, 1)
    assert torch.equal(v0.view(torch.int32), v1.view(torch.int32))
    assert torch.isfinite(v0).all()
    ow = oracle.quantize_fp4_2d(W.cpu(), "rtn")
    Wd = oracle.operand(ow, False)
    rng = np.random.default_rng(0)
    bands = rng.choice(16384 // 32, 64, replace=False)
    xs = X.cpu()
    got_all = gpu_buffers(out)
    for band in bands:
        r0 = int(band) * 32
        ox = oracle.quantize_fp4_2d(xs[r0:r0 + 32], "rtn")        # a 32-row band holds whole blocks
        A = oracle.operand(ox, False)
        got = {"codes": got_all["codes"][r0:r0 + 32], "scales": got_all["scales"][band:band + 1],
               "codes_t": got_all["codes_t"][:, r0 // 2:r0 // 2 + 16],
               "scales_t": got_all["scales_t"][:, band:band + 1], "rows": 32, "cols": 12288}
        # codes_t / scales_t of the band viewed as a 32-row matrix: pad to the layout width
        got["codes_t"] = np.pad(got["codes_t"], ((0, 0), (0, 48)))
        got["scales_t"] = np.pad(got["scales_t"], ((0, 0), (0, 3)))
        check_valid(got, A, Wd, "7B band %d" % band, min_exact=0.98)


# ------------------------------------------------------------------ stochastic rounding

SR_EXACT = [(128, 256, 256, 0, 0, "fp4", "fp4"), (300, 200, 160, 0, 1, "fp4", "fp4"),
            (257, 136, 96, 1, 1, "fp4", "fp4"), (33, 64, 64, 1, 0, "fp4", "fp4"),
            (2100, 4000, 384, 0, 0, "fp4", "fp4"), (4096, 2048, 640, 1, 1, "fp4", "fp4"),
            (1000, 704, 256, 0, 0, "fp4_1d", "fp4"), (600, 904, 320, 1, 1, "fp4", "fp4_1d")]


@pytest.mark.parametrize("M,N,K,ta,tb,fa,fb", SR_EXACT)
def test_stochastic_exact_products_bit_exact(q2d, M, N, K, ta, tb, fa, fb):
    a = _grid_matrix(K, M, M + K + 1) if ta else _grid_matrix(M, K, M + K + 1)
    b = _grid_matrix(K, N, N + 3 * K + 1) if tb else _grid_matrix(N, K, N + 3 * K + 1)
    qa, oa = _quant(q2d, a, fa)
    qb, ob = _quant(q2d, b, fb)
    A, B = oracle.operand(oa, bool(ta), fa), oracle.operand(ob, bool(tb), fb)
    seed, offset = 0x5EED + M, 2 ** 32 + N
    got = _run(q2d, qa, ta, qb, tb, M, N, "sr", seed, offset)
    want = oracle.gemm_quantized(A, B, "sr", seed, offset)
    assert_same_bytes(got, want, "SR %dx%dx%d %s %s" % (M, N, K, fa, fb))


def _sr_values(x, e, r16):
    codes = oracle.fp4_codes(x, e, True, r16)
    mag = GRID[codes & 7].astype(np.float64)
    return np.where(codes & 8, -mag, mag) * np.ldexp(1.0, e)


def check_valid_sr(got, A, B, seed, offset, label, min_exact=0.99):
    """got is the SR quantization, under each element's own draw, of a value
    within the float32 accumulation bound of the exact product, and mostly
    byte-equal to the oracle's."""
    M, N, K = A.shape[0], B.shape[0], A.shape[1]
    C = oracle.gemm(A, B)
    eps = (K / 64 + 2) * 2.0 ** -24 * (np.abs(A) @ np.abs(B).T)
    e = oracle.scale_exponents(got, 0)
    assert np.array_equal(e, oracle.scale_exponents(got, 1)), label
    v = oracle.dequantize(got, 0)
    assert np.array_equal(v, oracle.dequantize(got, 1)), label
    r16 = np.array([oracle.sr_bits(i, seed, offset) for i in range(M * N)], np.uint32).reshape(M, N)
    # SR is monotone in the value for a fixed draw and exponent
    lo, hi = _sr_values(C - eps, e, r16), _sr_values(C + eps, e, r16)
    bad = (v < lo) | (v > hi)
    assert not bad.any(), (label, int(bad.sum()), np.argwhere(bad)[:3])
    want = oracle.gemm_quantized(A, B, "sr", seed, offset)
    same = np.mean(oracle.dequantize(want, 0) == v)
    assert same >= min_exact, (label, same)


@pytest.mark.parametrize("M,N,K,ta,tb,fa,fb", [(300, 200, 160, 0, 0, "fp4", "fp4"),
                                              (257, 136, 96, 1, 1, "fp4", "fp4"),
                                              (512, 768, 2048, 0, 1, "fp4", "fp4"),
                                              (300, 512, 512, 0, 0, "fp4_1d", "fp4")])
def test_stochastic_general_products_valid(q2d, M, N, K, ta, tb, fa, fb):
    a = synth.normal((K, M) if ta else (M, K), 1e-3, 11 * M + K, torch.bfloat16)
    b = synth.normal((K, N) if tb else (N, K), 0.02, 13 * N + K, torch.bfloat16)
    qa, oa = _quant(q2d, a, fa)
    qb, ob = _quant(q2d, b, fb)
    A, B = oracle.operand(oa, bool(ta), fa), oracle.operand(ob, bool(tb), fb)
    got = _run(q2d, qa, ta, qb, tb, M, N, "sr", 77, 5)
    check_valid_sr(got, A, B, 77, 5, "SR %dx%dx%d" % (M, N, K))


def test_stochastic_full_7b_qkv_data_gradient_sampled(q2d):
    """dX = dY_qkv W_qkv at the 7B shape (16384 x 4096 x 12288) quantized with SR in
    the epilogue: both orientations equal, finite, and 8 sampled 32-row bands
    valid against the oracle's product under each element's draw."""
    dY = synth.normal((16384, 12288), 1e-3, 3041, torch.bfloat16, device=DEV)
    W = synth.normal((12288, 4096), 0.02, 3042, torch.bfloat16, device=DEV)
    qdy, qw = q2d.q2d_quantize(dY, "sr", 5, 2), q2d.q2d_quantize(W, "rtn")
    out = q2d.QTensor(q2d.FP4_2D, 16384, 4096, DEV)
    poison(out)
    seed, offset = 5, 9
    q2d.q2d_gemm_quantized(qdy, 0, qw, 1, "sr", out=out, seed=seed, offset=offset)
    torch.cuda.synchronize()
    v0, v1 = q2d.q2d_dequantize(out, 0), q2d.q2d_dequantize(out, 1)
    assert torch.equal(v0.view(torch.int32), v1.view(torch.int32))
    assert torch.isfinite(v0).all()
    Wt = oracle.operand(oracle.quantize_fp4_2d(W.cpu(), "rtn"), True)
    got_all = gpu_buffers(out)
    dys = dY.cpu()
    rng = np.random.default_rng(1)
    for band in rng.choice(16384 // 32, 8, replace=False):
        r0 = int(band) * 32
        # the band of dY quantized as the device did: rows r0.. of the full tensor,
        # so its SR draws use the full tensor's storage indices
        ody = oracle.quantize_fp4_2d(dys[r0:r0 + 32], "sr", 5, 2, index_base=r0 * 12288)
        A = oracle.operand(ody, False)
        C = oracle.gemm(A, Wt)
        eps = (12288 / 64 + 2) * 2.0 ** -24 * (np.abs(A) @ np.abs(Wt).T)
        e = oracle.scale_exponents({"codes": got_all["codes"][r0:r0 + 32], "scales": got_all["scales"][band:band + 1],
                                    "rows": 32, "cols": 4096}, 0)
        v = oracle.dequantize({"codes": got_all["codes"][r0:r0 + 32], "scales": got_all["scales"][band:band + 1],
                               "rows": 32, "cols": 4096}, 0)
        r16 = np.array([oracle.sr_bits((r0 + i) * 4096 + c, seed, offset) for i in range(32) for c in range(4096)],
                       np.uint32).reshape(32, 4096)
        lo, hi = _sr_values(C - eps, e, r16), _sr_values(C + eps, e, r16)
        assert not ((v < lo) | (v > hi)).any(), int(band)
