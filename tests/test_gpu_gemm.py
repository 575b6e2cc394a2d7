"""GPU parity of the block-scaled FP4 and MXFP8 GEMMs against the float64 oracle.

Float32 outputs: relative Frobenius error <= 1e-5 (fp32 accumulation of exact
FP4 x FP4 products).  Bfloat16 outputs: every element within one bf16 rounding
(2^-8 relative) of the float64 result.  Shapes span several 128 x 128 output
tiles and ragged M, N and K tails; all four transpose combinations are used,
the three GEMMs of a linear layer through q2d_linear_fwd/bwd, accumulation,
and the full 7B workload in the launch configuration of the benchmark (bf16 Y
and dX, fp32 dW) on sampled output rows.
"""
import numpy as np
import pytest
import torch

import fp8_mfma_model as fm
import oracle
import synth
from helpers import as_oracle_tensor, assert_same_bytes, check_bf16, gpu_buffers, rel_frob

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
TOL = 1e-5


@pytest.fixture(scope="module")
def q2d():
    import paper_2607_24953_amd as q
    return q


def quant(q2d, x, mode, seed=0, offset=0):
    """Device quantization of x and the oracle's own quantization of the same input
    (byte-equal; the oracle's copy feeds the float64 reference GEMM)."""
    q = q2d.q2d_quantize(x, mode, seed, offset)
    o = oracle.quantize_fp4_2d(x.cpu(), mode, seed, offset)
    assert_same_bytes(gpu_buffers(q), o, "operand")
    return q, o


GEMM_SHAPES = [(128, 256, 256), (300, 200, 160), (257, 129, 96), (1, 1, 32), (64, 640, 1000),
               (1000, 300, 2000), (384, 512, 4096),
               # enough 256 x 256 output tiles for the large-tile kernel: ragged M and N,
               # K shorter than its LDS pipeline (128, 384) and long (2048)
               (2048, 4096, 128), (2100, 4000, 384), (4096, 2048, 2048)]


@pytest.mark.parametrize("M,N,K", GEMM_SHAPES)
@pytest.mark.parametrize("ta,tb", [(0, 0), (0, 1), (1, 1), (1, 0)])
def test_gemm_fp4(q2d, M, N, K, ta, tb):
    a_shape = (K, M) if ta else (M, K)
    b_shape = (K, N) if tb else (N, K)
    A = synth.normal(a_shape, 1.0, M + K, torch.bfloat16, device=DEV)
    B = synth.normal(b_shape, 0.02, N + K + 1, torch.bfloat16, device=DEV)
    qa, oa = quant(q2d, A, "sr", 1, 0)
    qb, ob = quant(q2d, B, "rtn")
    ref = oracle.gemm(oracle.operand(oa, bool(ta)), oracle.operand(ob, bool(tb)))
    c32 = q2d.q2d_gemm(qa, ta, qb, tb, out_dtype=torch.float32)
    assert rel_frob(c32.cpu().numpy(), ref) <= TOL
    c16 = q2d.q2d_gemm(qa, ta, qb, tb, out_dtype=torch.bfloat16)
    check_bf16(c16, ref)


# More output tiles than the device has CUs, so every workgroup of the
# persistent kernel walks several tiles; K of 1, 3 and 5 K-tiles (fewer than,
# and more than, the LDS ring's four stages, so one tile's loads run into the
# next tile's) and ragged M and N edges.
MULTI_TILE_SHAPES = [(4200, 4100, 128), (4100, 4200, 384), (6000, 3000, 640)]


@pytest.mark.parametrize("M,N,K", MULTI_TILE_SHAPES)
@pytest.mark.parametrize("ta,tb", [(0, 0), (0, 1), (1, 1)])
def test_gemm_fp4_multi_tile_per_workgroup(q2d, M, N, K, ta, tb):
    a_shape = (K, M) if ta else (M, K)
    b_shape = (K, N) if tb else (N, K)
    A = synth.normal(a_shape, 1.0, 7 * M + K, torch.bfloat16, device=DEV)
    B = synth.normal(b_shape, 0.02, 7 * N + K + 1, torch.bfloat16, device=DEV)
    qa, oa = quant(q2d, A, "rtn")
    qb, ob = quant(q2d, B, "sr", 3, 0)
    ref = oracle.gemm(oracle.operand(oa, bool(ta)), oracle.operand(ob, bool(tb)))
    c32 = q2d.q2d_gemm(qa, ta, qb, tb, out_dtype=torch.float32)
    assert rel_frob(c32.cpu().numpy(), ref) <= TOL
    # bf16 output accumulated onto an existing C
    c0 = synth.normal((M, N), 0.5, 11, torch.bfloat16, device=DEV)
    c16 = c0.clone()
    q2d.q2d_gemm(qa, ta, qb, tb, out=c16, accumulate=True)
    check_bf16(c16, ref + c0.float().cpu().numpy().astype(np.float64))


# bf16 output of the persistent kernel into views of a wider buffer: an even
# row pitch (whole-line pair stores), an odd one and a base one element off
# (both one store per element), with and without accumulation; N is odd, so the
# last column of every row is a lone element.  Nothing outside the view changes.
@pytest.mark.parametrize("pad,base", [(6, 0), (1, 0), (2, 1)])
@pytest.mark.parametrize("acc", [False, True])
def test_gemm_bf16_strided_output(q2d, pad, base, acc):
    M, N, K = 2100, 4001, 384                       # 9 x 16 output tiles of 256 x 256
    A = synth.normal((M, K), 1.0, 31, torch.bfloat16, device=DEV)
    B = synth.normal((N, K), 0.02, 32, torch.bfloat16, device=DEV)
    qa, oa = quant(q2d, A, "rtn")
    qb, ob = quant(q2d, B, "sr", 5, 1)
    ref = oracle.gemm(oracle.operand(oa, False), oracle.operand(ob, False))
    ld = N + pad
    flat = synth.normal((M * ld + 2,), 0.5, 33, torch.bfloat16, device=DEV)
    before = flat.clone()
    c = flat[base:base + M * ld].view(M, ld)[:, :N]
    c0 = c.float().cpu().numpy().astype(np.float64)
    q2d.q2d_gemm(qa, 0, qb, 0, out=c, accumulate=acc)
    check_bf16(c, ref + c0 if acc else ref)
    inside = torch.zeros(M * ld + 2, dtype=torch.bool, device=DEV)
    inside[base:base + M * ld].view(M, ld)[:, :N] = True
    assert torch.equal(flat.view(torch.int16)[~inside], before.view(torch.int16)[~inside])


@pytest.mark.parametrize("pad,base", [(1, 0), (2, 1)])
def test_gemm_mxfp8_bf16_strided_output(q2d, pad, base):
    """The large-tile MXFP8 kernel's bf16 output into a view of a wider buffer with
    an odd row pitch or a base one element off (one store per element) equals,
    byte for byte, the same GEMM written contiguously (pair stores), with and
    without accumulation; the bytes outside the view are unchanged."""
    M, N, K = 2100, 4001, 512                       # 9 x 16 output tiles of 256 x 256
    A = synth.normal((M, K), 1.0, 41, torch.bfloat16, device=DEV)
    B = synth.normal((N, K), 0.02, 42, torch.bfloat16, device=DEV)
    qa, qb = q2d.mxfp8_quantize(A), q2d.mxfp8_quantize(B)
    ld = N + pad
    flat = synth.normal((M * ld + 2,), 0.5, 43, torch.bfloat16, device=DEV)
    before = flat.clone()
    c = flat[base:base + M * ld].view(M, ld)[:, :N]
    ref = c.contiguous()
    q2d.q2d_gemm(qa, 0, qb, 0, out=c, accumulate=True)
    q2d.q2d_gemm(qa, 0, qb, 0, out=ref, accumulate=True)
    assert torch.equal(c.contiguous().view(torch.int16), ref.view(torch.int16))
    inside = torch.zeros(M * ld + 2, dtype=torch.bool, device=DEV)
    inside[base:base + M * ld].view(M, ld)[:, :N] = True
    assert torch.equal(flat.view(torch.int16)[~inside], before.view(torch.int16)[~inside])
    q2d.q2d_gemm(qa, 0, qb, 0, out=c)
    q2d.q2d_gemm(qa, 0, qb, 0, out=ref)
    assert torch.equal(c.contiguous().view(torch.int16), ref.view(torch.int16))


def test_gemm_deterministic(q2d):
    """Two runs of each persistent-kernel GEMM (forward with bf16 output, weight
    gradient with fp32 output, the quantizing epilogue) on the same operands give
    identical bytes: no atomics, a fixed reduction order per output element."""
    T, N, K = 2048, 4096, 1024                      # 128 output tiles of 256 x 256
    X = synth.normal((T, K), 1.0, 611, torch.bfloat16, device=DEV)
    W = synth.normal((N, K), 0.02, 612, torch.bfloat16, device=DEV)
    dY = synth.normal((T, N), 1e-3, 613, torch.bfloat16, device=DEV)
    qx, qw, qdy = q2d.q2d_quantize(X, "sr", 1, 0), q2d.q2d_quantize(W, "sr", 1, 1), q2d.q2d_quantize(dY, "sr", 1, 2)
    runs = []
    for _ in range(2):
        y = torch.full((T, N), float("nan"), dtype=torch.bfloat16, device=DEV)
        dw = torch.full((N, K), float("nan"), dtype=torch.float32, device=DEV)
        q2d.q2d_gemm(qx, 0, qw, 0, out=y)
        q2d.q2d_gemm(qdy, 1, qx, 1, out=dw)
        qy = q2d.q2d_gemm_quantized(qx, 0, qw, 0, "rtn")
        torch.cuda.synchronize()
        runs.append([y.view(torch.int16).clone(), dw.view(torch.int32).clone(), qy.codes.clone(),
                     qy.codes_t.clone(), qy.scales.clone(), qy.scales_t.clone()])
    for a, b in zip(*runs):
        assert torch.equal(a, b)
    assert not torch.isnan(runs[0][0].view(torch.bfloat16)).any()


def test_gemm_accumulate_and_ldc(q2d):
    A = synth.normal((200, 320), 1.0, 1, torch.bfloat16, device=DEV)
    B = synth.normal((150, 320), 1.0, 2, torch.bfloat16, device=DEV)
    qa, oa = quant(q2d, A, "rtn")
    qb, ob = quant(q2d, B, "rtn")
    ref = oracle.gemm(oracle.operand(oa, False), oracle.operand(ob, False))
    big = torch.randn((200, 160), device=DEV, dtype=torch.float32)
    c0 = big[:, :150].clone()
    q2d.q2d_gemm(qa, 0, qb, 0, out=big[:, :150], accumulate=True)
    assert rel_frob(big[:, :150].cpu().numpy(), ref + c0.cpu().numpy().astype(np.float64)) <= TOL


def test_gemm_unit_scales_exact(q2d):
    """All scales 2^0: the GEMM is an exact integer matmul of 2 * E2M1 values."""
    rng = np.random.default_rng(4)
    g = np.array([0, .5, 1, 1.5, 2, 3, 4, 6])

    def grid(R, C):
        x = g[rng.integers(0, 8, (R, C))] * rng.choice([-1, 1], (R, C))
        x[::32, ::32] = 6.0
        return torch.from_numpy(x.astype(np.float32)).to(DEV)
    A, B = grid(256, 512), grid(192, 512)
    qa, _ = quant(q2d, A, "rtn")
    qb, _ = quant(q2d, B, "rtn")
    c = q2d.q2d_gemm(qa, 0, qb, 0).cpu().numpy().astype(np.float64)
    ai = (2 * A.cpu().numpy()).astype(np.int64)
    bi = (2 * B.cpu().numpy()).astype(np.int64)
    assert np.array_equal(c * 4, (ai @ bi.T).astype(np.float64))


@pytest.mark.parametrize("M,N,K,ta,tb", [(300, 200, 160, 0, 0), (2100, 4000, 384, 0, 1), (4096, 2048, 640, 1, 1)])
def test_gemm_non_finite_blocks(q2d, M, N, K, ta, tb):
    """A NaN and an infinity in two blocks of A give those blocks scale 0xFF (NaN):
    exactly the output entries whose dot product meets them are NaN, on the small and
    the persistent kernel, and the rest match the oracle."""
    A = synth.normal((K, M) if ta else (M, K), 1.0, 91, torch.float32)
    B = synth.normal((K, N) if tb else (N, K), 0.02, 92, torch.float32)
    A[5, 7] = float("nan")
    A[-1, -1] = float("inf")
    qa, oa = quant(q2d, A.to(DEV), "rtn")
    qb, ob = quant(q2d, B.to(DEV), "rtn")
    ref = oracle.gemm(oracle.operand(oa, bool(ta)), oracle.operand(ob, bool(tb)))
    c = q2d.q2d_gemm(qa, ta, qb, tb, out_dtype=torch.float32).cpu().numpy().astype(np.float64)
    nan = np.isnan(ref)
    assert nan.any() and not nan.all()
    assert np.array_equal(np.isnan(c), nan)
    assert rel_frob(c[~nan], ref[~nan]) <= TOL


@pytest.mark.parametrize("T,N,K", [(128, 256, 256), (96, 300, 200), (512, 1024, 768)])
def test_linear_fwd_bwd(q2d, T, N, K):
    X = synth.normal((T, K), 1.0, 1, torch.bfloat16, device=DEV)
    W = synth.normal((N, K), 0.02, 2, torch.bfloat16, device=DEV)
    dY = synth.normal((T, N), 1e-3, 3, torch.bfloat16, device=DEV)
    Y, qX, qW = q2d.q2d_linear_fwd(X, W, "sr", "sr", seed=9, offset_x=0, offset_w=1,
                                   y_dtype=torch.float32)
    dX, dW, qdY = q2d.q2d_linear_bwd(dY, qX, qW, "sr", seed=9, offset_dy=2,
                                     dx_dtype=torch.float32, dw_dtype=torch.float32)
    ox = oracle.quantize_fp4_2d(X.cpu(), "sr", 9, 0)
    ow = oracle.quantize_fp4_2d(W.cpu(), "sr", 9, 1)
    ody = oracle.quantize_fp4_2d(dY.cpu(), "sr", 9, 2)
    for name, gq, oq in (("X", qX, ox), ("W", qW, ow), ("dY", qdY, ody)):
        got = as_oracle_tensor(gq, oq["rows"], oq["cols"])
        for k in ("codes", "codes_t", "scales", "scales_t"):
            assert np.array_equal(got[k], oq[k]), (name, k)
    ref = oracle.linear(ox, ow, ody)
    assert rel_frob(Y.cpu().numpy(), ref["Y"]) <= TOL
    assert rel_frob(dX.cpu().numpy(), ref["dX"]) <= TOL
    assert rel_frob(dW.cpu().numpy(), ref["dW"]) <= TOL


@pytest.mark.parametrize("M,N,K", [(128, 256, 256), (300, 200, 160), (1000, 300, 2000),
                                   # enough 256 x 256 tiles for the large-tile kernel: ragged
                                   # edges, K shorter than its 4-stage ring (256 = 4 K-tiles of 64);
                                   # 16-byte scale groups of 8 K-tiles for K = 1024 and 1536 (an
                                   # odd number of groups), per-word scales for K = 640 and 256
                                   # (not multiples of 512)
                                   (4096, 2048, 1024), (4096, 2304, 1536), (4000, 2100, 640),
                                   (2048, 4224, 256)])
@pytest.mark.parametrize("ta,tb", [(0, 0), (0, 1), (1, 1), (1, 0)])
@pytest.mark.parametrize("data", ["normal", "adversarial"])
def test_gemm_mxfp8(q2d, M, N, K, ta, tb, data):
    """MXFP8 GEMMs within the bound derived from the measured E4M3 MFMA
    arithmetic (tests/fp8_mfma_model.py).  "adversarial" places in every
    group of 8 along K one product 2^13.2 times the seven others, which the
    instruction's 13-bit window cuts."""
    a_shape = (K, M) if ta else (M, K)
    b_shape = (K, N) if tb else (N, K)
    if data == "normal":
        A = synth.normal(a_shape, 1.0, 3 * M + K, torch.bfloat16, device=DEV)
        synth.add_outlier_channels(A, 5, frac=0.02)
        B = synth.normal(b_shape, 0.02, N + 7, torch.bfloat16, device=DEV)
    else:
        A = adversarial_k_groups(M, K, 1.75 * 2.0 ** -7, bool(ta))
        B = adversarial_k_groups(N, K, 2.0 ** -7, bool(tb))
    qa = q2d.mxfp8_quantize(A)
    qb = q2d.mxfp8_quantize(B)
    oa = oracle.quantize_mxfp8(A.cpu())
    ob = oracle.quantize_mxfp8(B.cpu())
    ga, gb = as_oracle_tensor(qa, *A.shape), as_oracle_tensor(qb, *B.shape)
    for k in ("codes", "codes_t", "scales", "scales_t"):
        assert np.array_equal(ga[k], oa[k]), k
        assert np.array_equal(gb[k], ob[k]), k
    a64 = oracle.operand(oa, bool(ta), "mxfp8")
    b64 = oracle.operand(ob, bool(tb), "mxfp8")
    ref = oracle.gemm(a64, b64)
    c = q2d.q2d_gemm(qa, ta, qb, tb, out_dtype=torch.float32).cpu().numpy().astype(np.float64)
    check_mxfp8(c, ref, oa, bool(ta), ob, bool(tb), a64, b64, adversarial=data == "adversarial")


def adversarial_k_groups(R, K, small, transpose):
    """R rows along K of 1.0 at every k % 8 == 0 and `small` elsewhere (bf16,
    stored transposed when the GEMM reads the operand's column copy)."""
    k = torch.arange(K)
    row = torch.where(k % 8 == 0, torch.tensor(1.0), torch.tensor(small)).to(torch.bfloat16)
    X = row.expand(R, K).contiguous()
    return (X.t().contiguous() if transpose else X).to(DEV)


def check_mxfp8(c, ref, oa, ta, ob, tb, a64, b64, rows=None, adversarial=False):
    """|C - C_ref| within the derived elementwise bound (fp8_mfma_model.error_bound);
    the decoding of the bound's helper equals the oracle's operands."""
    av, am = fm.operand_fields(oa, ta)
    bv, bm = fm.operand_fields(ob, tb)
    assert np.array_equal(av, a64) and np.array_equal(bv, b64)
    if rows is not None:
        av, am = av[rows], am[rows]
    bound = fm.error_bound(av, am, bv, bm)
    err = np.abs(c - ref)
    assert np.all(err <= bound), float((err / bound).max())
    if adversarial:
        # the cut products make the error exceed what random data suggests
        P = np.abs(av) @ np.abs(bv).T
        assert np.all(err > 2.0 ** -11 * P)


def _sample_rows(qt_np, trans, rows, fmt="fp4"):
    """float64 rows `rows` of op(X) from an oracle quantization."""
    if fmt == "fp4":
        codes = qt_np["codes_t" if trans else "codes"][rows]
        scales = qt_np["scales_t" if trans else "scales"]
        K = qt_np["rows"] if trans else qt_np["cols"]
        vals = oracle.fp4_values(np.stack([codes & 15, codes >> 4], -1).reshape(len(rows), -1)[:, :K])
        s = 2.0 ** (scales[np.asarray(rows) // 32][:, np.arange(K) // 32].astype(np.float64) - 127)
        return vals * s
    raise ValueError(fmt)


@pytest.mark.parametrize("name", ["dense_1b", "dense_7b", "mixed_7b"])
def test_full_launch_configuration(q2d, name):
    """Every FP4 GEMM of the 1B-class (SR on all operands), 7B-class (the benchmark's
    15) and mixed 7B-class (V, O, gate, up and down in 2D-block FP4 with SR on X,
    W and dY; its MXFP8 Q/K GEMMs have their own test) linear workloads at full
    size (bf16 Y and dX, fp32 dW), 48 sampled rows each.

    The oracle quantizes the same inputs (byte-equal to the device operands);
    the device GEMMs are compared with float64 products of the oracle's
    operands on sampled output rows."""
    w = synth.WORKLOADS[name](device=DEV)
    rng = np.random.default_rng(0)
    for lin in w.linears:
        if lin.fmt != "fp4":
            continue
        X, W, dY = w.tensors[lin.x], w.tensors[lin.w], w.tensors[lin.dy]
        Y, qX, qW = q2d.q2d_linear_fwd(X, W, w.rounding[lin.x], w.rounding[lin.w], seed=w.seed,
                                       offset_x=0, offset_w=1, y_dtype=torch.bfloat16)
        dX, dW, qdY = q2d.q2d_linear_bwd(dY, qX, qW, w.rounding[lin.dy], seed=w.seed, offset_dy=2,
                                         dx_dtype=torch.bfloat16, dw_dtype=torch.float32)
        torch.cuda.synchronize()
        ox = oracle.quantize_fp4_2d(X.cpu(), w.rounding[lin.x], w.seed, 0)
        ow = oracle.quantize_fp4_2d(W.cpu(), w.rounding[lin.w], w.seed, 1)
        ody = oracle.quantize_fp4_2d(dY.cpu(), w.rounding[lin.dy], w.seed, 2)
        for name, gq, oq in (("X", qX, ox), ("W", qW, ow), ("dY", qdY, ody)):
            assert_same_bytes(gpu_buffers(gq), oq, "%s %s %s" % (w.name, lin.name, name))
        print("%s linear %s: checking sampled rows" % (w.name, lin.name), flush=True)
        Wf = oracle.operand(ow, False)
        Wt = oracle.operand(ow, True)
        Xt = oracle.operand(ox, True)
        rows = np.sort(rng.choice(lin.tokens, 48, replace=False))
        ref_y = _sample_rows(ox, False, rows) @ Wf.T
        check_bf16(Y[torch.from_numpy(rows).to(DEV)], ref_y)
        ref_dx = _sample_rows(ody, False, rows) @ Wt.T
        check_bf16(dX[torch.from_numpy(rows).to(DEV)], ref_dx)
        rows_w = np.sort(rng.choice(lin.n_out, 48, replace=False))
        ref_dw = _sample_rows(ody, True, rows_w) @ Xt.T
        got_dw = dW[torch.from_numpy(rows_w).to(DEV)].cpu().numpy()
        assert rel_frob(got_dw, ref_dw) <= TOL
        del Y, dX, dW, qX, qW, qdY, Wf, Wt, Xt
    torch.cuda.empty_cache()


@pytest.mark.parametrize("data", ["synthetic", "adversarial"])
def test_full_mixed_7b_qk_launch_configuration(q2d, data):
    """The MXFP8 query/key GEMMs of the mixed 7B block at full size (tokens 16384,
    hidden 4096; float32 outputs), 32 sampled rows each, against float64
    products of the oracle's MXFP8 operands within the derived bound.  The
    adversarial form replaces X by rows that put one large and seven small
    values in every group of 8 along the hidden dimension."""
    w = synth.mixed_7b(device=DEV)
    rng = np.random.default_rng(2)
    X = w.tensors["X_qkv"]
    if data == "adversarial":
        X = adversarial_k_groups(X.shape[0], X.shape[1], 1.75 * 2.0 ** -7, False)
    qX = q2d.mxfp8_quantize(X)
    oX = oracle.quantize_mxfp8(X.cpu())
    assert_same_bytes(gpu_buffers(qX), oX, "X_qkv mxfp8")
    A = oracle.operand(oX, False, "mxfp8")
    Xt = oracle.operand(oX, True, "mxfp8")
    for name in ("q", "k"):
        W, dY = w.tensors["W_" + name], w.tensors["dY_" + name]
        if data == "adversarial":
            W = adversarial_k_groups(W.shape[0], W.shape[1], 2.0 ** -7, False)
        qW, qdY = q2d.mxfp8_quantize(W), q2d.mxfp8_quantize(dY)
        oW, odY = oracle.quantize_mxfp8(W.cpu()), oracle.quantize_mxfp8(dY.cpu())
        assert_same_bytes(gpu_buffers(qW), oW, "W mxfp8")
        assert_same_bytes(gpu_buffers(qdY), odY, "dY mxfp8")
        print("mixed 7B %s projection (%s): GEMMs" % (name, data), flush=True)
        Y = q2d.q2d_gemm(qX, 0, qW, 0, out_dtype=torch.float32)
        dX = q2d.q2d_gemm(qdY, 0, qW, 1, out_dtype=torch.float32)
        dW = q2d.q2d_gemm(qdY, 1, qX, 1, out_dtype=torch.float32)
        Wf, Wt = oracle.operand(oW, False, "mxfp8"), oracle.operand(oW, True, "mxfp8")
        dYf, dYt = oracle.operand(odY, False, "mxfp8"), oracle.operand(odY, True, "mxfp8")
        for what, got, (oa, ta, a), (ob, tb, b) in (
                ("Y", Y, (oX, False, A), (oW, False, Wf)),
                ("dX", dX, (odY, False, dYf), (oW, True, Wt)),
                ("dW", dW, (odY, True, dYt), (oX, True, Xt))):
            rows = np.sort(rng.choice(a.shape[0], 32, replace=False))
            ref = a[rows] @ b.T
            g = got[torch.from_numpy(rows).to(DEV)].cpu().numpy().astype(np.float64)
            check_mxfp8(g, ref, oa, ta, ob, tb, a, b, rows=rows,
                        adversarial=data == "adversarial" and what == "Y")
        del qW, qdY, Y, dX, dW
    torch.cuda.empty_cache()
