"""GPU parity of q2d_dequantize (the forward and backward copies X_fwd, X_bwd of
Sec. 2 and the maps of Fig. 1) against the oracle.

Bit-exact: float32 output equal to the oracle's float64 value rounded to float32
(exact except outside float32's range), bfloat16 output equal to its
round-to-nearest-even, NaN exactly where the oracle has NaN, and the int8
exponent maps equal, for 2D blocks (32 and 64), 1D blocks and MXFP8, both
copies, ragged shapes, every bf16 value under extreme and ordinary scales,
non-finite blocks, padded and misaligned outputs.  Then the paper's claim on
the full-size 7B tensors: the two 2D copies are identical, the 1D copies are
not.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from helpers import assert_same_bytes, gpu_buffers

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
FMTS = ["fp4", "fp4_b64", "fp4_1d", "mxfp8"]


@pytest.fixture(scope="module")
def q2d():
    import paper_2607_24953_amd as q
    return q


def quantize_both(q2d, x, fmt, mode="rtn", seed=0, offset=0):
    """Device and oracle quantization of x (bytes checked equal)."""
    if fmt == "mxfp8":
        q, o = q2d.mxfp8_quantize(x), oracle.quantize_mxfp8(x.cpu())
    elif fmt == "fp4_1d":
        q, o = q2d.q2d_quantize_1d(x, mode, seed, offset), oracle.quantize_fp4_1d(x.cpu(), mode, seed, offset)
    else:
        blk = 64 if fmt == "fp4_b64" else 32
        q = q2d.q2d_quantize(x, mode, seed, offset, block=blk)
        o = oracle.quantize_fp4_2d(x.cpu(), mode, seed, offset, block=blk)
    assert_same_bytes(gpu_buffers(q), o, "quantize %s" % fmt)
    return q, o


def _ofmt(fmt):
    return "fp4" if fmt == "fp4_b64" else fmt


def check_copy(q2d, q, o, fmt, copy, dtype, label, out=None):
    got, ex = q2d.q2d_dequantize(q, copy, dtype, exps=True, out=out)
    torch.cuda.synchronize()
    want = oracle.dequantize(o, copy, _ofmt(fmt))
    with np.errstate(over="ignore"):
        w32 = want.astype(np.float32)
    nan = np.isnan(w32)
    if dtype == torch.float32:
        g = got.cpu().numpy()
        assert np.array_equal(np.isnan(g), nan), label
        gb, wb = g.view(np.uint32), w32.view(np.uint32)
    else:
        g = got.cpu()
        assert np.array_equal(torch.isnan(g.float()).numpy(), nan), label
        gb = g.view(torch.int16).numpy()
        wb = torch.from_numpy(w32).to(torch.bfloat16).view(torch.int16).numpy()
    bad = (gb != wb) & ~nan
    if bad.any():
        r, c = np.argwhere(bad)[0]
        raise AssertionError("%s: %d values differ, first (%d, %d): gpu %r oracle %r"
                             % (label, bad.sum(), r, c, got[r, c].item(), want[r, c]))
    assert np.array_equal(ex.cpu().numpy().astype(np.int64), oracle.scale_exponents(o, copy, _ofmt(fmt))), label


SHAPES = [(128, 256), (100, 70), (33, 129), (1, 5), (257, 31), (300, 1000)]


@pytest.mark.parametrize("shape", SHAPES)
@pytest.mark.parametrize("fmt", FMTS)
def test_dequantize(q2d, shape, fmt):
    x = synth.normal(shape, 1.0, 900 + shape[0], torch.bfloat16, device=DEV)
    synth.add_outlier_channels(x, 9, frac=0.03)
    q, o = quantize_both(q2d, x, fmt, "sr" if fmt != "mxfp8" else "rtn", 4, 7)
    for copy in (0, 1):
        for dt in (torch.float32, torch.bfloat16):
            check_copy(q2d, q, o, fmt, copy, dt, "%s %s copy %d %s" % (shape, fmt, copy, dt))


def _every_value_matrix(exponents):
    """64 x n blocks of every finite bf16 value with |x| <= 6 * 2^e (both signs),
    each 32 x 32 block topped by 6 * 2^e, so each 2D, row and column block meets an
    extreme scale."""
    pos = (np.arange(0x7F80, dtype=np.uint32) << 16).view(np.float32)
    cols = []
    for e in exponents:
        top = np.float32(6.0 * 2.0 ** e)
        vals = pos[pos <= top]
        vals = np.concatenate([vals, -vals])
        n = -(-len(vals) // (64 * 32)) * 32
        flat = np.zeros(64 * n, dtype=np.float32)
        flat[:len(vals)] = vals
        blk = flat.reshape(64, n)
        blk[::32, ::32] = top
        blk[:, ::32] = top
        blk[::32, :] = top
        cols.append(blk)
    return torch.from_numpy(np.concatenate(cols, axis=1)).to(torch.bfloat16)


@pytest.mark.parametrize("fmt", FMTS)
def test_dequantize_extreme_scales(q2d, fmt):
    x = _every_value_matrix([-127, -126, -100, -3, 0, 5, 60, 124, 125]).to(DEV)
    q, o = quantize_both(q2d, x, fmt)
    for copy in (0, 1):
        for dt in (torch.float32, torch.bfloat16):
            check_copy(q2d, q, o, fmt, copy, dt, "extreme %s copy %d %s" % (fmt, copy, dt))


@pytest.mark.parametrize("fmt", FMTS)
def test_dequantize_non_finite_and_largest(q2d, fmt):
    x = synth.normal((96, 160), 1.0, 901, torch.float32)
    x[3, 40] = float("nan")
    x[50, 7] = float("inf")
    x[70, 100] = 3.0e38                        # rounds beyond float32 range in the output
    x[90, 150] = -3.3e38
    x[64:96, 128:160] = 0.0
    q, o = quantize_both(q2d, x.to(DEV), fmt)
    for copy in (0, 1):
        for dt in (torch.float32, torch.bfloat16):
            check_copy(q2d, q, o, fmt, copy, dt, "special %s copy %d %s" % (fmt, copy, dt))


def test_dequantize_padded_and_misaligned_output(q2d):
    x = synth.normal((130, 200), 1.0, 902, torch.bfloat16, device=DEV)
    for fmt in ("fp4", "fp4_1d", "mxfp8"):
        q, o = quantize_both(q2d, x, fmt)
        for dt in (torch.float32, torch.bfloat16):
            big = torch.full((130, 211), 7.0, dtype=dt, device=DEV)
            out = big[:, 1:201]                    # ldo 211, start misaligned for vector stores
            check_copy(q2d, q, o, fmt, 1, dt, "strided %s %s" % (fmt, dt), out=out)
            assert (big[:, 0] == 7).all() and (big[:, 201:] == 7).all()


def test_fig1_full_size_7b(q2d):
    """Forward/backward consistency (Fig. 1) on the 7B-class QKV input and weight:
    the 2D copies agree bit for bit (values and scales), the 1D copies do not."""
    x = synth.add_outlier_channels(synth.normal((16384, 4096), 1.0, 3021, torch.bfloat16, device=DEV), 3022)
    w = synth.normal((12288, 4096), 0.02, 3023, torch.bfloat16, device=DEV)
    for name, t in (("X", x), ("W", w)):
        print("fig1 %s %s" % (name, tuple(t.shape)), flush=True)
        q2 = q2d.q2d_quantize(t, "rtn")
        v0, e0 = q2d.q2d_dequantize(q2, 0, exps=True)
        v1, e1 = q2d.q2d_dequantize(q2, 1, exps=True)
        assert torch.equal(e0, e1) and torch.equal(v0.view(torch.int32), v1.view(torch.int32))
        q1 = q2d.q2d_quantize_1d(t, "rtn")
        v0, e0 = q2d.q2d_dequantize(q1, 0, exps=True)
        v1, e1 = q2d.q2d_dequantize(q1, 1, exps=True)
        assert (e0 != e1).any() and (v0 != v1).any()
        # round to nearest with equal scales gives equal values
        same = e0 == e1
        assert torch.equal(v0[same], v1[same])
        del q2, q1, v0, v1, e0, e1
    torch.cuda.empty_cache()


@pytest.mark.parametrize("fmt", ["fp4_2d", "fp4_2d_b64", "fp4_1d", "mxfp8"])
def test_consistency_report(q2d, fmt):
    """The Fig. 1 statistics of the consistency report against the same statistics
    of the oracle's two dequantized copies."""
    from paper_2607_24953_amd.consistency import transposition_consistency
    x = synth.add_outlier_channels(synth.normal((300, 520), 1.0, 903, torch.bfloat16), 904, frac=0.03)
    r = transposition_consistency(x.to(DEV), fmt, window=40)
    if fmt == "mxfp8":
        o, of = oracle.quantize_mxfp8(x), "mxfp8"
    elif fmt == "fp4_1d":
        o, of = oracle.quantize_fp4_1d(x, "rtn"), "fp4_1d"
    else:
        o, of = oracle.quantize_fp4_2d(x, "rtn", block=64 if fmt.endswith("b64") else 32), "fp4"
    v0, v1 = oracle.dequantize(o, 0, of), oracle.dequantize(o, 1, of)
    de = oracle.scale_exponents(o, 0, of) - oracle.scale_exponents(o, 1, of)
    x64 = oracle.to_float64(x)
    n = x64.size
    assert r["scale_mismatch_fraction"] == np.count_nonzero(de) / n
    assert r["scale_diff_max_abs"] == np.abs(de).max()
    assert r["values_differ_fraction"] == np.count_nonzero(v0 != v1) / n
    assert r["deviation_max_abs"] == np.abs(v0 - v1).max()
    assert abs(r["deviation_rel_frobenius"] - np.linalg.norm(v0 - v1) / np.linalg.norm(x64)) <= 1e-12
    assert np.array_equal(r["maps"]["scale_diff"].numpy(), de[:40, :40])
    if fmt.startswith("fp4_2d"):
        assert r["scale_mismatch_fraction"] == 0 and r["deviation_rel_frobenius"] == 0
    else:
        assert r["scale_mismatch_fraction"] > 0 and r["deviation_rel_frobenius"] > 0
