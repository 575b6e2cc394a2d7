"""Block-level pins of the oracle quantizer.

* Transposition invariance S(B_ij) = S(B_ij^T) (Sec. 3; App. D): quantizing the
  transposed view gives the other layout bit for bit; a materialised copy gives
  the same scales and round-to-nearest codes.
* Block indexing, scales and nibble layout, checked element by element against
  block maxima computed independently with numpy.
* Boundary blocks use valid entries only (App. D).
* Error bounds: |Q(x) - x| <= S * delta / 2 (nearest) and < S * delta (stochastic),
  never beyond the representable range (Sec. 3.1).
* Stochastic rounding is unbiased per element over many independent offsets.
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


def _block_max(x64, b=B):
    R, C = x64.shape
    nbr, nbc = -(-R // b), -(-C // b)
    M = np.zeros((nbr, nbc))
    for i in range(nbr):
        for j in range(nbc):
            M[i, j] = np.abs(x64[i * b:(i + 1) * b, j * b:(j + 1) * b]).max()
    return M


@pytest.mark.parametrize("shape", [(64, 96), (100, 70), (33, 129), (1, 5), (257, 31)])
@pytest.mark.parametrize("mode", ["rtn", "sr"])
def test_elementwise_definition(shape, mode):
    x = synth.normal(shape, 0.7, 11, torch.bfloat16)
    q = oracle.quantize_fp4_2d(x, mode, seed=5, offset=9)
    x64 = oracle.to_float64(x)
    R, C = shape
    e = np.vectorize(oracle.fp4_scale_exponent)(_block_max(x64)).astype(np.int64)
    lay = oracle.fp4_layout(R, C)
    assert q["codes"].shape == lay["codes"]
    np.testing.assert_array_equal(q["scales"][:, :e.shape[1]], (e + 127).astype(np.uint8))
    assert not q["scales"][:, e.shape[1]:].any()
    np.testing.assert_array_equal(q["scales_t"][:, :e.shape[0]], (e.T + 127).astype(np.uint8))
    eb = e[np.arange(R)[:, None] // B, np.arange(C)[None, :] // B]
    idx = np.arange(R)[:, None] * x.stride(0) + np.arange(C)[None, :]
    if mode == "sr":
        r16 = np.vectorize(lambda i: oracle.sr_bits(int(i), 5, 9))(idx).astype(np.uint32)
    else:
        r16 = None
    want = oracle.fp4_codes(x64, eb, mode == "sr", r16)
    got = _unpack(q["codes"], C)
    np.testing.assert_array_equal(got, want)
    assert not _unpack(q["codes"], lay["codes"][1] * 2)[:, C:].any()      # zero padding
    got_t = _unpack(q["codes_t"], R)
    np.testing.assert_array_equal(got_t, want.T)
    assert not _unpack(q["codes_t"], lay["codes_t"][1] * 2)[:, R:].any()


@pytest.mark.parametrize("mode", ["rtn", "sr"])
def test_transposed_view_swaps_layouts(mode):
    w = synth.normal((96, 160), 0.02, 3, torch.bfloat16)
    q = oracle.quantize_fp4_2d(w, mode, seed=1, offset=2)
    qt = oracle.quantize_fp4_2d(w.t(), mode, seed=1, offset=2)
    np.testing.assert_array_equal(qt["codes"], q["codes_t"][:, :qt["codes"].shape[1]])
    np.testing.assert_array_equal(qt["codes_t"][:, :q["codes"].shape[1]], q["codes"])
    sc = q["scales"][:, :5]
    np.testing.assert_array_equal(qt["scales"][:, :3], sc.T)


def test_materialised_transpose_same_scales_and_rtn():
    w = synth.normal((128, 64), 1.0, 4, torch.bfloat16)
    q = oracle.quantize_fp4_2d(w, "rtn")
    qc = oracle.quantize_fp4_2d(w.t().contiguous(), "rtn")
    np.testing.assert_array_equal(qc["scales"][:2, :4], q["scales"][:4, :2].T)
    np.testing.assert_array_equal(qc["codes"], q["codes_t"])
    a = oracle.operand(q, True)
    b = oracle.operand(qc, False)
    np.testing.assert_array_equal(a, b)


def test_boundary_block_uses_valid_entries_only():
    x = synth.normal((45, 70), 1.0, 8, torch.float32)
    x[40:, 66:] = 0.001        # the corner boundary block holds small values only
    q = oracle.quantize_fp4_2d(x, "rtn")
    sub = oracle.quantize_fp4_2d(x[32:, 64:].contiguous(), "rtn")
    assert q["scales"][1, 2] == sub["scales"][0, 0]
    np.testing.assert_array_equal(_unpack(q["codes"][32:], 70)[:, 64:], _unpack(sub["codes"], 6))


@pytest.mark.parametrize("mode", ["rtn", "sr"])
def test_error_bounds_and_no_clipping(mode):
    x = synth.normal((256, 256), 1.0, 21, torch.bfloat16)
    synth.add_outlier_channels(x, 22, frac=0.02)
    q = oracle.quantize_fp4_2d(x, mode, seed=3)
    x64 = oracle.to_float64(x)
    deq = oracle.operand(q, False)
    S = 2.0 ** (q["scales"][:8, :8].astype(np.int64) - 127)
    Sb = np.repeat(np.repeat(S, B, 0), B, 1)
    assert np.all(np.abs(x64) <= 6 * Sb)                      # truncation-free: nothing clipped
    assert np.all(np.abs(deq) <= 6 * Sb)
    v = np.abs(x64) / Sb
    delta = np.where(v < 2, 0.5, np.where(v < 4, 1.0, 2.0)) * Sb
    err = np.abs(deq - x64)
    if mode == "rtn":
        assert np.all(err <= delta / 2)
    else:
        assert np.all(err < delta)
    np.testing.assert_array_equal(oracle.operand(q, True), deq.T)     # both layouts agree


def test_sr_unbiased_per_element():
    """Mean error over 2000 offsets within 5 sigma (sigma <= delta / 2) + delta 2^-16."""
    x = synth.normal((32, 64), 1.0, 30, torch.float32)
    x64 = oracle.to_float64(x)
    n = 2000
    acc = np.zeros_like(x64)
    for off in range(n):
        acc += oracle.operand(oracle.quantize_fp4_2d(x, "sr", seed=77, offset=off), False) - x64
    mean = acc / n
    S = 2.0 ** (oracle.quantize_fp4_2d(x)["scales"][0, :2].astype(np.int64) - 127)
    Sb = np.repeat(S, B)[None, :]
    v = np.abs(x64) / Sb
    delta = np.where(v < 2, 0.5, np.where(v < 4, 1.0, 2.0)) * Sb
    assert np.all(np.abs(mean) <= 5 * (delta / 2) / np.sqrt(n) + delta * 2.0 ** -16)
    # and in aggregate the signed errors cancel: the mean over all 2048 elements is tiny
    assert abs(mean.mean()) <= 5 * (delta / 2).max() / np.sqrt(n * x64.size)


def test_non_finite_and_zero_blocks():
    x = synth.normal((64, 64), 1.0, 5, torch.float32)
    x[3, 40] = float("nan")
    x[40, 3] = float("inf")
    x[32:, 32:] = 0.0
    q = oracle.quantize_fp4_2d(x, "sr", seed=1)
    assert q["scales"][0, 1] == 0xFF and q["scales"][1, 0] == 0xFF
    assert q["scales"][1, 1] == 0x00
    u = _unpack(q["codes"], 64)
    assert not u[:32, 32:].any() and not u[32:, :32].any() and not u[32:, 32:].any()
    assert q["scales"][0, 0] not in (0x00, 0xFF) and u[:32, :32].any()


def test_grouped_segments_are_independent_matrices():
    counts = [0, 1, 31, 33, 127, 130, 64]
    off = synth.segment_offsets(counts)
    x = synth.normal((int(off[-1]), 96), 1.0, 40, torch.bfloat16)
    for mode in ("rtn", "sr"):
        g = oracle.quantize_fp4_grouped(x, off, mode, seed=2, offset=3)
        p = g["padded_rows"]
        for e in range(len(counts)):
            n = counts[e]
            if n == 0:
                continue
            seg = oracle.quantize_fp4_2d(x[off[e]:off[e + 1]], mode, seed=2, offset=3,
                                         index_base=int(off[e]) * x.stride(0))
            np.testing.assert_array_equal(g["codes"][p[e]:p[e] + n], seg["codes"])
            nb = -(-n // B)
            np.testing.assert_array_equal(g["scales"][p[e] // B:p[e] // B + nb], seg["scales"])
            rows_t = seg["codes_t"].shape[1]
            np.testing.assert_array_equal(g["codes_t"][:, p[e] // 2:p[e] // 2 + rows_t],
                                          seg["codes_t"])
            assert not g["codes"][p[e] + n:p[e + 1]].any()


# ------------------------------------------------------------------ 64 x 64 blocks (Table 4)

def _expand64(M64, nrows, ncols):
    """32-granular grid holding the byte of 64-block (i // 2, j // 2); 0 past the blocks."""
    g = np.zeros((nrows, ncols), dtype=M64.dtype)
    for i in range(nrows):
        for j in range(ncols):
            if i // 2 < M64.shape[0] and j // 2 < M64.shape[1]:
                g[i, j] = M64[i // 2, j // 2]
    return g


@pytest.mark.parametrize("shape", [(128, 192), (100, 70), (33, 129), (257, 31)])
@pytest.mark.parametrize("mode", ["rtn", "sr"])
def test_block64_elementwise_definition(shape, mode):
    x = synth.normal(shape, 0.7, 31, torch.bfloat16)
    q = oracle.quantize_fp4_2d(x, mode, seed=5, offset=9, block=64)
    x64 = oracle.to_float64(x)
    R, C = shape
    e64 = np.vectorize(oracle.fp4_scale_exponent)(_block_max(x64, 64)).astype(np.int64)
    lay = oracle.fp4_layout(R, C)
    np.testing.assert_array_equal(q["scales"], _expand64((e64 + 127).astype(np.uint8), *lay["scales"]))
    np.testing.assert_array_equal(q["scales_t"], _expand64((e64.T + 127).astype(np.uint8), *lay["scales_t"]))
    eb = e64[np.arange(R)[:, None] // 64, np.arange(C)[None, :] // 64]
    idx = np.arange(R)[:, None] * x.stride(0) + np.arange(C)[None, :]
    r16 = np.vectorize(lambda i: oracle.sr_bits(int(i), 5, 9))(idx).astype(np.uint32) if mode == "sr" else None
    want = oracle.fp4_codes(x64, eb, mode == "sr", r16)
    np.testing.assert_array_equal(_unpack(q["codes"], C), want)
    np.testing.assert_array_equal(_unpack(q["codes_t"], R), want.T)


@pytest.mark.parametrize("mode", ["rtn", "sr"])
def test_block64_transposed_view_swaps_layouts(mode):
    x = synth.normal((150, 200), 1.0, 32, torch.bfloat16)
    q = oracle.quantize_fp4_2d(x, mode, 3, 4, block=64)
    qt = oracle.quantize_fp4_2d(x.t(), mode, 3, 4, block=64)
    for a, b in (("codes", "codes_t"), ("scales", "scales_t")):
        np.testing.assert_array_equal(qt[a], q[b])
        np.testing.assert_array_equal(qt[b], q[a])


def test_block64_reduces_to_block32_when_subblock_maxima_agree():
    """If the four 32 x 32 sub-blocks of every 64 x 64 block share one maximum, both
    block sizes give the same scales and codes."""
    x = synth.normal((192, 256), 0.5, 33, torch.float32)
    x = torch.clamp(x, -3.0, 3.0)
    x[::32, ::32] = 7.0
    q32 = oracle.quantize_fp4_2d(x, "rtn")
    q64 = oracle.quantize_fp4_2d(x, "rtn", block=64)
    for k in ("codes", "codes_t", "scales", "scales_t"):
        np.testing.assert_array_equal(q64[k], q32[k])
