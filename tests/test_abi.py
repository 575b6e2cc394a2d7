"""Host-side checks of the C ABI (no GPU needed, no kernel is launched).

* libq2d.so loads and exports every function that include/q2d.h declares;
* q2d_tensor_init's layout equals the layout the oracle derives on its own;
* argument errors return their documented status before any launch.
"""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HDR = os.path.join(ROOT, "include", "q2d.h")


def declared_functions():
    text = open(HDR).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(\w+)\s*\(", text, flags=re.M)))


@pytest.fixture(scope="module")
def q2d():
    import paper_2607_24953_amd as q
    return q


def test_exports_every_declared_symbol(q2d):
    names = declared_functions()
    assert {"q2d_quantize", "q2d_gemm", "mxfp8_quantize", "q2d_linear_fwd", "q2d_linear_bwd",
            "q2d_tensor_init", "q2d_status_string", "q2d_grouped_tensor_init",
            "q2d_grouped_quantize", "q2d_grouped_gemm"} <= set(names)
    lib = ctypes.CDLL(q2d.lib_path)
    for n in names:
        assert hasattr(lib, n), n


@pytest.mark.parametrize("R,C", [(1, 1), (32, 32), (100, 70), (4096, 11008), (131, 257)])
def test_layout_matches_oracle(q2d, R, C):
    import oracle
    for fmt, lay in ((q2d.FP4_2D, oracle.fp4_layout(R, C)), (q2d.MXFP8, oracle.mxfp8_layout(R, C)),
                     (q2d.FP4_1D, oracle.fp4_1d_layout(R, C))):
        d = q2d._Tensor()
        sizes = (ctypes.c_int64 * 4)()
        assert q2d._lib.q2d_tensor_init(ctypes.byref(d), fmt, R, C, 32, sizes) == 0
        assert (d.ld_codes, d.ld_codes_t, d.ld_scales, d.ld_scales_t) == (
            lay["codes"][1], lay["codes_t"][1], lay["scales"][1], lay["scales_t"][1])
        for i, k in enumerate(("codes", "codes_t", "scales", "scales_t")):
            assert sizes[i] == lay[k][0] * lay[k][1]


def test_error_paths(q2d):
    L = q2d._lib
    d = q2d._Tensor()
    sizes = (ctypes.c_int64 * 4)()
    assert L.q2d_tensor_init(ctypes.byref(d), 0, 0, 5, 32, sizes) == 1
    assert L.q2d_tensor_init(ctypes.byref(d), 0, 5, 5, 16, sizes) == 2
    assert L.q2d_tensor_init(ctypes.byref(d), 7, 5, 5, 32, sizes) == 1
    assert L.q2d_tensor_init(None, 0, 5, 5, 32, sizes) == 1
    # extents beyond 2^31 (their layout products would overflow int64) are unsupported
    for huge in (2 ** 31 + 1, 2 ** 62, 2 ** 63 - 1):
        assert L.q2d_tensor_init(ctypes.byref(d), 0, huge, 64, 32, sizes) == 2
        assert L.q2d_tensor_init(ctypes.byref(d), 2, 64, huge, 32, sizes) == 2
        assert L.q2d_grouped_tensor_init(ctypes.byref(d), huge, 64, 4, 32, sizes) == 2
    assert L.q2d_tensor_init(ctypes.byref(d), 0, 64, 64, 32, sizes) == 0
    fake = 0x1000
    # no buffers attached
    assert L.q2d_quantize(fake, 1, 64, 64, 64, 1, 32, 0, 0, 0, ctypes.byref(d), None) == 1
    d.codes, d.scales = fake, fake
    d.codes_t, d.scales_t = fake, fake
    # null input, bad dtype, bad shape vs descriptor, bad strides, bad mode, bad block
    assert L.q2d_quantize(None, 1, 64, 64, 64, 1, 32, 0, 0, 0, ctypes.byref(d), None) == 1
    assert L.q2d_quantize(fake, 5, 64, 64, 64, 1, 32, 0, 0, 0, ctypes.byref(d), None) == 1
    assert L.q2d_quantize(fake, 1, 65, 64, 64, 1, 32, 0, 0, 0, ctypes.byref(d), None) == 1
    assert L.q2d_quantize(fake, 1, 64, 64, 0, 1, 32, 0, 0, 0, ctypes.byref(d), None) == 1
    assert L.q2d_quantize(fake, 1, 64, 64, 64, 1, 32, 9, 0, 0, ctypes.byref(d), None) == 1
    assert L.q2d_quantize(fake, 1, 64, 64, 64, 1, 32, 0x12, 0, 0, ctypes.byref(d), None) == 1  # flag + bad mode
    assert L.q2d_quantize(fake, 1, 64, 64, 64, 1, 32, 0x30, 0, 0, ctypes.byref(d), None) == 1  # unknown flag
    assert L.q2d_quantize(fake, 1, 64, 64, 64, 1, 16, 0, 0, 0, ctypes.byref(d), None) == 2
    assert L.q2d_quantize(fake, 1, 64, 64, 64, 1, 64, 0, 0, 0, ctypes.byref(d), None) == 1   # != out->block
    assert L.q2d_quantize(fake + 1, 1, 64, 64, 64, 1, 32, 0, 0, 0, ctypes.byref(d), None) == 1
    # misaligned code buffer and too-small leading dimension
    d.codes = fake + 8
    assert L.q2d_quantize(fake, 1, 64, 64, 64, 1, 32, 0, 0, 0, ctypes.byref(d), None) == 1
    d.codes = fake
    d.ld_codes = 16
    assert L.q2d_quantize(fake, 1, 64, 64, 64, 1, 32, 0, 0, 0, ctypes.byref(d), None) == 1
    d.ld_codes = 64
    # GEMM: K mismatch, bad flags, null output, ldc < N, fmt mismatch
    e = q2d._Tensor()
    assert L.q2d_tensor_init(ctypes.byref(e), 0, 64, 96, 32, sizes) == 0
    e.codes, e.scales, e.codes_t, e.scales_t = fake, fake, fake, fake
    assert L.q2d_gemm(ctypes.byref(d), 0, ctypes.byref(e), 0, fake, 0, 64, 0, None) == 1
    assert L.q2d_gemm(ctypes.byref(d), 2, ctypes.byref(d), 0, fake, 0, 64, 0, None) == 1
    assert L.q2d_gemm(ctypes.byref(d), 0, ctypes.byref(d), 0, None, 0, 64, 0, None) == 1
    assert L.q2d_gemm(ctypes.byref(d), 0, ctypes.byref(d), 0, fake, 0, 63, 0, None) == 1
    assert L.q2d_gemm(ctypes.byref(d), 0, ctypes.byref(d), 0, fake, 0, 64, 3, None) == 1
    f = q2d._Tensor()
    assert L.q2d_tensor_init(ctypes.byref(f), 1, 64, 64, 32, sizes) == 0
    f.codes, f.scales, f.codes_t, f.scales_t = fake, fake, fake, fake
    assert L.q2d_gemm(ctypes.byref(d), 0, ctypes.byref(f), 0, fake, 0, 64, 0, None) == 1
    # 1D FP4: the quantizer takes only FP4_1D descriptors and the 2D one only FP4_2D;
    # a 1D operand pairs with 2D FP4 in a GEMM but not with MXFP8
    h = q2d._Tensor()
    assert L.q2d_tensor_init(ctypes.byref(h), 2, 64, 64, 32, sizes) == 0
    assert L.q2d_quantize_1d(fake, 1, 64, 64, 64, 1, 32, 0, 0, 0, ctypes.byref(h), None) == 1   # no buffers
    h.codes, h.scales, h.codes_t, h.scales_t = fake, fake, fake, fake
    assert L.q2d_quantize_1d(fake, 1, 64, 64, 64, 1, 32, 0, 0, 0, ctypes.byref(d), None) == 1   # 2D descriptor
    assert L.q2d_quantize(fake, 1, 64, 64, 64, 1, 32, 0, 0, 0, ctypes.byref(h), None) == 1      # 1D descriptor
    assert L.q2d_quantize_1d(fake, 1, 64, 64, 64, 1, 64, 0, 0, 0, ctypes.byref(h), None) == 2
    assert L.q2d_quantize_1d(fake, 1, 64, 64, 64, 1, 32, 9, 0, 0, ctypes.byref(h), None) == 1
    assert L.q2d_quantize_1d(fake, 1, 64, 64, 64, 1, 32, 0x10, 0, 0, ctypes.byref(h), None) == 2  # floor rule: 2D only
    assert L.q2d_gemm(ctypes.byref(h), 0, ctypes.byref(f), 0, fake, 0, 64, 0, None) == 1
    assert L.q2d_gemm(ctypes.byref(f), 0, ctypes.byref(h), 0, fake, 0, 64, 0, None) == 1
    assert q2d.q2d_status_string(2) == "unsupported configuration"


def test_block64_descriptors(q2d):
    """64 x 64 blocks: FP4_2D only, the block-32 layout (32-granular scale grids);
    the quantizer needs the descriptor's block; 1D and grouped stay at 32."""
    import oracle
    L = q2d._lib
    sizes = (ctypes.c_int64 * 4)()
    fake = 0x1000
    d = q2d._Tensor()
    for R, C in ((100, 70), (4096, 11008)):
        assert L.q2d_tensor_init(ctypes.byref(d), 0, R, C, 64, sizes) == 0
        lay = oracle.fp4_layout(R, C)
        assert d.block == 64 and (d.ld_codes, d.ld_codes_t, d.ld_scales, d.ld_scales_t) == (
            lay["codes"][1], lay["codes_t"][1], lay["scales"][1], lay["scales_t"][1])
    assert L.q2d_tensor_init(ctypes.byref(d), 1, 64, 64, 64, sizes) == 2    # MXFP8
    assert L.q2d_tensor_init(ctypes.byref(d), 2, 64, 64, 64, sizes) == 2    # FP4_1D
    assert L.q2d_tensor_init(ctypes.byref(d), 0, 64, 64, 128, sizes) == 2
    assert L.q2d_grouped_tensor_init(ctypes.byref(d), 300, 64, 4, 64, sizes) == 2
    assert L.q2d_tensor_init(ctypes.byref(d), 0, 64, 64, 64, sizes) == 0
    d.codes, d.scales, d.codes_t, d.scales_t = fake, fake, fake, fake
    assert L.q2d_quantize(fake, 1, 64, 64, 64, 1, 32, 0, 0, 0, ctypes.byref(d), None) == 1   # != out->block
    assert L.q2d_quantize_1d(fake, 1, 64, 64, 64, 1, 64, 0, 0, 0, ctypes.byref(d), None) == 2
    # a block-64 operand is no MXFP8 partner
    f = q2d._Tensor()
    assert L.q2d_tensor_init(ctypes.byref(f), 1, 64, 64, 32, sizes) == 0
    f.codes, f.scales, f.codes_t, f.scales_t = fake, fake, fake, fake
    assert L.q2d_gemm(ctypes.byref(d), 0, ctypes.byref(f), 0, fake, 0, 64, 0, None) == 1


def test_gemm_quantized_error_paths(q2d):
    L = q2d._lib
    sizes = (ctypes.c_int64 * 4)()
    fake = 0x1000
    def t(fmt, R, C, block=32, bufs=True):
        d = q2d._Tensor()
        assert L.q2d_tensor_init(ctypes.byref(d), fmt, R, C, block, sizes) == 0
        if bufs:
            d.codes, d.scales, d.codes_t, d.scales_t = fake, fake, fake, fake
        return d
    a, b, out = t(0, 64, 96), t(0, 128, 96), t(0, 64, 128)
    P = ctypes.byref
    Q = lambda A, ta, B, tb, mode, o: L.q2d_gemm_quantized(A, ta, B, tb, mode, 0, 0, o, None)
    b130 = t(0, 130, 96)
    assert Q(P(a), 0, P(b130), 0, 1, P(t(0, 64, 130))) == 2                # SR needs N % 8 == 0
    assert Q(P(a), 0, P(b), 0, 5, P(out)) == 1                             # bad mode
    assert Q(None, 0, P(b), 0, 0, P(out)) == 1
    assert Q(P(a), 0, P(b), 0, 0, None) == 1
    assert Q(P(a), 0, P(b), 0, 0, P(t(0, 64, 127))) == 1                   # shape
    assert Q(P(a), 0, P(b), 0, 0, P(t(0, 64, 128, 64))) == 2               # block 64 output
    assert Q(P(a), 0, P(b), 0, 0, P(t(2, 64, 128))) == 1                   # 1D output
    assert Q(P(t(1, 64, 96)), 0, P(t(1, 128, 96)), 0, 0, P(out)) == 2      # MXFP8
    nt = t(0, 64, 128)
    nt.codes_t, nt.scales_t = None, None
    assert Q(P(a), 0, P(b), 0, 0, P(nt)) == 1                              # both orientations needed
    assert Q(P(a), 0, P(b), 1, 0, P(out)) == 1                             # K mismatch


def test_dequantize_error_paths(q2d):
    L = q2d._lib
    sizes = (ctypes.c_int64 * 4)()
    fake = 0x1000
    d = q2d._Tensor()
    assert L.q2d_tensor_init(ctypes.byref(d), 0, 64, 96, 32, sizes) == 0
    assert L.q2d_dequantize(ctypes.byref(d), 0, fake, 0, 96, None, 0, None) == 1     # no buffers
    d.codes, d.scales = fake, fake
    assert L.q2d_dequantize(ctypes.byref(d), 1, fake, 0, 96, None, 0, None) == 1     # no codes_t
    assert L.q2d_dequantize(None, 0, fake, 0, 96, None, 0, None) == 1
    assert L.q2d_dequantize(ctypes.byref(d), 2, fake, 0, 96, None, 0, None) == 1     # copy
    assert L.q2d_dequantize(ctypes.byref(d), 0, None, 0, 96, None, 0, None) == 1     # out
    assert L.q2d_dequantize(ctypes.byref(d), 0, fake, 3, 96, None, 0, None) == 1     # dtype
    assert L.q2d_dequantize(ctypes.byref(d), 0, fake, 0, 95, None, 0, None) == 1     # ldo < cols
    assert L.q2d_dequantize(ctypes.byref(d), 0, fake, 0, 96, fake, 90, None) == 1    # lde < cols
    d.ld_codes = 16
    assert L.q2d_dequantize(ctypes.byref(d), 0, fake, 0, 96, None, 0, None) == 1     # ld below layout
    d.block = 16
    assert L.q2d_dequantize(ctypes.byref(d), 0, fake, 0, 96, None, 0, None) == 2


@pytest.mark.parametrize("counts,C", [([0, 1, 31, 33, 127, 130], 96), ([256], 128),
                                      ([5] * 1024, 200), ([0, 0, 0], 32)])
def test_grouped_layout_holds_oracle_layout(q2d, counts, C):
    """The grouped capacity covers every padded segment the oracle lays out."""
    import oracle
    import synth
    off = synth.segment_offsets(counts)
    lay = oracle.fp4_grouped_layout(off, C)
    P = int(oracle.grouped_rows(off)[-1])
    S, E = int(off[-1]), len(counts)
    d = q2d._Tensor()
    sizes = (ctypes.c_int64 * 4)()
    st = q2d._lib.q2d_grouped_tensor_init(ctypes.byref(d), S, C, E, 32, sizes)
    if S == 0:
        assert st == 1
        return
    assert st == 0
    assert d.rows >= P and d.rows % 128 == 0 and d.cols == C
    assert d.ld_codes == lay["codes"][1] and d.ld_scales == lay["scales"][1]
    assert d.ld_codes_t >= lay["codes_t"][1] and d.ld_scales_t >= lay["scales_t"][1]


def test_grouped_error_paths(q2d):
    L = q2d._lib
    sizes = (ctypes.c_int64 * 4)()
    fake = 0x1000
    g = q2d._Tensor()
    assert L.q2d_grouped_tensor_init(ctypes.byref(g), 300, 64, 0, 32, sizes) == 1
    assert L.q2d_grouped_tensor_init(ctypes.byref(g), 300, 64, 1025, 32, sizes) == 1
    assert L.q2d_grouped_tensor_init(ctypes.byref(g), 300, 64, 4, 16, sizes) == 2
    assert L.q2d_grouped_tensor_init(ctypes.byref(g), 300, 64, 4, 32, sizes) == 0
    g.codes, g.scales, g.codes_t, g.scales_t = fake, fake, fake, fake
    Q = L.q2d_grouped_quantize
    ok = (fake, 1, 300, 64, 64, 4, fake, 32, 0, 0, 0, ctypes.byref(g), None)

    def call(**kw):
        names = ("x", "dt", "rows", "cols", "ld", "nseg", "off", "block", "mode", "seed",
                 "offset", "out", "stream")
        args = dict(zip(names, ok))
        args.update(kw)
        return Q(*[args[n] for n in names])

    assert call(off=None) == 1                # no segment offsets
    assert call(nseg=0) == 1 and call(nseg=1025) == 1
    assert call(off=fake + 4) == 1            # misaligned offsets
    assert call(nseg=5) == 1                  # capacity of another segment count
    assert call(rows=400) == 1                # capacity of another row count
    assert call(ld=32) == 1                   # row stride below cols
    assert call(mode=7) == 1 and call(block=64) == 2
    G = L.q2d_grouped_gemm
    w = q2d._Tensor()
    assert L.q2d_tensor_init(ctypes.byref(w), 0, 4 * 96, 64, 32, sizes) == 0
    w.codes, w.scales, w.codes_t, w.scales_t = fake, fake, fake, fake
    A, B = ctypes.byref(g), ctypes.byref(w)
    assert G(A, 0, B, 0, 4, None, 300, fake, 0, 96, 0, None) == 1       # no offsets
    assert G(A, 0, B, 0, 4, fake, 300, fake, 0, 95, 0, None) == 1       # ldc < N
    assert G(A, 0, B, 0, 4, fake, 400, fake, 0, 96, 0, None) == 1       # capacity mismatch
    w3 = q2d._Tensor()
    assert L.q2d_tensor_init(ctypes.byref(w3), 0, 4 * 96 + 1, 64, 32, sizes) == 0
    w3.codes, w3.scales = fake, fake
    assert G(A, 0, ctypes.byref(w3), 0, 4, fake, 300, fake, 0, 128, 0, None) == 1  # rows % nseg
    assert G(A, 2, B, 0, 4, fake, 300, fake, 0, 96, 0, None) == 1       # bad flag
    assert G(A, 1, B, 0, 4, fake, 300, fake, 0, 96, 0, None) == 1       # ragged K needs transB
    w2 = q2d._Tensor()
    assert L.q2d_tensor_init(ctypes.byref(w2), 0, 4 * 80, 64, 32, sizes) == 0
    w2.codes, w2.scales = fake, fake
    assert G(A, 0, ctypes.byref(w2), 0, 4, fake, 300, fake, 0, 80, 0, None) == 2  # N % 32
    m = q2d._Tensor()
    assert L.q2d_tensor_init(ctypes.byref(m), 1, 4 * 96, 64, 32, sizes) == 0
    m.codes, m.scales = fake, fake
    assert G(A, 0, ctypes.byref(m), 0, 4, fake, 300, fake, 0, 96, 0, None) == 2   # MXFP8


def test_binding_refuses_host_buffers(q2d):
    """Host tensors never reach a kernel: descriptors and outputs must be on the GPU
    (checked before any launch, so this runs without one)."""
    import torch
    cpu_q = q2d.QTensor(q2d.FP4_2D, 64, 96, "cpu")
    with pytest.raises(q2d.Q2DError):
        q2d.q2d_gemm(cpu_q, 0, cpu_q, 1)
    with pytest.raises(q2d.Q2DError):
        q2d.q2d_gemm_quantized(cpu_q, 0, cpu_q, 1)
    with pytest.raises(q2d.Q2DError):
        q2d.q2d_dequantize(cpu_q, 0)
    with pytest.raises(q2d.Q2DError):
        q2d.q2d_quantize(torch.zeros(64, 96))
