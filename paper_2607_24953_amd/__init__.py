"""Python binding of libq2d (argument marshalling only).

Every step of the quantization and GEMM path runs in the HIP kernels of
``libq2d.so``; this module allocates output buffers with PyTorch, passes raw
device pointers and the current HIP stream through the C ABI declared in
``include/q2d.h``, and turns status codes into exceptions.  There is no CPU
fallback: importing this package without the built library raises.
"""
from __future__ import annotations

import ctypes
import os

import torch

__all__ = [
    "Q2DError", "QTensor", "RTN", "SR", "FLOOR_SCALE", "FP4_2D", "MXFP8", "FP4_1D", "lib_path",
    "q2d_tensor_init", "q2d_quantize", "q2d_quantize_1d", "mxfp8_quantize", "q2d_gemm",
    "q2d_linear_fwd", "q2d_linear_bwd", "q2d_grouped_tensor_init", "q2d_grouped_quantize",
    "q2d_grouped_gemm", "q2d_dequantize", "q2d_gemm_quantized", "q2d_status_string",
]

_HERE = os.path.dirname(os.path.abspath(__file__))
lib_path = os.path.join(_HERE, "libq2d.so")

RTN, SR = 0, 1
FP4_2D, MXFP8, FP4_1D = 0, 1, 2
_F32, _BF16 = 0, 1
FLOOR_SCALE = 0x10        # scale rule of the truncation-free ablation (2D FP4 only)
_ROUND = {"rtn": RTN, "sr": SR, RTN: RTN, SR: SR,
          "rtn-floor": RTN | FLOOR_SCALE, "sr-floor": SR | FLOOR_SCALE,
          RTN | FLOOR_SCALE: RTN | FLOOR_SCALE, SR | FLOOR_SCALE: SR | FLOOR_SCALE}


class Q2DError(RuntimeError):
    pass


class _Tensor(ctypes.Structure):
    _fields_ = [("fmt", ctypes.c_int32), ("block", ctypes.c_int32),
                ("rows", ctypes.c_int64), ("cols", ctypes.c_int64),
                ("codes", ctypes.c_void_p), ("ld_codes", ctypes.c_int64),
                ("codes_t", ctypes.c_void_p), ("ld_codes_t", ctypes.c_int64),
                ("scales", ctypes.c_void_p), ("ld_scales", ctypes.c_int64),
                ("scales_t", ctypes.c_void_p), ("ld_scales_t", ctypes.c_int64)]


def _load():
    if not os.path.exists(lib_path):
        raise ImportError("libq2d.so is not built (run __graft_entry__.build()): " + lib_path)
    L = ctypes.CDLL(lib_path)
    P, I64, I32, U64 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_uint64
    TP = ctypes.POINTER(_Tensor)
    L.q2d_tensor_init.argtypes = [TP, I32, I64, I64, I32, ctypes.POINTER(ctypes.c_int64)]
    L.q2d_quantize.argtypes = [P, I32, I64, I64, I64, I64, I32, I32, U64, U64, TP, P]
    L.q2d_quantize_1d.argtypes = [P, I32, I64, I64, I64, I64, I32, I32, U64, U64, TP, P]
    L.mxfp8_quantize.argtypes = [P, I32, I64, I64, I64, I64, TP, P]
    L.q2d_gemm.argtypes = [TP, I32, TP, I32, P, I32, I64, I32, P]
    L.q2d_linear_fwd.argtypes = [P, P, I32, I64, I64, I64, I32, I32, U64, U64, U64, TP, TP, P, I32, P]
    L.q2d_linear_bwd.argtypes = [P, I32, TP, TP, I32, U64, U64, TP, P, I32, P, I32, I32, P]
    L.q2d_grouped_tensor_init.argtypes = [TP, I64, I64, I32, I32, ctypes.POINTER(ctypes.c_int64)]
    L.q2d_grouped_quantize.argtypes = [P, I32, I64, I64, I64, I32, P, I32, I32, U64, U64, TP, P]
    L.q2d_grouped_gemm.argtypes = [TP, I32, TP, I32, I32, P, I64, P, I32, I64, I32, P]
    L.q2d_dequantize.argtypes = [TP, I32, P, I32, I64, P, I64, P]
    L.q2d_gemm_quantized.argtypes = [TP, I32, TP, I32, I32, U64, U64, TP, P]
    L.q2d_status_string.argtypes = [I32]
    L.q2d_status_string.restype = ctypes.c_char_p
    for name in ("q2d_tensor_init", "q2d_quantize", "mxfp8_quantize", "q2d_gemm",
                 "q2d_linear_fwd", "q2d_linear_bwd", "q2d_grouped_tensor_init",
                 "q2d_grouped_quantize", "q2d_grouped_gemm", "q2d_quantize_1d", "q2d_dequantize",
                 "q2d_gemm_quantized"):
        getattr(L, name).restype = I32
    return L


_lib = _load()


def q2d_status_string(status: int) -> str:
    return _lib.q2d_status_string(int(status)).decode()


def _check(status: int, what: str):
    if status != 0:
        raise Q2DError("%s: %s (status %d)" % (what, q2d_status_string(status), status))


def _stream(device) -> ctypes.c_void_p:
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _dtype_code(t: torch.dtype) -> int:
    if t == torch.float32:
        return _F32
    if t == torch.bfloat16:
        return _BF16
    raise Q2DError("unsupported dtype %s (float32 or bfloat16)" % t)


class QTensor:
    """A quantized matrix in both orientations (device buffers + C descriptor).

    ``codes``/``scales`` hold the row-major copy, ``codes_t``/``scales_t`` the
    transposed one; each is a 2-D uint8 tensor of shape (rows, leading dim).

    With ``nseg`` set it is the padded grouped form of ``rows`` rows cut into
    ``nseg`` segments: ``rows`` is then the padded capacity and
    ``total_rows`` the number of input rows."""

    def __init__(self, fmt: int, rows: int, cols: int, device, block: int = 32,
                 orientations=(True, True), nseg: int | None = None):
        self.desc = _Tensor()
        sizes = (ctypes.c_int64 * 4)()
        if nseg is None:
            _check(_lib.q2d_tensor_init(ctypes.byref(self.desc), fmt, rows, cols, block, sizes),
                   "q2d_tensor_init")
        else:
            if fmt != FP4_2D:
                raise Q2DError("grouped tensors are 2D-block FP4 only")
            _check(_lib.q2d_grouped_tensor_init(ctypes.byref(self.desc), rows, cols, nseg, block,
                                                sizes), "q2d_grouped_tensor_init")
        d = self.desc
        self.fmt, self.rows, self.cols, self.device = fmt, d.rows, cols, torch.device(device)
        self.total_rows, self.nseg = rows, nseg
        shapes = {"codes": (sizes[0] // d.ld_codes, d.ld_codes),
                  "codes_t": (sizes[1] // d.ld_codes_t, d.ld_codes_t),
                  "scales": (sizes[2] // d.ld_scales, d.ld_scales),
                  "scales_t": (sizes[3] // d.ld_scales_t, d.ld_scales_t)}
        want = {"codes": orientations[0], "scales": orientations[0],
                "codes_t": orientations[1], "scales_t": orientations[1]}
        for k, shp in shapes.items():
            t = torch.empty(shp, dtype=torch.uint8, device=self.device) if want[k] else None
            setattr(self, k, t)
            setattr(d, k, t.data_ptr() if t is not None else None)

    def ptr(self):
        return ctypes.byref(self.desc)


def q2d_tensor_init(fmt: int, rows: int, cols: int, device, block: int = 32) -> QTensor:
    return QTensor(fmt, rows, cols, device, block)


def _check_input(x: torch.Tensor):
    if not x.is_cuda or x.dim() != 2:
        raise Q2DError("expected a 2-D device tensor")


def _norm(device) -> torch.device:
    d = torch.device(device)
    if d.type == "cuda" and d.index is None:
        d = torch.device("cuda", torch.cuda.current_device())
    return d


def _same_device(device, *objs):
    """Every tensor / QTensor in objs (None skipped) lives on `device`, a GPU: the
    kernels write through these pointers, so a host buffer must not reach them."""
    ref = _norm(device)
    if ref.type != "cuda":
        raise Q2DError("expected device tensors, got %s" % ref)
    for o in objs:
        if o is not None and _norm(o.device) != ref:
            raise Q2DError("all operands must be on %s (got %s)" % (ref, o.device))


def q2d_quantize(x: torch.Tensor, mode="rtn", seed: int = 0, offset: int = 0,
                 out: QTensor | None = None, block: int = 32) -> QTensor:
    """2D-block FP4 quantization of ``x`` (any 2-D view) into both layouts."""
    _check_input(x)
    R, C = x.shape
    if out is None:
        out = QTensor(FP4_2D, R, C, x.device, block)
    _same_device(x.device, out)
    _check(_lib.q2d_quantize(x.data_ptr(), _dtype_code(x.dtype), R, C, x.stride(0), x.stride(1),
                             block, _ROUND[mode], int(seed), int(offset), out.ptr(),
                             _stream(x.device)), "q2d_quantize")
    return out


def q2d_quantize_1d(x: torch.Tensor, mode="rtn", seed: int = 0, offset: int = 0,
                    out: QTensor | None = None, block: int = 32) -> QTensor:
    """1D FP4 quantization of activations: 1x32 rowwise copy and 32x1 colwise copy."""
    _check_input(x)
    R, C = x.shape
    if out is None:
        out = QTensor(FP4_1D, R, C, x.device, block)
    _same_device(x.device, out)
    _check(_lib.q2d_quantize_1d(x.data_ptr(), _dtype_code(x.dtype), R, C, x.stride(0), x.stride(1),
                                block, _ROUND[mode], int(seed), int(offset), out.ptr(),
                                _stream(x.device)), "q2d_quantize_1d")
    return out


def mxfp8_quantize(x: torch.Tensor, out: QTensor | None = None) -> QTensor:
    """MXFP8 (E4M3, 1x32) quantization: rowwise and colwise copies in one pass."""
    _check_input(x)
    R, C = x.shape
    if out is None:
        out = QTensor(MXFP8, R, C, x.device)
    _same_device(x.device, out)
    _check(_lib.mxfp8_quantize(x.data_ptr(), _dtype_code(x.dtype), R, C, x.stride(0), x.stride(1),
                               out.ptr(), _stream(x.device)), "mxfp8_quantize")
    return out


def q2d_dequantize(q: QTensor, copy: int = 0, out_dtype=torch.float32, exps: bool = False,
                   out: torch.Tensor | None = None):
    """Values of one stored copy of ``q`` as an R x C tensor (copy 0: the forward
    copy codes/scales; 1: the backward copy codes_t/scales_t, mapped back to
    (r, c)).  With exps=True also returns the int8 scale exponent of every element
    (-128 for a non-finite block)."""
    R, C = q.rows, q.cols
    if out is None:
        out = torch.empty((R, C), dtype=out_dtype, device=q.device)
    if out.dim() != 2 or out.stride(1) != 1 or tuple(out.shape) != (R, C):
        raise Q2DError("output must be a row-major R x C tensor")
    e = torch.empty((R, C), dtype=torch.int8, device=q.device) if exps else None
    _same_device(q.device, out, e)
    _check(_lib.q2d_dequantize(q.ptr(), int(copy), out.data_ptr(), _dtype_code(out.dtype), out.stride(0),
                               e.data_ptr() if e is not None else None, C, _stream(q.device)),
           "q2d_dequantize")
    return (out, e) if exps else out


def q2d_gemm(A: QTensor, transA: int, B: QTensor, transB: int, out: torch.Tensor | None = None,
             out_dtype=torch.float32, accumulate: bool = False) -> torch.Tensor:
    """C = op(A) op(B)^T with op(X) = X or X^T (K-major quantized operands)."""
    M = A.cols if transA else A.rows
    N = B.cols if transB else B.rows
    if out is None:
        out = torch.empty((M, N), dtype=out_dtype, device=A.device)
    if out.dim() != 2 or out.stride(1) != 1:
        raise Q2DError("output must be a row-major 2-D tensor")
    _same_device(A.device, B, out)
    _check(_lib.q2d_gemm(A.ptr(), int(transA), B.ptr(), int(transB), out.data_ptr(),
                         _dtype_code(out.dtype), out.stride(0), int(bool(accumulate)),
                         _stream(A.device)), "q2d_gemm")
    return out


def q2d_gemm_quantized(A: QTensor, transA: int, B: QTensor, transB: int, mode="rtn",
                       out: QTensor | None = None, seed: int = 0, offset: int = 0) -> QTensor:
    """op(A) op(B)^T quantized to 2D-block FP4 in the GEMM's epilogue (round to
    nearest, or stochastic rounding with the stream (seed, offset) keyed by the
    row-major storage index of the M x N result); returns the quantized result
    with both orientations."""
    M = A.cols if transA else A.rows
    N = B.cols if transB else B.rows
    if out is None:
        out = QTensor(FP4_2D, M, N, A.device)
    _same_device(A.device, B, out)
    _check(_lib.q2d_gemm_quantized(A.ptr(), int(transA), B.ptr(), int(transB), _ROUND[mode], int(seed),
                                   int(offset), out.ptr(), _stream(A.device)), "q2d_gemm_quantized")
    return out


def q2d_linear_fwd(X: torch.Tensor, W: torch.Tensor, mode_x="rtn", mode_w="rtn", seed: int = 0,
                   offset_x: int = 0, offset_w: int = 1, y_dtype=torch.bfloat16,
                   qX: QTensor | None = None, qW: QTensor | None = None, Y=None, fmt_x: int = FP4_2D,
                   block: int = 32):
    """Y = Q(X) Q(W)^T; returns (Y, qX, qW) with both orientations kept.  fmt_x
    FP4_1D quantizes X in 1D blocks (the activation placement of the paper);
    block 64 gives the 2D-block operands 64 x 64 blocks."""
    _check_input(X)
    _check_input(W)
    T, K = X.shape
    N = W.shape[0]
    if not (X.is_contiguous() and W.is_contiguous()) or W.shape[1] != K or X.dtype != W.dtype:
        raise Q2DError("q2d_linear_fwd expects contiguous X [T,K] and W [N,K] of one dtype")
    qX = qX or QTensor(fmt_x, T, K, X.device, 32 if fmt_x == FP4_1D else block)
    qW = qW or QTensor(FP4_2D, N, K, X.device, block)
    if Y is None:
        Y = torch.empty((T, N), dtype=y_dtype, device=X.device)
    _same_device(X.device, W, qX, qW, Y)
    _check(_lib.q2d_linear_fwd(X.data_ptr(), W.data_ptr(), _dtype_code(X.dtype), T, N, K,
                               _ROUND[mode_x], _ROUND[mode_w], int(seed), int(offset_x),
                               int(offset_w), qX.ptr(), qW.ptr(), Y.data_ptr(),
                               _dtype_code(Y.dtype), _stream(X.device)), "q2d_linear_fwd")
    return Y, qX, qW


def q2d_linear_bwd(dY: torch.Tensor, qX: QTensor, qW: QTensor, mode_dy="sr", seed: int = 0,
                   offset_dy: int = 2, dx_dtype=torch.bfloat16, dw_dtype=torch.float32,
                   dW: torch.Tensor | None = None, accumulate_dw: bool = False,
                   qdY: QTensor | None = None, dX=None, block: int = 32):
    """dX = Q(dY) Q(W), dW = Q(dY)^T Q(X) reusing the forward's operands; returns
    (dX, dW, qdY).  block: dY's block edge (32, or 64 for 64 x 64 blocks)."""
    _check_input(dY)
    T, N = dY.shape
    K = qX.cols
    if not dY.is_contiguous():
        raise Q2DError("q2d_linear_bwd expects a contiguous dY")
    qdY = qdY or QTensor(FP4_2D, T, N, dY.device, block)
    if dX is None:
        dX = torch.empty((T, K), dtype=dx_dtype, device=dY.device)
    if dW is None:
        dW = torch.zeros((N, K), dtype=dw_dtype, device=dY.device) if accumulate_dw else \
            torch.empty((N, K), dtype=dw_dtype, device=dY.device)
    _same_device(dY.device, qX, qW, qdY, dX, dW)
    _check(_lib.q2d_linear_bwd(dY.data_ptr(), _dtype_code(dY.dtype), qX.ptr(), qW.ptr(),
                               _ROUND[mode_dy], int(seed), int(offset_dy), qdY.ptr(),
                               dX.data_ptr(), _dtype_code(dX.dtype), dW.data_ptr(),
                               _dtype_code(dW.dtype), int(bool(accumulate_dw)),
                               _stream(dY.device)), "q2d_linear_bwd")
    return dX, dW, qdY


def q2d_grouped_tensor_init(rows: int, cols: int, nseg: int, device, block: int = 32) -> QTensor:
    return QTensor(FP4_2D, rows, cols, device, block, nseg=nseg)


def _check_offsets(seg_offsets: torch.Tensor, device) -> int:
    if (not seg_offsets.is_cuda or seg_offsets.dtype != torch.int64 or seg_offsets.dim() != 1
            or not seg_offsets.is_contiguous() or seg_offsets.device != torch.device(device)):
        raise Q2DError("seg_offsets must be a contiguous int64 device tensor of nseg + 1 entries")
    return seg_offsets.numel() - 1


def q2d_grouped_quantize(x: torch.Tensor, seg_offsets: torch.Tensor, mode="rtn", seed: int = 0,
                         offset: int = 0, out: QTensor | None = None, block: int = 32) -> QTensor:
    """Per-expert 2D-block FP4 quantization of the expert segments of ``x`` (rows
    seg_offsets[e] .. seg_offsets[e+1]) into the padded grouped layouts."""
    _check_input(x)
    if x.stride(1) != 1:
        raise Q2DError("grouped input must have unit column stride")
    S, C = x.shape
    nseg = _check_offsets(seg_offsets, x.device)
    if out is None:
        out = QTensor(FP4_2D, S, C, x.device, block, nseg=nseg)
    _same_device(x.device, out)
    _check(_lib.q2d_grouped_quantize(x.data_ptr(), _dtype_code(x.dtype), S, C, x.stride(0), nseg,
                                     seg_offsets.data_ptr(), block, _ROUND[mode], int(seed),
                                     int(offset), out.ptr(), _stream(x.device)),
           "q2d_grouped_quantize")
    return out


def q2d_grouped_gemm(A: QTensor, transA: int, B: QTensor, transB: int, seg_offsets: torch.Tensor,
                     out: torch.Tensor | None = None, out_dtype=torch.float32,
                     accumulate: bool = False) -> torch.Tensor:
    """Per-expert GEMMs.  transA = 0: C[rows of e] = A_e op(B)_e^T over the stacked
    expert matrices in B; transA = 1: C_e = A_e^T B_e stacked along rows."""
    nseg = _check_offsets(seg_offsets, A.device)
    S = A.total_rows
    if transA:
        shape = (nseg * A.cols, B.cols)
    else:
        shape = (S, B.cols if transB else B.rows // nseg)
    if out is None:
        out = torch.empty(shape, dtype=out_dtype, device=A.device)
    if out.dim() != 2 or out.stride(1) != 1 or tuple(out.shape) != shape:
        raise Q2DError("output must be a row-major %s tensor" % (shape,))
    _same_device(A.device, B, out)
    _check(_lib.q2d_grouped_gemm(A.ptr(), int(transA), B.ptr(), int(transB), nseg,
                                 seg_offsets.data_ptr(), S, out.data_ptr(), _dtype_code(out.dtype),
                                 out.stride(0), int(bool(accumulate)), _stream(A.device)),
           "q2d_grouped_gemm")
    return out
