"""CPU oracle for the 2D-block FP4 method (test infrastructure only).

Only the tests, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  It shares no code with the HIP library:
the element arithmetic lives in ``q2d_oracle.c`` (plain C, double precision),
the GEMM is the plain fp64 definition on dequantized operands.

What each function follows:
  * ``quantize_fp4_2d``: 2D square blocks, block maximum, truncation-free
    power-of-two scale, round-to-nearest or stochastic rounding (Sec. 3,
    Sec. 3.1, App. D, App. E);
  * ``dequant_fp4*``: the quantized block S * round(B / S) (App. D);
  * ``gemm``: Y = X W^T, dX = dY W, dW = dY^T X on quantized operands
    (Sec. 3, "Application to linear layers"; App. C);
  * ``quantize_mxfp8``: MXFP8 for the query/key projections (Sec. 3.2; App. C);
  * ``quantize_fp4_1d``: 1D FP4 for activations, 1x32 blocks for the forward
    copy and 32x1 blocks for the weight-gradient copy (Sec. 3, "Application to
    linear layers"; App. C, "Activations");
  * ``quantize_fp4_grouped``: each expert's row segment is its own matrix
    (the MoE setting of Sec. 4.1) with boundary blocks over valid rows only
    (App. D).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "q2d_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

E2M1 = np.array([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0], dtype=np.float64)
BLOCK = 32


def build(force: bool = False) -> str:
    """Compile the C oracle with gcc (strict IEEE, OpenMP)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c99",
                               "-fno-fast-math", "-ffp-contract=off", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build()
        L = ctypes.CDLL(_LIB_PATH)
        P, I64, I32, U64 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_uint64
        L.or_philox4x32_10.argtypes = [P, P, P]
        L.or_sr_bits.argtypes = [I64, U64, U64]
        L.or_sr_bits.restype = ctypes.c_uint32
        L.or_fp4_scale_exponent.argtypes = [ctypes.c_double]
        L.or_fp4_scale_exponent.restype = I32
        L.or_fp4_floor_exponent.argtypes = [ctypes.c_double]
        L.or_fp4_floor_exponent.restype = I32
        L.or_fp8_scale_exponent.argtypes = [ctypes.c_double]
        L.or_fp8_scale_exponent.restype = I32
        L.or_fp4_code.argtypes = [ctypes.c_double, I32, I32, ctypes.c_uint32]
        L.or_fp4_code.restype = ctypes.c_uint
        L.or_e4m3_code.argtypes = [ctypes.c_double, I32]
        L.or_e4m3_code.restype = ctypes.c_uint
        L.or_quantize_fp4_2d.argtypes = [P, I32, I64, I64, I64, I64, I64, I32, I32, U64, U64,
                                         P, I64, P, I64, P, I64, P, I64, I32]
        L.or_quantize_mxfp8.argtypes = [P, I32, I64, I64, I64, I64,
                                        P, I64, P, I64, P, I64, P, I64, I32]
        L.or_quantize_fp4_1d.argtypes = [P, I32, I64, I64, I64, I64, I32, U64, U64,
                                         P, I64, P, I64, P, I64, P, I64, I32]
        L.or_fp4_codes.argtypes = [P, P, P, I32, I64, P]
        L.or_e4m3_codes.argtypes = [P, P, I64, P]
        L.or_max_threads.restype = I32
        _lib = L
    return _lib


def max_threads() -> int:
    return int(lib().or_max_threads())


# ------------------------------------------------------------------ scalars

def philox4x32_10(ctr, key):
    c = np.ascontiguousarray(np.asarray(ctr, dtype=np.uint32))
    k = np.ascontiguousarray(np.asarray(key, dtype=np.uint32))
    out = np.zeros(4, dtype=np.uint32)
    lib().or_philox4x32_10(c.ctypes.data, k.ctypes.data, out.ctypes.data)
    return out


def sr_bits(idx: int, seed: int, offset: int) -> int:
    return int(lib().or_sr_bits(int(idx), int(seed), int(offset)))


def fp4_scale_exponent(M: float) -> int:
    return int(lib().or_fp4_scale_exponent(float(M)))


def fp4_floor_exponent(M: float) -> int:
    """Scale exponent of the truncation-free ablation: floor(log2 M) - 2, clamped to -127."""
    return int(lib().or_fp4_floor_exponent(float(M)))


def fp8_scale_exponent(M: float) -> int:
    return int(lib().or_fp8_scale_exponent(float(M)))


def fp4_code(x: float, e: int, stochastic: bool = False, r16: int = 0) -> int:
    return int(lib().or_fp4_code(float(x), int(e), int(bool(stochastic)), int(r16)))


def e4m3_code(x: float, e: int) -> int:
    return int(lib().or_e4m3_code(float(x), int(e)))


def fp4_codes(x, e, stochastic: bool = False, r16=None) -> np.ndarray:
    """Vector form of ``fp4_code`` (x float64, e int, r16 uint32 arrays)."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    e = np.ascontiguousarray(np.broadcast_to(e, x.shape), dtype=np.int32)
    out = np.zeros(x.shape, dtype=np.uint8)
    rp = None
    if r16 is not None:
        r16 = np.ascontiguousarray(np.broadcast_to(r16, x.shape), dtype=np.uint32)
        rp = r16.ctypes.data
    lib().or_fp4_codes(x.ctypes.data, e.ctypes.data, rp, int(bool(stochastic)), x.size,
                       out.ctypes.data)
    return out


def e4m3_codes(x, e) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.float64)
    e = np.ascontiguousarray(np.broadcast_to(e, x.shape), dtype=np.int32)
    out = np.zeros(x.shape, dtype=np.uint8)
    lib().or_e4m3_codes(x.ctypes.data, e.ctypes.data, x.size, out.ctypes.data)
    return out


# ------------------------------------------------------------------ layouts

def _rup(a: int, m: int) -> int:
    return (a + m - 1) // m * m


def fp4_layout(R: int, C: int) -> dict:
    """Buffer shapes of the packed 2D-block FP4 layouts (rows, bytes per row)."""
    return {
        "codes": (R, _rup(C, 128) // 2),
        "codes_t": (C, _rup(R, 128) // 2),
        "scales": ((R + BLOCK - 1) // BLOCK, _rup(C, 128) // BLOCK),
        "scales_t": ((C + BLOCK - 1) // BLOCK, _rup(R, 128) // BLOCK),
    }


def mxfp8_layout(R: int, C: int) -> dict:
    return {
        "codes": (R, _rup(C, 128)),
        "scales": (R, _rup(C, 128) // 32),
        "codes_t": (C, _rup(R, 128)),
        "scales_t": (C, _rup(R, 128) // 32),
    }


def fp4_1d_layout(R: int, C: int) -> dict:
    """1D FP4: codes packed as for 2D blocks; one scale per row (per column for
    the transposed copy) and 32-element K-group, stored as one 4-byte word per
    row and K-tile of 128: [K-tiles][rows * 4] bytes."""
    return {
        "codes": (R, _rup(C, 128) // 2),
        "scales": (_rup(C, 128) // 128, 4 * R),
        "codes_t": (C, _rup(R, 128) // 2),
        "scales_t": (_rup(R, 128) // 128, 4 * C),
    }


def scale_grid_1d(words: np.ndarray, rows: int) -> np.ndarray:
    """The [rows][K-groups] E8M0 bytes of a 1D scale buffer in word layout."""
    nkt = words.shape[0]
    return words.reshape(nkt, -1, 4)[:, :rows].transpose(1, 0, 2).reshape(rows, nkt * 4)


def grouped_rows(offsets) -> np.ndarray:
    """Padded start row of every segment (segments are padded to 128 rows)."""
    off = np.asarray(offsets, dtype=np.int64)
    n = off[1:] - off[:-1]
    p = np.zeros(len(off), dtype=np.int64)
    p[1:] = np.cumsum(((n + 127) // 128) * 128)
    return p


def fp4_grouped_layout(offsets, C: int) -> dict:
    P = int(grouped_rows(offsets)[-1])
    return {
        "codes": (P, _rup(C, 128) // 2),
        "codes_t": (C, P // 2),
        "scales": (P // BLOCK, _rup(C, 128) // BLOCK),
        "scales_t": ((C + BLOCK - 1) // BLOCK, P // BLOCK),
    }


# ------------------------------------------------------------------ inputs

def _as_input(x):
    """(pointer holder, dtype code, rows, cols, stride_r, stride_c) of a 2-D CPU input.

    Accepts torch tensors (float32 or bfloat16, any strides) or numpy arrays
    (float32, or uint16 holding bfloat16 bits)."""
    try:
        import torch
        if isinstance(x, torch.Tensor):
            assert x.device.type == "cpu" and x.dim() == 2
            if x.dtype == torch.float32:
                dt = 0
            elif x.dtype == torch.bfloat16:
                dt = 1
            else:
                raise TypeError("oracle input must be float32 or bfloat16")
            return x, x.data_ptr(), dt, x.shape[0], x.shape[1], x.stride(0), x.stride(1)
    except ImportError:
        pass
    a = np.asarray(x)
    assert a.ndim == 2
    if a.dtype == np.float32:
        dt = 0
    elif a.dtype == np.uint16:
        dt = 1
    else:
        raise TypeError("oracle input must be float32 or bfloat16 bits (uint16)")
    st = [s // a.itemsize for s in a.strides]
    return a, a.ctypes.data, dt, a.shape[0], a.shape[1], st[0], st[1]


def to_float64(x) -> np.ndarray:
    """Exact float64 copy of a float32 / bfloat16 input."""
    try:
        import torch
        if isinstance(x, torch.Tensor):
            return x.to(torch.float64).numpy()
    except ImportError:
        pass
    a = np.asarray(x)
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return a.astype(np.float64)


# ------------------------------------------------------------------ quantizers

def _mode_bits(mode: str) -> int:
    """Rounding and scale rule of the 2D quantizer: bit 0 stochastic rounding, bit 1
    the floor scale rule of the truncation-free ablation ("rtn-floor", "sr-floor")."""
    bits = {"rtn": 0, "sr": 1, "rtn-floor": 2, "sr-floor": 3}
    if mode not in bits:
        raise ValueError("unknown rounding mode " + repr(mode))
    return bits[mode]


def quantize_fp4_2d(x, mode: str = "rtn", seed: int = 0, offset: int = 0,
                    threads: int = 0, index_base: int = 0, block: int = BLOCK) -> dict:
    """2D-block FP4 quantization of a 2-D CPU tensor into both packed layouts.

    ``index_base`` is added to every storage index before it keys the random
    stream (the grouped form uses the segment's first storage index).
    ``block`` 64 (the larger block of the block-size trade-off, Table 4): the
    blocks are 64 x 64 and the scale grids keep the 32-granular layout, the byte
    of 64-block (i, j) in the four entries (2i .. 2i+1, 2j .. 2j+1)."""
    hold, ptr, dt, R, C, sr, sc = _as_input(x)
    lay = fp4_layout(R, C)
    out = {k: np.zeros(v, dtype=np.uint8) for k, v in lay.items()}
    if block == BLOCK:
        sc_buf, sct_buf = out["scales"], out["scales_t"]
    else:
        assert block == 64
        nr, nc = -(-R // block), -(-C // block)
        sc_buf, sct_buf = np.zeros((nr, nc), np.uint8), np.zeros((nc, nr), np.uint8)
    lib().or_quantize_fp4_2d(ptr, dt, R, C, sr, sc, int(index_base), int(block),
                             _mode_bits(mode),
                             int(seed), int(offset),
                             out["codes"].ctypes.data, lay["codes"][1],
                             out["codes_t"].ctypes.data, lay["codes_t"][1],
                             sc_buf.ctypes.data, sc_buf.shape[1],
                             sct_buf.ctypes.data, sct_buf.shape[1], int(threads))
    if block != BLOCK:
        for name, comp in (("scales", sc_buf), ("scales_t", sct_buf)):
            g = out[name]
            i = np.arange(g.shape[0]) // 2
            j = np.arange(g.shape[1]) // 2
            inside = j < comp.shape[1]
            g[:, inside] = comp[i][:, j[inside]]
    out["rows"], out["cols"] = R, C
    return out


def quantize_fp4_grouped(x, offsets, mode: str = "rtn", seed: int = 0, offset: int = 0,
                         threads: int = 0) -> dict:
    """Per-segment 2D-block FP4: segment e (rows offsets[e]..offsets[e+1]) is its own
    matrix; its blocks start at its first row; it is stored from padded row p[e]."""
    hold, ptr, dt, S, C, sr, sc = _as_input(x)
    off = np.asarray(offsets, dtype=np.int64)
    assert off[0] == 0 and off[-1] == S
    p = grouped_rows(off)
    lay = fp4_grouped_layout(off, C)
    out = {k: np.zeros(v, dtype=np.uint8) for k, v in lay.items()}
    esize = 4 if dt == 0 else 2
    for e in range(len(off) - 1):
        n = int(off[e + 1] - off[e])
        if n == 0:
            continue
        base = ptr + int(off[e]) * sr * esize
        pe = int(p[e])
        lib().or_quantize_fp4_2d(
            base, dt, n, C, sr, sc, int(off[e]) * sr, BLOCK, _mode_bits(mode),
            int(seed), int(offset),
            out["codes"].ctypes.data + pe * lay["codes"][1], lay["codes"][1],
            out["codes_t"].ctypes.data + pe // 2, lay["codes_t"][1],
            out["scales"].ctypes.data + (pe // BLOCK) * lay["scales"][1], lay["scales"][1],
            out["scales_t"].ctypes.data + pe // BLOCK, lay["scales_t"][1], int(threads))
    out["rows"], out["cols"], out["padded_rows"] = S, C, p
    return out


def quantize_mxfp8(x, threads: int = 0) -> dict:
    """MXFP8 E4M3: rowwise 1x32 copy and colwise 32x1 copy (stored transposed)."""
    hold, ptr, dt, R, C, sr, sc = _as_input(x)
    lay = mxfp8_layout(R, C)
    out = {k: np.zeros(v, dtype=np.uint8) for k, v in lay.items()}
    lib().or_quantize_mxfp8(ptr, dt, R, C, sr, sc,
                            out["codes"].ctypes.data, lay["codes"][1],
                            out["scales"].ctypes.data, lay["scales"][1],
                            out["codes_t"].ctypes.data, lay["codes_t"][1],
                            out["scales_t"].ctypes.data, lay["scales_t"][1], int(threads))
    out["rows"], out["cols"] = R, C
    return out


def quantize_fp4_1d(x, mode: str = "rtn", seed: int = 0, offset: int = 0, threads: int = 0) -> dict:
    """1D FP4: rowwise 1x32 copy (codes/scales) and colwise 32x1 copy stored
    transposed (codes_t/scales_t); truncation-free scales, E2M1 codes, the
    element's one stochastic draw used in both copies."""
    hold, ptr, dt, R, C, sr, sc = _as_input(x)
    lay = fp4_1d_layout(R, C)
    out = {k: np.zeros(v, dtype=np.uint8) for k, v in lay.items()}
    lib().or_quantize_fp4_1d(ptr, dt, R, C, sr, sc, 1 if mode == "sr" else 0,
                             int(seed), int(offset),
                             out["codes"].ctypes.data, lay["codes"][1],
                             out["scales"].ctypes.data, lay["scales"][1],
                             out["codes_t"].ctypes.data, lay["codes_t"][1],
                             out["scales_t"].ctypes.data, lay["scales_t"][1], int(threads))
    out["rows"], out["cols"] = R, C
    return out


# ------------------------------------------------------------------ dequantization

def _scale_values(sbytes: np.ndarray) -> np.ndarray:
    e = sbytes.astype(np.float64) - 127.0
    v = np.ldexp(1.0, e.astype(np.int64))
    return np.where(sbytes == 0xFF, np.nan, v)


def fp4_values(nibbles: np.ndarray) -> np.ndarray:
    mag = E2M1[nibbles & 7]
    return np.where(nibbles & 8, -mag, mag)


def _unpack(packed: np.ndarray, n: int) -> np.ndarray:
    lo = packed & 0x0F
    hi = packed >> 4
    u = np.empty((packed.shape[0], packed.shape[1] * 2), dtype=np.uint8)
    u[:, 0::2] = lo
    u[:, 1::2] = hi
    return u[:, :n]


def dequant_fp4(codes: np.ndarray, scales: np.ndarray, R: int, C: int) -> np.ndarray:
    """R x C float64 values S * code of a row-packed operand (row r, K index c)."""
    q = fp4_values(_unpack(codes[:R], C))
    s = _scale_values(scales)
    rb = np.arange(R) // BLOCK
    cb = np.arange(C) // BLOCK
    return q * s[rb][:, cb]


def dequant_fp4_1d(codes: np.ndarray, scales: np.ndarray, R: int, C: int) -> np.ndarray:
    """R x C float64 values of a 1x32-block FP4 operand (row r, K index c)."""
    q = fp4_values(_unpack(codes[:R], C))
    s = _scale_values(scale_grid_1d(scales, R))
    return q * s[:, np.arange(C) // 32]


def dequant_mxfp8(codes: np.ndarray, scales: np.ndarray, R: int, C: int) -> np.ndarray:
    """R x C float64 values of a 1x32-block E4M3 operand (K index along columns)."""
    b = codes[:R, :C].astype(np.int64)
    E = (b >> 3) & 15
    m = b & 7
    mag = np.where(E == 0, np.ldexp(m.astype(np.float64), -9),
                   np.ldexp(1.0 + m / 8.0, (E - 7)))
    mag = np.where((b & 0x7F) == 0x7F, np.nan, mag)        # E4M3FN: S.1111.111 is NaN
    val = np.where(b & 0x80, -mag, mag)
    s = _scale_values(scales[:R])
    return val * s[:, np.arange(C) // 32]


def operand(q: dict, transpose: bool, fmt: str = "fp4") -> np.ndarray:
    """op(A) as float64 with K along columns: the row-packed copy, or the
    column-packed copy for transpose=True."""
    R, C = q["rows"], q["cols"]
    if fmt == "fp4":
        if not transpose:
            return dequant_fp4(q["codes"], q["scales"], R, C)
        return dequant_fp4(q["codes_t"], q["scales_t"], C, R)
    if fmt == "fp4_1d":
        if not transpose:
            return dequant_fp4_1d(q["codes"], q["scales"], R, C)
        return dequant_fp4_1d(q["codes_t"], q["scales_t"], C, R)
    if not transpose:
        return dequant_mxfp8(q["codes"], q["scales"], R, C)
    return dequant_mxfp8(q["codes_t"], q["scales_t"], C, R)


def dequantize(q: dict, copy: int, fmt: str = "fp4") -> np.ndarray:
    """R x C float64 values of one stored copy (0: codes/scales, the copy the
    forward GEMM reads; 1: codes_t/scales_t, the backward GEMMs' copy) in the
    matrix's own orientation: the quantized operands X_fwd and X_bwd of Sec. 2
    ("Bias induced by scale inconsistency")."""
    return operand(q, False, fmt) if copy == 0 else operand(q, True, fmt).T


def scale_exponents(q: dict, copy: int, fmt: str = "fp4") -> np.ndarray:
    """R x C int64 scale exponent e of each element's block in one stored copy
    (-128 for scale byte 0xFF); copy 0 minus copy 1 is the scale-difference map
    of Fig. 1."""
    R, C = q["rows"], q["cols"]
    if copy == 0:
        K, S, sc = C, R, q["scales"]
    else:
        K, S, sc = R, C, q["scales_t"]
    if fmt == "fp4":
        g = sc[:(S + BLOCK - 1) // BLOCK]
        e = g[np.arange(S) // BLOCK][:, np.arange(K) // BLOCK]
    elif fmt == "fp4_1d":
        e = scale_grid_1d(sc, S)[:, np.arange(K) // 32]
    else:
        e = sc[:S][:, np.arange(K) // 32]
    e = np.where(e == 0xFF, -128, e.astype(np.int64) - 127)
    return e if copy == 0 else e.T


def gemm(a: np.ndarray, b: np.ndarray) -> np.ndarray:
    """C = A B^T in float64 for K-major operands A [M, K], B [N, K]."""
    return np.asarray(a, dtype=np.float64) @ np.asarray(b, dtype=np.float64).T


def gemm_quantized(a: np.ndarray, b: np.ndarray, mode: str = "rtn", seed: int = 0, offset: int = 0) -> dict:
    """A GEMM whose result is quantized (App. C: a layer's output is the next
    GEMM's operand): C = A B^T in float64, rounded once to float32 (the
    precision the result has before it is quantized), then 2D-block FP4 of the
    row-major M x N result: round to nearest, or stochastic rounding with the
    stream (seed, offset) for a gradient output (App. E)."""
    c = gemm(a, b)
    with np.errstate(over="ignore"):
        c32 = c.astype(np.float32)
    return quantize_fp4_2d(np.ascontiguousarray(c32), mode, seed, offset)


def linear(qx: dict, qw: dict, qdy: dict, fmt: str = "fp4", fmt_x: str | None = None) -> dict:
    """The three GEMMs of a linear layer on quantized operands (App. C):
    Y = X W^T, dX = dY W, dW = dY^T X, each operand quantized once.  fmt_x
    (default fmt) is the format of X: "fp4_1d" for the paper's activation
    placement (App. C, "Activations")."""
    fx = fmt if fmt_x is None else fmt_x
    X = operand(qx, False, fx)
    W = operand(qw, False, fmt)
    dY = operand(qdy, False, fmt)
    Xt = operand(qx, True, fx)
    Wt = operand(qw, True, fmt)
    dYt = operand(qdy, True, fmt)
    return {"Y": gemm(X, W), "dX": gemm(dY, Wt), "dW": gemm(dYt, Xt)}
