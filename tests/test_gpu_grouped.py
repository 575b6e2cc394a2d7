"""GPU parity of the grouped (mixture-of-experts) path against the oracle.

Quantizer: every byte of the padded grouped layouts (all padded segments, both
orientations) equals ``oracle.quantize_fp4_grouped`` of the same input, for
RTN and SR, bf16 and fp32, dense and row-strided inputs; segment lengths
cover empty experts, single rows, lengths around the 32-row block and the
128-row padding, and several 256-row GEMM tiles; the maximum of 1024 experts.
Each padded segment also equals an ungrouped quantization of that expert's
rows (device against device).

GEMMs: per expert, relative Frobenius error <= 1e-5 (fp32 output) of the
device result against float64 products of the oracle's operands; bf16
outputs within one bf16 rounding.  Ragged M (forward and data gradient, both
layouts of the stacked expert weights) and ragged K (weight gradient, with
accumulation and empty experts), and the 30B-class MoE expert FFN at full
size in the benchmark's launch configuration on sampled rows.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from helpers import assert_same_bytes, check_bf16, gpu_buffers, rel_frob

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
TOL = 1e-5
BUFS = ("codes", "codes_t", "scales", "scales_t")

COUNTS = {
    "edges": [0, 1, 31, 33, 127, 130, 256, 300],
    "one": [513],
    "sparse": [0, 0, 5, 0],
}


@pytest.fixture(scope="module")
def q2d():
    import paper_2607_24953_amd as q
    return q


def dev_offsets(off):
    return torch.tensor(np.asarray(off, dtype=np.int64), device=DEV)


def grouped_bytes(q, P):
    """Host copy of the written region (the first P padded rows) of a grouped tensor."""
    torch.cuda.synchronize()
    return {"codes": q.codes[:P].cpu().numpy(), "scales": q.scales[:P // 32].cpu().numpy(),
            "codes_t": q.codes_t[:, :P // 2].cpu().numpy(),
            "scales_t": q.scales_t[:, :P // 32].cpu().numpy()}


def assert_grouped_equal(q, o, label):
    P = int(o["padded_rows"][-1])
    got = grouped_bytes(q, P)
    for k in BUFS:
        g, w = got[k], o[k]
        assert g.shape == w.shape, (label, k, g.shape, w.shape)
        if not np.array_equal(g, w):
            bad = np.argwhere(g != w)
            r, c = bad[0]
            raise AssertionError("%s %s: %d bytes differ, first at (%d, %d): gpu %#04x oracle %#04x"
                                 % (label, k, len(bad), r, c, g[r, c], w[r, c]))


def quant_grouped(q2d, x, off, mode, seed=0, offset=0, x_cpu=None):
    q = q2d.q2d_grouped_quantize(x, dev_offsets(off), mode, seed, offset)
    o = oracle.quantize_fp4_grouped(x.cpu() if x_cpu is None else x_cpu, off, mode, seed, offset)
    assert_grouped_equal(q, o, "grouped operand")
    return q, o


# ------------------------------------------------------------------ quantizer

@pytest.mark.parametrize("counts", ["edges", "sparse"])
@pytest.mark.parametrize("C", [200, 384])
def test_grouped_equals_per_expert_calls(q2d, counts, C):
    """Each padded segment of a grouped RTN quantization holds exactly what an
    ungrouped q2d_quantize of that expert's rows writes (GPU against GPU):
    segments are quantized as matrices of their own, from row 0 of the segment."""
    cnt = COUNTS[counts]
    off = np.concatenate([[0], np.cumsum(cnt)]).astype(np.int64)
    S = max(int(off[-1]), 1)
    x = synth.normal((S, C), 1.0, 4242 + C, torch.bfloat16, device=DEV)
    q = q2d.q2d_grouped_quantize(x, dev_offsets(off), "rtn")
    P = 0
    for e, n in enumerate(cnt):
        if n:
            u = q2d.q2d_quantize(x[off[e]:off[e] + n], "rtn")
            np_ = -(-n // 128) * 128
            torch.cuda.synchronize()
            got = {"codes": q.codes[P:P + n], "scales": q.scales[P // 32:P // 32 + -(-n // 32)],
                   "codes_t": q.codes_t[:, P // 2:P // 2 + np_ // 2],
                   "scales_t": q.scales_t[:, P // 32:P // 32 + np_ // 32]}
            want = {"codes": u.codes[:n], "scales": u.scales[:-(-n // 32)],
                    "codes_t": u.codes_t[:, :np_ // 2], "scales_t": u.scales_t[:, :np_ // 32]}
            for k in BUFS:
                assert torch.equal(got[k], want[k]), (counts, C, e, n, k)
            P += np_



@pytest.mark.parametrize("counts", list(COUNTS))
@pytest.mark.parametrize("C", [96, 200, 384])
@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
@pytest.mark.parametrize("mode", ["rtn", "sr"])
def test_grouped_quantize(q2d, counts, C, dtype, mode):
    off = synth.segment_offsets(COUNTS[counts])
    S = int(off[-1])
    x = synth.normal((S, C), 1.0, S + C, dtype, device=DEV)
    synth.add_outlier_channels(x, 3, frac=0.05)
    q = q2d.q2d_grouped_quantize(x, dev_offsets(off), mode, 5, 11)
    q.codes.fill_(0xAA), q.codes_t.fill_(0xAA), q.scales.fill_(0xAA), q.scales_t.fill_(0xAA)
    q2d.q2d_grouped_quantize(x, dev_offsets(off), mode, 5, 11, out=q)
    o = oracle.quantize_fp4_grouped(x.cpu(), off, mode, 5, 11)
    assert_grouped_equal(q, o, "%s C=%d %s %s" % (counts, C, dtype, mode))


@pytest.mark.parametrize("mode", ["rtn", "sr"])
@pytest.mark.parametrize("dtype,stride", [(torch.bfloat16, 264), (torch.bfloat16, 261),
                                          (torch.float32, 260)])
def test_grouped_quantize_row_stride(q2d, mode, dtype, stride):
    """Rows of x taken from a wider buffer (row stride > cols): vector loads with
    8-aligned storage indices (264), element-wise loads (261), and vector loads
    whose rows start off the 8-element Philox block (fp32, 260)."""
    off = synth.segment_offsets(COUNTS["edges"])
    S = int(off[-1])
    base = synth.normal((S, stride), 1.0, 77, dtype, device=DEV)
    x = base[:, :200]
    x_cpu = base.cpu()[:, :200]
    quant_grouped(q2d, x, off, mode, 3, 0, x_cpu=x_cpu)


def test_grouped_quantize_max_experts(q2d):
    """1024 experts (the maximum), mostly tiny segments; 1025 is rejected."""
    rng = np.random.default_rng(8)
    counts = rng.integers(0, 40, 1024)
    counts[::97] = 129
    off = synth.segment_offsets(counts)
    S = int(off[-1])
    x = synth.normal((S, 128), 1.0, 9, torch.bfloat16, device=DEV)
    quant_grouped(q2d, x, off, "sr", 1, 2)
    bad = synth.segment_offsets(np.ones(1025, dtype=np.int64))
    xb = synth.normal((1025, 64), 1.0, 9, torch.bfloat16, device=DEV)
    with pytest.raises(q2d.Q2DError):
        q2d.q2d_grouped_quantize(xb, dev_offsets(bad), "rtn")


# ------------------------------------------------------------------ GEMMs

def expert_rows(o, off, e, trans=False):
    """float64 operand rows of expert e from an oracle grouped quantization:
    the row-packed copy [n_e, C] or (trans) the column-packed copy [C, n_e]."""
    P = int(o["padded_rows"][-1])
    p, n = int(o["padded_rows"][e]), int(off[e + 1] - off[e])
    C = o["cols"]
    if not trans:
        return oracle.dequant_fp4(o["codes"], o["scales"], P, C)[p:p + n]
    return oracle.dequant_fp4(o["codes_t"], o["scales_t"], C, P)[:, p:p + n]


@pytest.mark.parametrize("counts", list(COUNTS))
@pytest.mark.parametrize("C", [96, 200, 384])
@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
@pytest.mark.parametrize("mode", ["rtn", "sr"])
def test_grouped_quantize(q2d, counts, C, dtype, mode):
    off = synth.segment_offsets(COUNTS[counts])
    S = int(off[-1])
    x = synth.normal((S, C), 1.0, S + C, dtype, device=DEV)
    synth.add_outlier_channels(x, 3, frac=0.05)
    q = q2d.q2d_grouped_quantize(x, dev_offsets(off), mode, 5, 11)
    q.codes.fill_(0xAA), q.codes_t.fill_(0xAA), q.scales.fill_(0xAA), q.scales_t.fill_(0xAA)
    q2d.q2d_grouped_quantize(x, dev_offsets(off), mode, 5, 11, out=q)
    o = oracle.quantize_fp4_grouped(x.cpu(), off, mode, 5, 11)
    assert_grouped_equal(q, o, "%s C=%d %s %s" % (counts, C, dtype, mode))


@pytest.mark.parametrize("mode", ["rtn", "sr"])
@pytest.mark.parametrize("dtype,stride", [(torch.bfloat16, 264), (torch.bfloat16, 261),
                                          (torch.float32, 260)])
def test_grouped_quantize_row_stride(q2d, mode, dtype, stride):
    """Rows of x taken from a wider buffer (row stride > cols): vector loads with
    8-aligned storage indices (264), element-wise loads (261), and vector loads
    whose rows start off the 8-element Philox block (fp32, 260)."""
    off = synth.segment_offsets(COUNTS["edges"])
    S = int(off[-1])
    base = synth.normal((S, stride), 1.0, 77, dtype, device=DEV)
    x = base[:, :200]
    x_cpu = base.cpu()[:, :200]
    quant_grouped(q2d, x, off, mode, 3, 0, x_cpu=x_cpu)


def test_grouped_quantize_max_experts(q2d):
    """1024 experts (the maximum), mostly tiny segments; 1025 is rejected."""
    rng = np.random.default_rng(8)
    counts = rng.integers(0, 40, 1024)
    counts[::97] = 129
    off = synth.segment_offsets(counts)
    S = int(off[-1])
    x = synth.normal((S, 128), 1.0, 9, torch.bfloat16, device=DEV)
    quant_grouped(q2d, x, off, "sr", 1, 2)
    bad = synth.segment_offsets(np.ones(1025, dtype=np.int64))
    xb = synth.normal((1025, 64), 1.0, 9, torch.bfloat16, device=DEV)
    with pytest.raises(q2d.Q2DError):
        q2d.q2d_grouped_quantize(xb, dev_offsets(bad), "rtn")


# ------------------------------------------------------------------ GEMMs

def expert_rows(o, off, e, trans=False):
    """float64 operand rows of expert e from an oracle grouped quantization:
    the row-packed copy [n_e, C] or (trans) the column-packed copy [C, n_e]."""
    P = int(o["padded_rows"][-1])
    p, n = int(o["padded_rows"][e]), int(off[e + 1] - off[e])
    C = o["cols"]
    if not trans:
        return oracle.dequant_fp4(o["codes"], o["scales"], P, C)[p:p + n]
    return oracle.dequant_fp4(o["codes_t"], o["scales_t"], C, P)[:, p:p + n]


def check_bf16(got, ref):
    got = got.float().cpu().numpy().astype(np.float64)
    err = np.abs(got - ref)
    rms = float(np.sqrt(np.mean(ref * ref))) if ref.size else 0.0
    tol = np.abs(ref) * 2.0 ** -8 + 1e-5 * rms + 1e-38
    assert np.all(err <= tol), float((err / tol).max())


@pytest.mark.parametrize("counts", list(COUNTS))
@pytest.mark.parametrize("N,K", [(96, 256), (320, 200), (64, 1024)])
def test_grouped_gemm_ragged_m(q2d, counts, N, K):
    """Forward: Y_e = X_e W_e^T with W stacked [E*N, K] (row-packed copy)."""
    cnt = COUNTS[counts]
    E = len(cnt)
    off = synth.segment_offsets(cnt)
    S = int(off[-1])
    X = synth.normal((S, K), 1.0, 21, torch.bfloat16, device=DEV)
    W = synth.normal((E * N, K), 0.02, 22, torch.bfloat16, device=DEV)
    qX, oX = quant_grouped(q2d, X, off, "rtn")
    qW = q2d.q2d_quantize(W, "rtn")
    oW = oracle.quantize_fp4_2d(W.cpu(), "rtn")
    Wf = oracle.operand(oW, False)
    Y = q2d.q2d_grouped_gemm(qX, 0, qW, 0, dev_offsets(off), out_dtype=torch.float32)
    Yb = q2d.q2d_grouped_gemm(qX, 0, qW, 0, dev_offsets(off), out_dtype=torch.bfloat16)
    Y, Yb = Y.cpu().numpy(), Yb.cpu()
    for e in range(E):
        a, b = int(off[e]), int(off[e + 1])
        if a == b:
            continue
        ref = oracle.gemm(expert_rows(oX, off, e), Wf[e * N:(e + 1) * N])
        assert rel_frob(Y[a:b], ref) <= TOL, e
        check_bf16(Yb[a:b], ref)


@pytest.mark.parametrize("counts", list(COUNTS))
@pytest.mark.parametrize("Ng,Kin", [(256, 200), (128, 640)])
def test_grouped_gemm_ragged_m_transposed_b(q2d, counts, Ng, Kin):
    """Data gradient: dX_e = dY_e W_e with W stacked [E*Ng, Kin] (column-packed copy)."""
    cnt = COUNTS[counts]
    E = len(cnt)
    off = synth.segment_offsets(cnt)
    S = int(off[-1])
    dY = synth.normal((S, Ng), 1e-3, 31, torch.bfloat16, device=DEV)
    W = synth.normal((E * Ng, Kin), 0.02, 32, torch.bfloat16, device=DEV)
    qdY, odY = quant_grouped(q2d, dY, off, "sr", 4, 2)
    qW = q2d.q2d_quantize(W, "rtn")
    oW = oracle.quantize_fp4_2d(W.cpu(), "rtn")
    Wt = oracle.operand(oW, True)          # [Kin, E*Ng]
    dX = q2d.q2d_grouped_gemm(qdY, 0, qW, 1, dev_offsets(off), out_dtype=torch.float32)
    dX = dX.cpu().numpy()
    for e in range(E):
        a, b = int(off[e]), int(off[e + 1])
        if a == b:
            continue
        ref = oracle.gemm(expert_rows(odY, off, e), Wt[:, e * Ng:(e + 1) * Ng])
        assert rel_frob(dX[a:b], ref) <= TOL, e


@pytest.mark.parametrize("counts", list(COUNTS))
@pytest.mark.parametrize("Ng,K", [(256, 200), (96, 384)])
def test_grouped_gemm_ragged_k(q2d, counts, Ng, K):
    """Weight gradient: dW_e = dY_e^T X_e (K = n_e), plain and accumulating; an
    empty expert gets zeros, or keeps its values when accumulating."""
    cnt = COUNTS[counts]
    E = len(cnt)
    off = synth.segment_offsets(cnt)
    S = int(off[-1])
    dY = synth.normal((S, Ng), 1e-3, 41, torch.bfloat16, device=DEV)
    X = synth.normal((S, K), 1.0, 42, torch.bfloat16, device=DEV)
    qdY, odY = quant_grouped(q2d, dY, off, "sr", 6, 2)
    qX, oX = quant_grouped(q2d, X, off, "rtn")
    dW = torch.full((E * Ng, K), 7.0, device=DEV)
    q2d.q2d_grouped_gemm(qdY, 1, qX, 1, dev_offsets(off), out=dW)
    init = synth.normal((E * Ng, K), 1e-3, 43, torch.float32, device=DEV)
    acc = init.clone()
    q2d.q2d_grouped_gemm(qdY, 1, qX, 1, dev_offsets(off), out=acc, accumulate=True)
    dW, acc, init = dW.cpu().numpy(), acc.cpu().numpy(), init.cpu().numpy().astype(np.float64)
    for e in range(E):
        rows = slice(e * Ng, (e + 1) * Ng)
        if off[e] == off[e + 1]:
            assert np.all(dW[rows] == 0) and np.array_equal(acc[rows], init[rows].astype(np.float32))
            continue
        ref = oracle.gemm(expert_rows(odY, off, e, True), expert_rows(oX, off, e, True))
        assert rel_frob(dW[rows], ref) <= TOL, e
        assert rel_frob(acc[rows], ref + init[rows]) <= TOL, e


def expert_slicer(o, off, trans=False):
    """expert_rows with the grouped operand dequantized once."""
    P, C = int(o["padded_rows"][-1]), o["cols"]
    full = (oracle.dequant_fp4(o["codes_t"], o["scales_t"], C, P) if trans
            else oracle.dequant_fp4(o["codes"], o["scales"], P, C))

    def rows(e):
        p, n = int(o["padded_rows"][e]), int(off[e + 1] - off[e])
        return full[:, p:p + n] if trans else full[p:p + n]
    return rows


def skewed_counts(E, total, seed):
    """Zipf(1.1)-weighted expert sizes with a few empty experts: many tiles per
    workgroup, experts of very different K-tile counts and equal ones (ties)."""
    rng = np.random.default_rng(seed)
    p = 1.0 / np.arange(1, E + 1) ** 1.1
    cnt = np.floor(total * p / p.sum()).astype(np.int64)
    cnt = cnt[rng.permutation(E)]
    cnt[rng.choice(E, E // 16, replace=False)] = 0
    return [int(c) for c in cnt]


def test_grouped_gemm_ragged_k_many_tiles(q2d):
    """Weight gradients of 200 Zipf-sized experts (400 output tiles for 256
    workgroups, walked in the cost-sorted serpentine order): every expert
    against the oracle."""
    cnt = skewed_counts(200, 24000, 61)
    E = len(cnt)
    off = synth.segment_offsets(cnt)
    S = int(off[-1])
    Ng, K = 256, 512
    dY = synth.normal((S, Ng), 1e-3, 62, torch.bfloat16, device=DEV)
    X = synth.normal((S, K), 1.0, 63, torch.bfloat16, device=DEV)
    qdY, odY = quant_grouped(q2d, dY, off, "sr", 7, 2)
    qX, oX = quant_grouped(q2d, X, off, "rtn")
    dW = torch.full((E * Ng, K), 7.0, device=DEV)
    q2d.q2d_grouped_gemm(qdY, 1, qX, 1, dev_offsets(off), out=dW)
    dW = dW.cpu().numpy()
    dy_e, x_e = expert_slicer(odY, off, True), expert_slicer(oX, off, True)
    for e in range(E):
        rows = slice(e * Ng, (e + 1) * Ng)
        if off[e] == off[e + 1]:
            assert np.all(dW[rows] == 0), e
            continue
        ref = oracle.gemm(dy_e(e), x_e(e))
        assert rel_frob(dW[rows], ref) <= TOL, e


def test_grouped_gemm_ragged_m_many_tiles(q2d):
    """Forward GEMMs of 200 Zipf-sized experts with 768-wide outputs (3 column
    tiles: the XCD-contiguous tile order), several tiles per workgroup: every
    expert against the oracle, float32 and bf16 outputs."""
    cnt = skewed_counts(200, 24000, 71)
    E = len(cnt)
    off = synth.segment_offsets(cnt)
    S = int(off[-1])
    N, K = 768, 256
    X = synth.normal((S, K), 1.0, 72, torch.bfloat16, device=DEV)
    W = synth.normal((E * N, K), 0.02, 73, torch.bfloat16, device=DEV)
    qX, oX = quant_grouped(q2d, X, off, "rtn")
    qW = q2d.q2d_quantize(W, "rtn")
    oW = oracle.quantize_fp4_2d(W.cpu(), "rtn")
    Wf = oracle.operand(oW, False)
    Y = q2d.q2d_grouped_gemm(qX, 0, qW, 0, dev_offsets(off), out_dtype=torch.float32).cpu().numpy()
    Yb = q2d.q2d_grouped_gemm(qX, 0, qW, 0, dev_offsets(off), out_dtype=torch.bfloat16).cpu()
    x_e = expert_slicer(oX, off)
    for e in range(E):
        a, b = int(off[e]), int(off[e + 1])
        if a == b:
            continue
        ref = oracle.gemm(x_e(e), Wf[e * N:(e + 1) * N])
        assert rel_frob(Y[a:b], ref) <= TOL, e
        check_bf16(Yb[a:b], ref)


@pytest.mark.parametrize("pad,base", [(1, 0), (2, 1)])
def test_grouped_gemm_ragged_m_bf16_strided_output(q2d, pad, base):
    """bf16 ragged-M output into a view of a wider buffer with an odd row pitch or a
    base one element off (one store per element instead of pair stores): every
    expert against the oracle, the bytes outside the view unchanged."""
    cnt = skewed_counts(64, 12000, 81)
    E = len(cnt)
    off = synth.segment_offsets(cnt)
    S = int(off[-1])
    N, K = 768, 256
    X = synth.normal((S, K), 1.0, 82, torch.bfloat16, device=DEV)
    W = synth.normal((E * N, K), 0.02, 83, torch.bfloat16, device=DEV)
    qX, oX = quant_grouped(q2d, X, off, "rtn")
    qW = q2d.q2d_quantize(W, "rtn")
    Wf = oracle.operand(oracle.quantize_fp4_2d(W.cpu(), "rtn"), False)
    ld = N + pad
    flat = synth.normal((S * ld + 2,), 0.5, 84, torch.bfloat16, device=DEV)
    before = flat.clone()
    y = flat[base:base + S * ld].view(S, ld)[:, :N]
    q2d.q2d_grouped_gemm(qX, 0, qW, 0, dev_offsets(off), out=y)
    Yb = y.cpu()
    x_e = expert_slicer(oX, off)
    for e in range(E):
        a, b = int(off[e]), int(off[e + 1])
        if a < b:
            check_bf16(Yb[a:b], oracle.gemm(x_e(e), Wf[e * N:(e + 1) * N]))
    inside = torch.zeros(S * ld + 2, dtype=torch.bool, device=DEV)
    inside[base:base + S * ld].view(S, ld)[:, :N] = True
    assert torch.equal(flat.view(torch.int16)[~inside], before.view(torch.int16)[~inside])


def test_grouped_gemm_bf16_weight_gradient(q2d):
    off = synth.segment_offsets(COUNTS["edges"])
    E, S = len(COUNTS["edges"]), int(off[-1])
    dY = synth.normal((S, 128), 1e-3, 51, torch.bfloat16, device=DEV)
    X = synth.normal((S, 160), 1.0, 52, torch.bfloat16, device=DEV)
    qdY, odY = quant_grouped(q2d, dY, off, "sr", 2, 2)
    qX, oX = quant_grouped(q2d, X, off, "rtn")
    dW = q2d.q2d_grouped_gemm(qdY, 1, qX, 1, dev_offsets(off), out_dtype=torch.bfloat16).cpu()
    for e in range(E):
        if off[e] == off[e + 1]:
            continue
        ref = oracle.gemm(expert_rows(odY, off, e, True), expert_rows(oX, off, e, True))
        check_bf16(dW[e * 128:(e + 1) * 128], ref)


def _rows(o, rows):
    """float64 rows of the row-packed copy of an oracle quantization (padded row
    indices for a grouped one).  The column-packed copy holds the same values
    transposed, so these rows also give the operands of the transposed GEMMs."""
    C = o["cols"]
    codes = o["codes"][np.asarray(rows)]
    vals = oracle.fp4_values(np.stack([codes & 15, codes >> 4], -1).reshape(len(rows), -1)[:, :C])
    s = 2.0 ** (o["scales"][np.asarray(rows) // 32][:, np.arange(C) // 32].astype(np.float64) - 127)
    return vals * s


def test_full_moe_30b_launch_configuration(q2d):
    """The MoE expert FFN of the benchmark at full size (128 experts, 131072 token
    slots, hidden 2048, FFN 768): all six grouped GEMMs, bf16 activations and
    data gradients, fp32 weight gradients, 48 sampled output rows per GEMM
    checked against float64 products of the oracle's operands."""
    w = synth.moe_30b(device=DEV)
    off, E, Hd, F = w.extra["offsets"], w.extra["experts"], w.extra["hidden"], w.extra["ffn"]
    t = w.tensors
    doff = dev_offsets(off)
    rng = np.random.default_rng(1)
    ops = {}
    for k in ("X", "H", "dY_gu", "dY_d"):
        print("moe_30b quantize %s" % k, flush=True)
        ops[k] = quant_grouped(q2d, t[k], off, w.rounding[k], w.seed, 3)
    for k in ("W_gu", "W_d"):
        print("moe_30b quantize %s" % k, flush=True)
        q = q2d.q2d_quantize(t[k], w.rounding[k], w.seed, 3)
        o = oracle.quantize_fp4_2d(t[k].cpu(), w.rounding[k], w.seed, 3)
        assert_same_bytes(gpu_buffers(q), o, k)
        ops[k] = (q, o)
    pad = oracle.grouped_rows(off)
    slot_e = np.searchsorted(off, np.arange(int(off[-1])), side="right") - 1

    def segment(o, e):
        return _rows(o, np.arange(pad[e], pad[e] + off[e + 1] - off[e]))

    def ragged_m(a, b, transB, nb, label):
        (qa, oa), (qb, ob) = ops[a], ops[b]
        print("moe_30b %s" % label, flush=True)
        Y = q2d.q2d_grouped_gemm(qa, 0, qb, transB, doff, out_dtype=torch.bfloat16)
        rows = np.sort(rng.choice(int(off[-1]), 48, replace=False))
        e = slot_e[rows]
        A = _rows(oa, pad[e] + rows - off[e])
        ref = np.empty((len(rows), Y.shape[1]))
        for ex in np.unique(e):
            We = _rows(ob, np.arange(ex * nb, (ex + 1) * nb))      # expert weights [nb, cols]
            sel = e == ex
            ref[sel] = A[sel] @ (We if transB else We.T)
        check_bf16(Y[torch.from_numpy(rows).to(DEV)], ref)

    def ragged_k(a, b, label):
        (qa, oa), (qb, ob) = ops[a], ops[b]
        print("moe_30b %s" % label, flush=True)
        dW = q2d.q2d_grouped_gemm(qa, 1, qb, 1, doff, out_dtype=torch.float32)
        M = oa["cols"]
        rows = np.sort(rng.choice(E * M, 48, replace=False))
        got = dW[torch.from_numpy(rows).to(DEV)].cpu().numpy()
        ref = np.zeros((len(rows), ob["cols"]))
        for ex in np.unique(rows // M):
            if off[ex] == off[ex + 1]:
                continue
            sel = rows // M == ex
            ref[sel] = segment(oa, ex)[:, rows[sel] % M].T @ segment(ob, ex)
        assert rel_frob(got, ref) <= TOL

    ragged_m("X", "W_gu", 0, 2 * F, "gate/up forward")
    ragged_m("H", "W_d", 0, Hd, "down forward")
    ragged_m("dY_d", "W_d", 1, Hd, "down data gradient")
    ragged_m("dY_gu", "W_gu", 1, 2 * F, "gate/up data gradient")
    ragged_k("dY_gu", "X", "gate/up weight gradient")
    ragged_k("dY_d", "H", "down weight gradient")
    del ops, w
    torch.cuda.empty_cache()


# ------------------------------------------------------------------ offsets the host cannot check

# (device offsets, rows): descending entries, negative entries, entries beyond
# the row count, a first entry above 0 and a last entry below the row count
BAD_OFFSETS = [([-5, 100, 60, 300, 900, 650, 700], 700),
               ([0, 50, 40, 200, 150], 260),
               ([10, 500, 400, 420], 300)]


def sanitized(off, rows):
    """The table the kernels use: o'[i] = min(max(0, off[0..i]), rows)."""
    return np.minimum(np.maximum.accumulate(np.maximum(np.asarray(off, np.int64), 0)), rows)


@pytest.mark.parametrize("case", range(len(BAD_OFFSETS)))
def test_invalid_offsets_stay_in_bounds(q2d, case):
    """Offsets live on the device, so the C ABI cannot reject a bad table before
    the launch.  The kernels use its sanitized form (ascending, inside
    [0, rows]): the quantizer and both grouped GEMMs then give exactly the
    results of that table, and nothing outside the buffers is touched."""
    off, S = BAD_OFFSETS[case]
    good = sanitized(off, S)
    E = len(off) - 1
    K, N = 256, 96
    X = synth.normal((S, K), 1.0, 61 + case, torch.bfloat16, device=DEV)
    dY = synth.normal((S, N), 1e-3, 62 + case, torch.bfloat16, device=DEV)
    W = synth.normal((E * N, K), 0.02, 63, torch.bfloat16, device=DEV)
    qX = q2d.q2d_grouped_quantize(X, dev_offsets(off), "rtn")
    qdY = q2d.q2d_grouped_quantize(dY, dev_offsets(off), "rtn")
    # the oracle's grouped form starts at row 0: hand it the rows the table covers
    lo, hi = int(good[0]), int(good[-1])
    oX = oracle.quantize_fp4_grouped(X.cpu()[lo:hi], good - lo, "rtn")
    odY = oracle.quantize_fp4_grouped(dY.cpu()[lo:hi], good - lo, "rtn")
    assert_grouped_equal(qX, oX, "X")
    assert_grouped_equal(qdY, odY, "dY")
    qW = q2d.q2d_quantize(W, "rtn")
    Wf = oracle.operand(oracle.quantize_fp4_2d(W.cpu(), "rtn"), False)
    Y = torch.full((S, N), 3.0, device=DEV)
    q2d.q2d_grouped_gemm(qX, 0, qW, 0, dev_offsets(off), out=Y)
    dW = torch.full((E * N, K), 3.0, device=DEV)
    q2d.q2d_grouped_gemm(qdY, 1, qX, 1, dev_offsets(off), out=dW)
    Y, dW = Y.cpu().numpy(), dW.cpu().numpy()
    for e in range(E):
        a, b = int(good[e]), int(good[e + 1])
        rows = slice(e * N, (e + 1) * N)
        if a == b:
            assert np.all(dW[rows] == 0)
            continue
        ref = oracle.gemm(expert_rows(oX, good - lo, e), Wf[e * N:(e + 1) * N])
        assert rel_frob(Y[a:b], ref) <= TOL, e
        refw = oracle.gemm(expert_rows(odY, good - lo, e, True), expert_rows(oX, good - lo, e, True))
        assert rel_frob(dW[rows], refw) <= TOL, e
    # rows outside every segment are left as they were
    assert np.all(Y[:lo] == 3.0) and np.all(Y[hi:] == 3.0)
