"""The library under HIP graph capture: a quantized linear layer's forward and
backward (quantizers and GEMMs, including the quantizing epilogue) captured on
torch's current stream, replayed several times with eager work and
synchronisations in between; every replay must reproduce the eager results
bit for bit (the kernels are deterministic: no atomics, fixed reduction
order).  The library allocates nothing and issues no memset, so nothing in a
captured call depends on host state.
"""
import pytest
import torch

import synth

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


@pytest.fixture(scope="module")
def q2d():
    import paper_2607_24953_amd as q
    return q


def test_linear_layer_graph_replays(q2d):
    T, N, K = 512, 768, 640
    X = synth.normal((T, K), 1.0, 81, torch.bfloat16, device=DEV)
    W = synth.normal((N, K), 0.02, 82, torch.bfloat16, device=DEV)
    dY = synth.normal((T, N), 1e-3, 83, torch.bfloat16, device=DEV)
    qX = q2d.QTensor(q2d.FP4_2D, T, K, DEV)
    qW = q2d.QTensor(q2d.FP4_2D, N, K, DEV)
    qdY = q2d.QTensor(q2d.FP4_2D, T, N, DEV)
    qY = q2d.QTensor(q2d.FP4_2D, T, N, DEV)
    Y = torch.empty((T, N), dtype=torch.float32, device=DEV)
    dX = torch.empty((T, K), dtype=torch.bfloat16, device=DEV)
    dW = torch.empty((N, K), dtype=torch.float32, device=DEV)

    def step():
        q2d.q2d_linear_fwd(X, W, "rtn", "rtn", 5, 0, 1, torch.float32, qX=qX, qW=qW, Y=Y)
        q2d.q2d_linear_bwd(dY, qX, qW, "sr", 5, 2, torch.bfloat16, torch.float32, dW=dW, qdY=qdY, dX=dX)
        q2d.q2d_gemm_quantized(qX, 0, qW, 0, "rtn", out=qY)

    def snapshot():
        torch.cuda.synchronize()
        out = {"Y": Y.clone(), "dX": dX.clone(), "dW": dW.clone()}
        for name, q in (("qX", qX), ("qW", qW), ("qdY", qdY), ("qY", qY)):
            for k in ("codes", "codes_t", "scales", "scales_t"):
                out[name + "." + k] = getattr(q, k).clone()
        return out

    step()
    want = snapshot()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        step()                                         # warm-up on the capture stream
    torch.cuda.current_stream().wait_stream(s)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    for rep in range(3):
        for t in (Y, dX, dW):
            t.fill_(float("nan"))
        for q in (qX, qW, qdY, qY):
            q.codes.fill_(0xAA)
            q.codes_t.fill_(0xAA)
        torch.cuda.synchronize()
        _ = torch.randn(1000, device=DEV).sum().item()    # eager work between replays
        g.replay()
        got = snapshot()
        for k, v in want.items():
            assert torch.equal(got[k].view(torch.uint8) if got[k].dtype != torch.uint8 else got[k],
                               v.view(torch.uint8) if v.dtype != torch.uint8 else v), (rep, k)


def test_grouped_and_mxfp8_graph_replays(q2d):
    """The MoE expert GEMMs (grouped quantizer, ragged-M and ragged-K grouped GEMMs)
    and an MXFP8 GEMM under capture: every replay equals the eager results."""
    counts = [0, 1, 300, 31, 33, 700, 0, 127, 515]
    off = torch.tensor([0] + list(torch.tensor(counts).cumsum(0).tolist()), dtype=torch.int64, device=DEV)
    E, S, Hd, F = len(counts), sum(counts), 256, 384
    X = synth.normal((S, Hd), 1.0, 91, torch.bfloat16, device=DEV)
    Wg = synth.normal((E * F, Hd), 0.02, 92, torch.bfloat16, device=DEV)
    dY = synth.normal((S, F), 1e-3, 93, torch.bfloat16, device=DEV)
    X8 = synth.normal((512, 640), 1.0, 94, torch.bfloat16, device=DEV)
    W8 = synth.normal((384, 640), 0.02, 95, torch.bfloat16, device=DEV)
    qX = q2d.QTensor(q2d.FP4_2D, S, Hd, DEV, nseg=E)
    qdY = q2d.QTensor(q2d.FP4_2D, S, F, DEV, nseg=E)
    qW = q2d.QTensor(q2d.FP4_2D, E * F, Hd, DEV)
    qX8 = q2d.QTensor(q2d.MXFP8, 512, 640, DEV)
    qW8 = q2d.QTensor(q2d.MXFP8, 384, 640, DEV)
    Y = torch.empty((S, F), dtype=torch.bfloat16, device=DEV)
    dX = torch.empty((S, Hd), dtype=torch.bfloat16, device=DEV)
    dW = torch.empty((E * F, Hd), dtype=torch.float32, device=DEV)
    Y8 = torch.empty((512, 384), dtype=torch.float32, device=DEV)

    def step():
        q2d.q2d_grouped_quantize(X, off, "rtn", 3, 0, out=qX)
        q2d.q2d_grouped_quantize(dY, off, "sr", 3, 1, out=qdY)
        q2d.q2d_quantize(Wg, "rtn", 3, 2, out=qW)
        q2d.q2d_grouped_gemm(qX, 0, qW, 0, off, out=Y)
        q2d.q2d_grouped_gemm(qdY, 0, qW, 1, off, out=dX)
        q2d.q2d_grouped_gemm(qdY, 1, qX, 1, off, out=dW)
        q2d.mxfp8_quantize(X8, out=qX8)
        q2d.mxfp8_quantize(W8, out=qW8)
        q2d.q2d_gemm(qX8, 0, qW8, 0, out=Y8)

    outs = {"Y": Y, "dX": dX, "dW": dW, "Y8": Y8}
    qts = {"qX": qX, "qdY": qdY, "qW": qW, "qX8": qX8, "qW8": qW8}

    def snapshot():
        torch.cuda.synchronize()
        out = {k: v.clone() for k, v in outs.items()}
        for name, q in qts.items():
            for k in ("codes", "codes_t", "scales", "scales_t"):
                out[name + "." + k] = getattr(q, k).clone()
        return out

    def poison():
        # the grouped layouts hold capacity rows no call writes: both the eager
        # reference and every replay start from the same bytes there
        for t in outs.values():
            t.fill_(float("nan"))
        for q in qts.values():
            q.codes.fill_(0xAA)
            q.codes_t.fill_(0xAA)
            q.scales.fill_(0x55)
            q.scales_t.fill_(0x55)

    poison()
    step()
    want = snapshot()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        step()
    torch.cuda.current_stream().wait_stream(s)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    for rep in range(3):
        poison()
        torch.cuda.synchronize()
        _ = torch.randn(1000, device=DEV).sum().item()    # eager work between replays
        g.replay()
        got = snapshot()
        for k, v in want.items():
            a = got[k].view(torch.uint8) if got[k].dtype != torch.uint8 else got[k]
            b = v.view(torch.uint8) if v.dtype != torch.uint8 else v
            assert torch.equal(a, b), (rep, k)
