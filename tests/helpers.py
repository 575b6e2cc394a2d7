"""Shared helpers of the GPU parity tests (comparison only; no method arithmetic)."""
import numpy as np
import torch

BUFS = ("codes", "codes_t", "scales", "scales_t")


def gpu_buffers(q) -> dict:
    torch.cuda.synchronize()
    return {k: getattr(q, k).cpu().numpy() for k in BUFS if getattr(q, k) is not None}


def poison(q, value: int = 0xAA):
    """Fill every output buffer with a marker so that unwritten bytes show up."""
    for k in BUFS:
        t = getattr(q, k)
        if t is not None:
            t.fill_(value)


def assert_same_bytes(got: dict, want: dict, label: str = ""):
    for k in BUFS:
        if k not in got:
            continue
        g, w = got[k], want[k]
        assert g.shape == w.shape, (label, k, g.shape, w.shape)
        if not np.array_equal(g, w):
            bad = np.argwhere(g != w)
            r, c = bad[0]
            raise AssertionError("%s %s: %d bytes differ, first at (%d, %d): gpu %#04x oracle %#04x"
                                 % (label, k, len(bad), r, c, g[r, c], w[r, c]))


def rel_frob(got: np.ndarray, ref: np.ndarray) -> float:
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    den = np.linalg.norm(ref)
    return float(np.linalg.norm(got - ref) / (den if den > 0 else 1.0))


def as_oracle_tensor(q, rows, cols, fmt="fp4") -> dict:
    """Oracle-style dict of a device QTensor (bytes copied to the host)."""
    d = gpu_buffers(q)
    d["rows"], d["cols"] = rows, cols
    return d


def grouped_written(q, P: int) -> dict:
    """Host copy of the written region (the first P padded rows) of a grouped tensor."""
    torch.cuda.synchronize()
    return {"codes": q.codes[:P].cpu().numpy(), "scales": q.scales[:P // 32].cpu().numpy(),
            "codes_t": q.codes_t[:, :P // 2].cpu().numpy(),
            "scales_t": q.scales_t[:, :P // 32].cpu().numpy()}


def check_bf16(got, ref):
    """bf16 output = RNE(fp32 accumulation): within 2^-9 |ref| of the fp32 value, which is
    itself within the fp32 accumulation error (taken as 1e-5 * rms(ref)) of the exact result."""
    got = got.float().cpu().numpy().astype(np.float64)
    err = np.abs(got - ref)
    rms = float(np.sqrt(np.mean(ref * ref))) if ref.size else 0.0
    tol = np.abs(ref) * 2.0 ** -8 + 1e-5 * rms + 1e-38
    assert np.all(err <= tol), float((err / tol).max())
