"""Inputs placed exactly at the stochastic-rounding threshold (test helper).

The SR contract (App. E): an element with scaled magnitude v = G[k] + d,
0 <= d < Delta = G[k+1] - G[k], rounds up iff floor(2^16 d / Delta) + r16 >= 2^16,
where r16 is the element's 16-bit Philox draw (keyed by its storage index).
For every element this builds v with F = floor(2^16 d / Delta) equal to
2^16 - r16 (the smallest F that rounds up) or 2^16 - r16 - 1 (the largest
that does not), so every element sits on one side of its own threshold.  The
values are exact in float32 (at most 20 significant bits).

Each 32 x 32 tile carries 6 * 2^e on its diagonal, so every 32 x 32 block, every
1 x 32 row segment and every 32 x 1 column segment has maximum 6 * 2^e and scale
exponent e; the diagonal elements are grid points (code 7)."""
import numpy as np

import oracle

G = np.array([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0])


def boundary_input(R: int, C: int, seed: int, offset: int, rng, exps=(-3, 0, 7, -30, 20)):
    """(x float32 [R, C] row-major, expected magnitude index [R, C]); the block
    exponents cycle through `exps` over the 32 x 32 tiles."""
    idx = np.arange(R * C, dtype=np.int64).reshape(R, C)
    r16 = np.array([oracle.sr_bits(int(i), seed, offset) for i in idx.ravel()], np.int64).reshape(R, C)
    k = rng.integers(0, 7, size=(R, C))
    up = (rng.random((R, C)) < 0.5) & (r16 > 0)
    F = np.where(up, 65536 - r16, 65535 - r16)
    v = G[k] + F * (G[k + 1] - G[k]) / 65536.0
    mag = np.where(up, k + 1, k)
    ti = (np.arange(R) // 32)[:, None] + 3 * (np.arange(C) // 32)[None, :]
    e = np.asarray(exps)[ti % len(exps)]
    diag = (np.arange(R) % 32)[:, None] == (np.arange(C) % 32)[None, :]
    v = np.where(diag, 6.0, v)
    mag = np.where(diag, 7, mag)
    sign = np.where(rng.random((R, C)) < 0.5, -1.0, 1.0)
    x = (sign * np.ldexp(v, e)).astype(np.float32)
    assert np.array_equal(x.astype(np.float64), sign * np.ldexp(v, e))     # exact in float32
    code = mag + np.where(sign < 0, 8, 0)
    return x, code


def unpack(packed: np.ndarray, rows: int, cols: int) -> np.ndarray:
    u = np.empty((packed.shape[0], packed.shape[1] * 2), np.uint8)
    u[:, 0::2] = packed & 15
    u[:, 1::2] = packed >> 4
    return u[:rows, :cols]
