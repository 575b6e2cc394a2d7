"""Pins of the oracle's element codecs against brute force and exact arithmetic.

* Truncation-free scale (Sec. 3.1, App. D): for every positive finite bfloat16
  block maximum M, the exponent is the smallest e with 6 * 2^e >= M, checked
  with exact rationals (no saturation: M / 2^e <= 6; minimality: M / 2^(e-1) > 6
  unless the clamp at -127 is hit).
* Round to nearest (App. E): every bfloat16 value x times every exponent e in
  [-12, 12] against an arg-min over the E2M1 grid, ties to the even code.
* Stochastic rounding (Sec. 3.1, App. E): enumerating all 2^16 random draws
  gives exactly floor(2^16 d / delta) round-ups, so the mean is the input to
  within delta * 2^-16 (exactly the input when d / delta has <= 16 fraction bits).
* E4M3 (Sec. 3.2): against torch's float8_e4m3fn cast of the exact value.
"""
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle

GRID = [Fraction(0), Fraction(1, 2), Fraction(1), Fraction(3, 2), Fraction(2), Fraction(3),
        Fraction(4), Fraction(6)]


def all_bf16_finite():
    bits = np.arange(1 << 16, dtype=np.uint32)
    f = (bits << 16).view(np.float32)
    return f[np.isfinite(f)].astype(np.float64)


def _exact(x: float) -> Fraction:
    return Fraction(x)


def test_scale_exponent_exhaustive_bf16():
    xs = all_bf16_finite()
    Ms = np.unique(np.abs(xs))
    for M in Ms:
        e = oracle.fp4_scale_exponent(M)
        fm = _exact(M)
        assert -127 <= e <= 127
        assert 6 * Fraction(2) ** e >= fm                     # no saturation
        if e > -127:
            assert 6 * Fraction(2) ** (e - 1) < fm             # minimal


def test_scale_exponent_fp32_edges():
    rng = np.random.default_rng(3)
    vals = list(rng.standard_normal(20000).astype(np.float32) * 10.0 ** rng.integers(-30, 30, 20000))
    for k in range(-149, 128):
        for m in (1.0, 1.5, 1.75, 1.25):
            v = np.float32(np.ldexp(m, k))
            if np.isfinite(v) and v > 0:
                vals += [v, np.nextafter(v, np.float32(np.inf)), np.nextafter(v, np.float32(0))]
    vals.append(np.finfo(np.float32).max)
    for v in vals:
        M = abs(float(v))
        if M == 0 or not np.isfinite(M):
            continue
        e = oracle.fp4_scale_exponent(M)
        assert 6 * Fraction(2) ** e >= Fraction(M)
        if e > -127:
            assert 6 * Fraction(2) ** (e - 1) < Fraction(M)
    assert oracle.fp4_scale_exponent(0.0) == -127


def test_fp8_scale_exponent():
    for M in np.unique(np.abs(all_bf16_finite()))[::7]:
        e = oracle.fp8_scale_exponent(M)
        assert 448 * Fraction(2) ** e >= Fraction(M)
        if e > -127:
            assert 448 * Fraction(2) ** (e - 1) < Fraction(M)


def _rtn_bruteforce(x: np.ndarray, e: int) -> np.ndarray:
    """Nearest signed E2M1 value * 2^e by arg-min; ties to the even magnitude code."""
    mags = np.array([float(g) for g in GRID])
    v = np.abs(x) * 2.0 ** (-e)
    d = np.abs(v[:, None] - mags[None, :])
    best = d.min(axis=1, keepdims=True)
    cand = d == best
    # among tied candidates take the even index (two ties always straddle odd/even)
    even = cand & (np.arange(8)[None, :] % 2 == 0)
    idx = np.where(even.any(axis=1), even.argmax(axis=1), cand.argmax(axis=1))
    sign = np.signbit(x).astype(np.int64)
    return (sign << 3 | idx).astype(np.uint8)


@pytest.mark.parametrize("e", list(range(-12, 13)))
def test_rtn_exhaustive_bf16(e):
    xs = all_bf16_finite()
    xs = xs[np.abs(xs) * 2.0 ** (-e) <= 6]      # the codec's domain under truncation-free scaling
    got = oracle.fp4_codes(xs, e)
    np.testing.assert_array_equal(got, _rtn_bruteforce(xs, e))


def test_rtn_fp32_midpoints():
    mids = [0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0]
    xs = []
    for m in mids + [0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0]:
        f = np.float32(m)
        xs += [f, np.nextafter(f, np.float32(0)), np.nextafter(f, np.float32(10))]
    rng = np.random.default_rng(0)
    xs += list((rng.random(200000) * 6).astype(np.float32))
    xs = np.array(xs, dtype=np.float64)
    xs = np.concatenate([xs, -xs])
    for e in (-3, 0, 5):
        got = oracle.fp4_codes(xs * 2.0 ** e, e)
        np.testing.assert_array_equal(got, _rtn_bruteforce(xs * 2.0 ** e, e))
    # the tie rule spelled out: 0.25->0, 0.75->1.0, 1.25->1.0, 1.75->2, 2.5->2, 3.5->4, 5->4
    assert [oracle.fp4_code(m, 0) for m in mids] == [0, 2, 2, 4, 4, 6, 6]
    assert oracle.fp4_code(-0.1, 0) == 8          # sign kept at zero magnitude


def _floor_index(v: Fraction) -> int:
    return max(k for k in range(8) if GRID[k] <= v)


@pytest.mark.parametrize("x", [0.1, 0.3, 0.6, 0.74, 1.1, 1.6, 2.2, 2.9, 3.3, 4.4, 5.9,
                               1.0 / 3.0, 0.7001953125, 5.75, 1e-3, 3.0, 6.0])
def test_sr_enumeration_counts(x):
    """Over all 2^16 draws the round-up count equals floor(2^16 * d / delta)."""
    xf = float(np.float32(x))
    v = Fraction(xf)
    k = _floor_index(v)
    codes = oracle.fp4_codes(np.full(1 << 16, xf), 0, True, np.arange(1 << 16, dtype=np.uint32))
    mags = codes & 7
    assert set(np.unique(mags)).issubset({k, min(k + 1, 7)})
    ups = int((mags == k + 1).sum()) if k < 7 else 0
    if k == 7:
        assert ups == 0
        return
    d = v - GRID[k]
    delta = GRID[k + 1] - GRID[k]
    F = (d / delta * 65536).__floor__()
    assert ups == F
    mean = GRID[k] + delta * Fraction(ups, 65536)
    assert abs(mean - v) <= delta / 65536
    if (d / delta * 65536).denominator == 1:
        assert mean == v


def test_sr_exact_on_bf16_grid():
    """For bfloat16 inputs with v >= 2^-10 the 16-bit contract is exactly unbiased."""
    xs = all_bf16_finite()
    xs = xs[(np.abs(xs) >= 2.0 ** -10) & (np.abs(xs) <= 6)]
    v = np.abs(xs)
    k = np.searchsorted(np.array([float(g) for g in GRID]), v, side="right") - 1
    delta = np.array([0.5, 0.5, 0.5, 0.5, 1, 1, 2, 2])[k]
    frac = (v - np.array([float(g) for g in GRID])[k]) / delta * 65536
    assert np.all(frac == np.floor(frac))


def test_sr_statistical_unbiased():
    """10^6 draws of the real Philox stream: |mean error| within 5 sigma + delta 2^-16."""
    n = 1_000_000
    xs = np.float64(np.float32(0.3))
    idx = np.arange(n, dtype=np.int64)
    r16 = np.array([oracle.sr_bits(int(i), 1, 0) for i in idx[:n // 10]], dtype=np.uint32)
    # draws for the remaining indices come from further offsets of the same stream
    parts = [r16]
    for off in range(1, 10):
        parts.append(np.array([oracle.sr_bits(int(i), 1, off) for i in idx[:n // 10]],
                              dtype=np.uint32))
    r = np.concatenate(parts)
    codes = oracle.fp4_codes(np.full(n, xs), 0, True, r)
    vals = oracle.fp4_values(codes)
    err = vals - xs
    sigma = err.std()
    assert abs(err.mean()) <= 5 * sigma / np.sqrt(n) + 0.5 * 2.0 ** -16


def test_e4m3_against_torch_cast():
    xs = all_bf16_finite()
    for e in (-9, -3, 0, 2, 7):
        v = xs[np.abs(xs) * 2.0 ** (-e) <= 448]
        got = oracle.e4m3_codes(v, e)
        ref = torch.from_numpy((v * 2.0 ** (-e)).astype(np.float32)).to(torch.float8_e4m3fn)
        ref = ref.view(torch.uint8).numpy()
        np.testing.assert_array_equal(got, ref)


def _golden_examples():
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden",
                        "scale_and_round_examples.txt")
    rows = []
    with open(path) as f:
        for line in f:
            line = line.split("#", 1)[0].split()
            if line:
                rows.append(line)
    return rows


def test_hand_derived_examples():
    """Worked examples derived by hand from the scale rule (Sec. 3.1; App. D) and the
    rounding rules (App. E); each line of the fixture states its derivation."""
    rows = _golden_examples()
    kinds = [r[0] for r in rows]
    assert kinds.count("scale") >= 8 and kinds.count("rtn") >= 10 and kinds.count("sr") >= 10
    for r in rows:
        if r[0] == "scale":
            M, e, byte = float(r[1]), int(r[2]), int(r[3], 16)
            got = oracle.fp4_scale_exponent(M)
            assert got == e, r
            assert got + 127 == byte, r
        elif r[0] == "rtn":
            assert oracle.fp4_code(float(r[1]), int(r[2])) == int(r[3], 16), r
        elif r[0] == "sr":
            assert oracle.fp4_code(float(r[1]), int(r[2]), True, int(r[3])) == int(r[4], 16), r
        else:
            raise AssertionError(r)
