"""Pins of the oracle's Philox4x32-10 stream (the random source of stochastic
rounding, Sec. 3.1 and App. E) against rocRAND's independent host
implementation (compiled here from the ROCm headers), including counter and
key carries across 2^32, and a uniformity check of the 16-bit draws."""
import os
import shutil
import subprocess

import numpy as np
import pytest

import oracle

HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.fixture(scope="module")
def rocrand_ref(tmp_path_factory):
    hdr = "/opt/rocm/include/rocrand/rocrand_philox4x32_10.h"
    if not os.path.exists(hdr) or shutil.which("g++") is None:
        pytest.skip("rocRAND headers or g++ not available")
    exe = str(tmp_path_factory.mktemp("rr") / "rr")
    subprocess.check_call(["g++", "-O1", "-I/opt/rocm/include", "-D__HIP_PLATFORM_AMD__",
                           os.path.join(HERE, "rocrand_philox_ref.cpp"), "-o", exe])
    return exe


def test_counter_mapping_matches_rocrand(rocrand_ref):
    rng = np.random.default_rng(7)
    cases = [(0, 0, 0), (0, 0, 1), (1, 0, 0), (0, 1, 0),
             (2**32 - 1, 2**32 - 1, 2**32 - 1), (2**32, 2**32, 2**32),
             (2**64 - 1, 2**64 - 1, 2**61 - 1), (12345678901234, 987654321, 2**40 + 3)]
    for _ in range(200):
        cases.append((int(rng.integers(0, 2**63)), int(rng.integers(0, 2**63)),
                      int(rng.integers(0, 2**60))))
    inp = "".join("%d %d %d\n" % c for c in cases)
    out = subprocess.run([rocrand_ref], input=inp, capture_output=True, text=True,
                         check=True).stdout.split("\n")
    for (seed, off, g), line in zip(cases, out):
        want = [int(t, 16) for t in line.split()]
        got = oracle.philox4x32_10([g & 0xFFFFFFFF, g >> 32, off & 0xFFFFFFFF, off >> 32],
                                   [seed & 0xFFFFFFFF, seed >> 32])
        assert [int(v) for v in got] == want, (seed, off, g)
        # the per-element 16-bit draws of the eight storage indices 8g .. 8g+7
        for j in range(8):
            r16 = oracle.sr_bits(8 * g + j, seed, off)
            assert r16 == (want[j >> 1] >> (16 * (j & 1))) & 0xFFFF


def test_halves_uniform():
    """Chi-square of the 16-bit draws' top 6 bits over 2^15 consecutive indices."""
    vals = np.array([oracle.sr_bits(i, 11, 5) for i in range(1 << 15)], dtype=np.int64)
    counts = np.bincount(vals >> 10, minlength=64)
    exp = len(vals) / 64
    chi2 = float(((counts - exp) ** 2 / exp).sum())
    assert chi2 < 130.0     # 63 dof: P(chi2 > 130) < 1e-6
