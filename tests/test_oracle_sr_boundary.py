"""The oracle's stochastic rounding at its exact threshold (App. E): an element
with F = 2^16 - r16 rounds up, one with F = 2^16 - r16 - 1 does not, for every
grid interval, both signs and both nibbles of a byte, in both stored copies."""
import numpy as np
import pytest
import torch

import oracle
from sr_boundary import boundary_input, unpack


@pytest.mark.parametrize("seed,offset", [(0, 0), (0x123456789ABCDEF, 2 ** 32 + 5)])
def test_2d_threshold(seed, offset):
    rng = np.random.default_rng(seed & 0xFFFF)
    x, want = boundary_input(70, 96, seed, offset, rng)
    q = oracle.quantize_fp4_2d(torch.from_numpy(x), "sr", seed, offset)
    assert np.array_equal(unpack(q["codes"], 70, 96), want)
    assert np.array_equal(unpack(q["codes_t"], 96, 70), want.T)
    # the input covers both sides of the threshold, every interval and both nibbles
    assert len(np.unique(want & 7)) == 8


def test_1d_threshold():
    rng = np.random.default_rng(3)
    x, want = boundary_input(64, 96, 7, 11, rng)
    q = oracle.quantize_fp4_1d(torch.from_numpy(x), "sr", 7, 11)
    assert np.array_equal(unpack(q["codes"], 64, 96), want)
    assert np.array_equal(unpack(q["codes_t"], 96, 64), want.T)
