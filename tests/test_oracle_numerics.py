"""Pins for the oracle's storage-format rounding against library conversions and
hand-worked values (IEEE-754 round-to-nearest-even)."""
import numpy as np
import pytest
import torch

from oracle.numerics import round_bf16, round_f16, round_f32


def _bf16_ties():
    # 1 + k/256 for odd k sit exactly halfway between bfloat16 neighbours near 1.
    return np.array([1 + k / 256 for k in range(1, 32, 2)] + [-(1 + k / 256) for k in range(1, 32, 2)])


def test_bf16_hand_values():
    assert round_bf16(1 + 2 ** -8) == 1.0                 # tie, even neighbour is 1.0
    assert round_bf16(1 + 3 * 2 ** -8) == 1 + 2 ** -6     # tie, even neighbour rounds up
    assert round_bf16(1 + 2 ** -8 + 2 ** -30) == 1 + 2 ** -7   # just above the tie
    assert round_bf16(3.0) == 3.0
    assert round_bf16(0.0) == 0.0
    assert np.isinf(round_bf16(3.5e38))
    assert round_bf16(-2 ** -133) == -2 ** -133           # smallest subnormal
    assert round_bf16(2 ** -135) == 0.0                   # below half the smallest subnormal


def test_bf16_matches_torch_conversion():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(20000) * 10.0 ** rng.integers(-30, 30, 20000),
                        _bf16_ties()]).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(round_bf16(x.astype(np.float64)), ref)


def test_f16_matches_numpy_conversion():
    rng = np.random.default_rng(1)
    x = np.concatenate([rng.standard_normal(20000) * 10.0 ** rng.integers(-9, 6, 20000),
                        [65504.0, 65520.0, 65519.99, 2.0 ** -24, 2.0 ** -25, 3 * 2.0 ** -26,
                         1 + 2 ** -11, 1 + 3 * 2 ** -11]])
    with np.errstate(over="ignore"):
        ref = x.astype(np.float16).astype(np.float64)
    np.testing.assert_array_equal(round_f16(x), ref)


def test_f32_matches_numpy_conversion():
    rng = np.random.default_rng(2)
    x = rng.standard_normal(20000) * 10.0 ** rng.integers(-40, 38, 20000)
    np.testing.assert_array_equal(round_f32(x), x.astype(np.float32).astype(np.float64))
