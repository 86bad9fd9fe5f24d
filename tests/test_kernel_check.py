"""CPU checks of the acceptance rule the kernel-by-kernel GPU test applies: a
bf16 result must be the rounding of a value within the stated arithmetic error
bound of the exact one, an fp32 result within its bound.  Correct roundings
pass, near-ties rounded the other way pass, a value off by more than its bound
fails."""
import numpy as np
import pytest

from oracle.numerics import round_bf16
from test_gpu_kernels import check_bf16, check_f32


def bits(x):
    """bf16 bit patterns of values that are exact bf16 numbers."""
    return (np.asarray(x, dtype=np.float32).view(np.uint32) >> 16).astype(np.uint16)


def padded(y, got, bound, n=200):
    """One checked element among n - 1 exactly rounded ones (the rule allows at
    most 1% of a step's elements off the exact rounding)."""
    rest = np.linspace(0.5, 2.0, n - 1)
    return (np.concatenate([got, bits(round_bf16(rest))]), np.concatenate([y, rest]),
            np.concatenate([bound, 1e-12 * rest]))


def test_exact_roundings_pass():
    rng = np.random.default_rng(0)
    y = rng.normal(size=1000)
    stats = {}
    check_bf16("t", bits(round_bf16(y)), y, 1e-12 * np.abs(y), stats)
    assert stats["t"][0] == 0


def test_a_near_tie_rounded_the_other_way_passes():
    # 1 + 2^-8 + tiny lies just above the midpoint between 1 and 1 + 2^-7
    y = np.array([1.0 + 2.0 ** -8 + 1e-9])
    other = bits([1.0])                         # the neighbour below
    stats = {}
    check_bf16("t", *padded(y, other, np.array([1e-8])), stats)
    assert stats["t"][0] == 1 and stats["t"][2] <= 1.0
    with pytest.raises(AssertionError):         # the bound does not reach the midpoint
        check_bf16("t", *padded(y, other, np.array([1e-10])), {})


def test_a_value_off_by_more_than_its_bound_fails():
    y = np.array([1.5])
    with pytest.raises(AssertionError):                                   # two ulps away
        check_bf16("t", *padded(y, bits([1.5 + 2 * 2.0 ** -7]), np.array([1e-4])), {})
    with pytest.raises(AssertionError):
        check_f32("t", np.array([1.0 + 2e-4]), np.array([1.0]), np.array([1e-4]), {})


def test_a_value_near_zero_within_a_wide_bound_passes():
    # cancellation: the bound spans many ulps of a tiny exact value
    y = np.array([6.06e-7])
    got = bits(round_bf16(np.array([7.8e-7])))
    check_bf16("t", *padded(y, got, np.array([1.6e-3])), {})
    with pytest.raises(AssertionError):
        check_bf16("t", *padded(y, got, np.array([1e-9])), {})


def test_fp32_results_within_bound_and_bar_pass():
    stats = {}
    check_f32("t", np.array([1.0 + 1e-6]), np.array([1.0]), np.array([1e-5]), stats)
    assert stats["t"][0] == pytest.approx(1e-6)
