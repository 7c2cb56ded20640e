"""Self-tests of the parity checker: a zero or slightly wrong output must fail."""
import numpy as np
import pytest

from parity import check, check_out


def test_zero_output_fails_the_bf16_check():
    rng = np.random.default_rng(0)
    ref = rng.standard_normal((32, 64)) * 0.03      # typical near-uniform attention output
    with pytest.raises(AssertionError):
        check_out(np.zeros_like(ref), ref, True)


def test_small_relative_error_passes_and_large_fails():
    rng = np.random.default_rng(1)
    ref = rng.standard_normal((32, 64))
    check_out(ref + 1e-3 * rng.standard_normal(ref.shape), ref, True)
    with pytest.raises(AssertionError):
        check_out(ref * 1.05, ref, True)
    with pytest.raises(AssertionError):
        check_out(ref + 2e-5, ref, False)


def test_non_finite_entries_must_match():
    ref = np.array([1.0, -np.inf])
    check(np.array([1.0, -np.inf]), ref, 1e-5)
    with pytest.raises(AssertionError):
        check(np.array([1.0, 0.0]), ref, 1e-5)
    with pytest.raises(AssertionError):
        check(np.array([np.nan, -np.inf]), ref, 1e-5)
