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


def test_lse_tolerance_scale_and_teeth():
    from parity import abs_score, abs_score_verify, check_lse, lse_tol
    rng = np.random.default_rng(2)
    d, scale = 64, 64 ** -0.5
    q = rng.standard_normal((4, d))
    k = rng.standard_normal((3000, d))
    A = abs_score(q, k, scale)
    tol = lse_tol(A, np.full(4, 9.0), d)
    assert np.all(tol > 1e-5) and np.all(tol < 3e-5)          # N(0,1) inputs: about 2e-5
    assert lse_tol(50.0, 50.0, d) < 1e-4                       # scores near 50: about 8e-5
    ref = np.full(4, 9.0)
    check_lse(ref + 0.5 * tol, ref, A, d)
    with pytest.raises(AssertionError):
        check_lse(ref + 1e-4, ref, A, d)                       # an error well above rounding fails
    with pytest.raises(AssertionError):
        check_lse(np.array([9.0, 9.0, 9.0, 0.0]), np.array([9.0, 9.0, 9.0, -np.inf]), A, d)
    # verify: query t sees rows 0 .. len-T+t
    B, T, Hq, Hkv, cap = 2, 3, 4, 2, 10
    qv = rng.standard_normal((B, T, Hq, d))
    kv = rng.standard_normal((B, Hkv, cap, d))
    L = [7, 10]
    Av = abs_score_verify(qv, kv, L, scale)
    for b in range(B):
        for t in range(T):
            for h in range(Hq):
                n = L[b] - T + t + 1
                assert abs(Av[b, t, h] - scale * (np.abs(qv[b, t, h]) @ np.abs(kv[b, h // 2, :n]).T).max()) < 1e-12
