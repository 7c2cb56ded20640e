"""Pins of the oracle's stochastic accept/reject rule (Sec. 2.1, Sec. 3.3: the
target keeps the standard rejection-sampling rule, which preserves its output
distribution).  Nothing here compares the oracle with itself:

  * lossless property (Monte Carlo): with the drafted token drawn from q and
    fresh uniforms, the first emitted token is distributed as p, and a draft is
    accepted with probability sum_v min(p(v), q(v));
  * one-hot distributions reduce the rule to greedy accept (pinned separately);
  * when every draft is accepted the emitted token is the inverse-CDF draw from
    p, checked against numpy's searchsorted on the cumulative sum;
  * the acceptance test is strict (u q = p rejects); T = 1 samples from p_0.
"""
import numpy as np
import pytest

import oracle


def _dist(rng, shape, temp=1.0):
    x = rng.standard_normal(shape) / temp
    e = np.exp(x - x.max(-1, keepdims=True))
    return (e / e.sum(-1, keepdims=True)).astype(np.float32)


def test_first_emitted_token_is_distributed_as_the_target():
    rng = np.random.default_rng(11)
    V, N = 5, 200_000
    p0 = _dist(rng, (V,), 0.7)
    q0 = _dist(rng, (V,), 0.7)
    p = np.broadcast_to(np.stack([p0, _dist(rng, (V,))]), (N, 2, V)).copy()
    q = np.broadcast_to(q0, (N, 1, V)).copy()
    x = rng.choice(V, size=N, p=q0.astype(np.float64) / q0.sum())
    u = rng.random((N, 2)).astype(np.float32)
    na, nx = oracle.accept_stochastic(p, q, x[:, None], u)
    first = np.where(na >= 1, x, nx)
    emp = np.bincount(first, minlength=V) / N
    assert np.abs(emp - p0).max() < 5e-3, (emp, p0)
    acc = float((na >= 1).mean())
    assert abs(acc - float(np.minimum(p0, q0).sum())) < 5e-3


def test_one_hot_distributions_reduce_to_greedy():
    rng = np.random.default_rng(12)
    B, T, V = 64, 5, 50
    hot = rng.integers(0, V, size=(B, T))
    p = np.zeros((B, T, V), np.float32)
    np.put_along_axis(p, hot[..., None], 1.0, axis=-1)
    draft = hot[:, :T - 1].copy()
    miss = rng.random((B, T - 1)) < 0.3
    draft[miss] = (draft[miss] + 1 + rng.integers(0, V - 1, size=int(miss.sum()))) % V
    q = np.zeros((B, T - 1, V), np.float32)
    np.put_along_axis(q, draft[..., None], 1.0, axis=-1)
    u = rng.random((B, T)).astype(np.float32)
    na, nx = oracle.accept_stochastic(p, q, draft, u)
    ga, gx = oracle.accept_greedy(p, draft)
    assert np.array_equal(na, ga) and np.array_equal(nx, gx)


def test_all_accepted_draws_the_bonus_token_by_inverse_cdf():
    rng = np.random.default_rng(13)
    B, T, V = 32, 4, 1000
    p = _dist(rng, (B, T, V))
    q = p[:, :T - 1].copy()                     # identical drafts: u q < p for u < 1
    draft = rng.integers(0, V, size=(B, T - 1))
    u = rng.random((B, T)).astype(np.float32)
    na, nx = oracle.accept_stochastic(p, q, draft, u)
    assert np.all(na == T - 1)
    for b in range(B):
        c = np.cumsum(p[b, T - 1].astype(np.float64))
        assert nx[b] == np.searchsorted(c, float(u[b, T - 1]) * c[-1], side="right")


def test_equality_at_the_threshold_rejects_and_resamples_the_residual():
    V = 4
    p = np.array([[[0.1, 0.2, 0.3, 0.4], [0.25, 0.25, 0.25, 0.25]]], np.float32)
    q = np.array([[[0.1, 0.4, 0.3, 0.2]]], np.float32)
    # u * q(1) = 0.5 * 0.4 = 0.2 = p(1): not below, so draft token 1 is rejected
    na, nx = oracle.accept_stochastic(p, q, np.array([[1]]), np.array([[0.5, 0.0]], np.float32))
    assert na[0] == 0
    # residual max(0, p - q) = [0, 0, 0, 0.2]: every uniform lands on token 3
    assert nx[0] == 3
    na, _ = oracle.accept_stochastic(p, q, np.array([[1]]), np.array([[0.49, 0.0]], np.float32))
    assert na[0] == 1


def test_single_query_samples_from_the_first_target_row():
    rng = np.random.default_rng(14)
    B, V = 16, 300
    p = _dist(rng, (B, 1, V))
    u = rng.random((B, 1)).astype(np.float32)
    na, nx = oracle.accept_stochastic(p, np.zeros((B, 0, V), np.float32), np.zeros((B, 0), np.int32), u)
    assert np.all(na == 0)
    for b in range(B):
        c = np.cumsum(p[b, 0].astype(np.float64))
        assert nx[b] == np.searchsorted(c, float(u[b, 0]) * c[-1], side="right")
