"""Pins of the fp64 oracle against things other than itself.

Each test checks one oracle routine against a closed form, an invariant, an
independent library routine (torch SDPA, numpy, scipy) or brute force on tiny
inputs, chosen so that a plausible mistake (dropped term, wrong sign or index,
transposed operand, wrong GQA head mapping, off-by-one causal edge) fails.
"""
import math
from fractions import Fraction

import numpy as np
import pytest
import torch
import torch.nn.functional as F
from scipy.special import logsumexp

pytestmark = pytest.mark.filterwarnings("ignore::UserWarning")


def rng(seed):
    return np.random.default_rng(seed)


# --------------------------------------------------------------------------
# attention
# --------------------------------------------------------------------------

def _sdpa(q, k, v, scale, mask=None):
    """float64 torch SDPA; q [Hq, Lq, d], k/v [Hkv, n, d] -> [Hq, Lq, d]."""
    tq, tk, tv = (torch.from_numpy(np.ascontiguousarray(a))[None] for a in (q, k, v))
    m = None if mask is None else torch.from_numpy(mask)[None, None]
    out = F.scaled_dot_product_attention(tq, tk, tv, attn_mask=m, scale=scale, enable_gqa=True)
    return out[0].numpy()


@pytest.mark.parametrize("G,d,n", [(1, 8, 1), (4, 64, 37), (4, 64, 192), (8, 128, 65), (3, 16, 5)])
def test_attend_matches_torch_sdpa(oracle, G, d, n):
    r = rng(1000 + G * 7 + n)
    q = r.standard_normal((G, d))
    k = r.standard_normal((n, d))
    v = r.standard_normal((n, d))
    s = 1.0 / math.sqrt(d)
    o, lse = oracle.attend(q, k, v, s)
    ref = _sdpa(q[:, None, :], k[None], v[None], s)[:, 0, :]
    np.testing.assert_allclose(o, ref, rtol=0, atol=1e-12)
    # lse against scipy's logsumexp of the scaled scores
    np.testing.assert_allclose(lse, logsumexp(s * q @ k.T, axis=1), rtol=0, atol=1e-12)


def test_attend_batched_gqa_head_mapping(oracle):
    """Query head h reads KV head h // G: checked against SDPA's own GQA."""
    r = rng(7)
    B, Hq, Hkv, d, nmax = 3, 8, 2, 16, 11
    n = np.array([11, 4, 7], np.int32)
    q = r.standard_normal((B, Hq, d))
    k = r.standard_normal((B, Hkv, nmax, d))
    v = r.standard_normal((B, Hkv, nmax, d))
    o, lse = oracle.attend_batched(q, k, v, n, 0.25)
    for b in range(B):
        ref = _sdpa(q[b][:, None, :], k[b][:, : n[b]], v[b][:, : n[b]], 0.25)[:, 0, :]
        np.testing.assert_allclose(o[b], ref, rtol=0, atol=1e-12)
    # a G=1 mapping mistake (h % Hkv) would read other heads: make sure heads differ
    assert np.abs(k[:, 0] - k[:, 1]).max() > 0.1


def test_attend_brute_force_exact_rationals(oracle):
    """Tiny case with scores chosen so that exp weights are exact powers of e:
    scores s_j = j * ln 2 makes weights 2^j / sum 2^j -- rational."""
    d = 2
    q = np.array([[math.log(2.0), 0.0]])
    k = np.array([[0.0, 5.0], [1.0, -3.0], [2.0, 1.0], [3.0, 0.0]])
    v = np.array([[1.0, 0.0], [0.0, 1.0], [2.0, 2.0], [-1.0, 4.0]])
    o, lse = oracle.attend(q, k, v, 1.0)
    w = [Fraction(2 ** j, 15) for j in range(4)]
    exp_o = [float(sum(wj * Fraction(vj[c]) for wj, vj in zip(w, v))) for c in range(d)]
    np.testing.assert_allclose(o[0], exp_o, rtol=0, atol=1e-14)
    assert abs(lse[0] - math.log(15.0)) < 1e-14


def test_attend_closed_forms(oracle):
    r = rng(11)
    d = 32
    # one key: output is that value, lse is the single score
    q = r.standard_normal((2, d)); k = r.standard_normal((1, d)); v = r.standard_normal((1, d))
    o, lse = oracle.attend(q, k, v, 0.3)
    np.testing.assert_allclose(o, np.repeat(v, 2, 0), atol=1e-15)
    np.testing.assert_allclose(lse, 0.3 * q @ k[0], atol=1e-13)
    # identical keys: uniform weights -> mean of values, lse = score + ln n
    n = 9
    k = np.repeat(r.standard_normal((1, d)), n, 0); v = r.standard_normal((n, d))
    o, lse = oracle.attend(q, k, v, 0.3)
    np.testing.assert_allclose(o, np.repeat(v.mean(0, keepdims=True), 2, 0), atol=1e-14)
    np.testing.assert_allclose(lse, 0.3 * q @ k[0] + math.log(n), atol=1e-13)
    # zero query: uniform as well
    o, _ = oracle.attend(np.zeros((1, d)), r.standard_normal((n, d)), v, 1.0)
    np.testing.assert_allclose(o[0], v.mean(0), atol=1e-14)
    # two keys: logistic weights
    k = r.standard_normal((2, d)); v = r.standard_normal((2, d)); q1 = r.standard_normal((1, d))
    s = 0.125 * (q1 @ k.T)[0]
    a = 1.0 / (1.0 + math.exp(s[1] - s[0]))
    o, _ = oracle.attend(q1, k, v, 0.125)
    np.testing.assert_allclose(o[0], a * v[0] + (1 - a) * v[1], atol=1e-14)


def test_attend_weights_sum_to_one_and_permutation_invariance(oracle):
    r = rng(12)
    q = r.standard_normal((4, 64)) * 3
    k = r.standard_normal((300, 64)); v = r.standard_normal((300, 64))
    o, lse, ws = oracle.attend(q, k, v, 0.125, with_wsum=True)
    assert np.abs(ws - 1).max() < 1e-12
    perm = r.permutation(300)
    o2, lse2 = oracle.attend(q, k[perm], v[perm], 0.125)
    np.testing.assert_allclose(o2, o, atol=1e-13)
    np.testing.assert_allclose(lse2, lse, atol=1e-12)


def test_attend_peaky_no_overflow(oracle):
    r = rng(13)
    d, n = 64, 500
    k = r.standard_normal((n, d)); v = r.standard_normal((n, d))
    j = 123
    q = (40.0 * k[j])[None]
    o, lse = oracle.attend(q, k, v, 1.0)
    assert np.all(np.isfinite(o)) and np.isfinite(lse[0])
    np.testing.assert_allclose(o[0], v[j], atol=1e-10)


def test_attend_empty_list(oracle):
    o, lse = oracle.attend(np.ones((2, 8)), np.zeros((0, 8)), np.zeros((0, 8)), 1.0)
    assert np.all(o == 0) and np.all(np.isneginf(lse))


# --------------------------------------------------------------------------
# verify attention
# --------------------------------------------------------------------------

def test_verify_matches_sdpa_with_causal_mask(oracle):
    r = rng(21)
    B, T, Hq, Hkv, d, cap = 2, 5, 8, 2, 16, 40
    length = np.array([40, 17], np.int32)
    q = r.standard_normal((B, T, Hq, d))
    k = r.standard_normal((B, Hkv, cap, d)); v = r.standard_normal((B, Hkv, cap, d))
    o, lse = oracle.verify(q, k, v, length, 0.2)
    for b in range(B):
        L = int(length[b])
        mask = np.zeros((T, L), bool)
        for t in range(T):
            mask[t, : L - T + t + 1] = True      # prefix + new tokens 0..t
        ref = _sdpa(q[b].transpose(1, 0, 2), k[b][:, :L], v[b][:, :L], 0.2, mask)
        np.testing.assert_allclose(o[b], ref.transpose(1, 0, 2), atol=1e-12)


def test_verify_T1_reduces_to_decode_and_future_keys_do_not_leak(oracle):
    r = rng(22)
    B, Hq, Hkv, d, cap = 1, 4, 1, 8, 20
    k = r.standard_normal((B, Hkv, cap, d)); v = r.standard_normal((B, Hkv, cap, d))
    q = r.standard_normal((B, 1, Hq, d))
    o, lse = oracle.verify(q, k, v, np.array([13], np.int32), 0.5)
    o2, lse2 = oracle.attend_batched(q[:, 0], k, v, np.array([13], np.int32), 0.5)
    np.testing.assert_allclose(o[:, 0], o2, atol=1e-14)
    # T = 5: perturb the keys after query t's last visible key -> query t unchanged
    T = 5
    q = r.standard_normal((B, T, Hq, d))
    o, _ = oracle.verify(q, k, v, np.array([18], np.int32), 0.5)
    for t in range(T):
        k2, v2 = k.copy(), v.copy()
        k2[:, :, 18 - T + t + 1:] += 5.0
        v2[:, :, 18 - T + t + 1:] -= 7.0
        o2, _ = oracle.verify(q, k2, v2, np.array([18], np.int32), 0.5)
        np.testing.assert_allclose(o2[:, t], o[:, t], atol=1e-14)
        if t < T - 1:
            assert np.abs(o2[:, t + 1] - o[:, t + 1]).max() > 1e-6


# --------------------------------------------------------------------------
# projection and RoPE
# --------------------------------------------------------------------------

def test_project_matches_numpy(oracle):
    r = rng(31)
    x = r.standard_normal((5, 48)); w = r.standard_normal((24, 48)) * 0.02
    np.testing.assert_allclose(oracle.project(x, w), x @ w.T, atol=1e-13)


def test_rope_against_complex_rotation(oracle):
    """Pair (k_i, k_{i+d/2}) is the complex number k_i + 1j*k_{i+d/2}; RoPE
    multiplies it by exp(1j * pos * base^(-2i/d))."""
    r = rng(32)
    R, H, d, base = 3, 2, 16, 500000.0
    k = r.standard_normal((R, H, d))
    pos = np.array([0, 7, 32769], np.int32)
    out = oracle.rope(k, pos, base)
    half = d // 2
    theta = base ** (-np.arange(half) * 2.0 / d)
    z = (k[..., :half] + 1j * k[..., half:]) * np.exp(1j * pos[:, None, None] * theta[None, None, :])
    np.testing.assert_allclose(out[..., :half], z.real, atol=1e-12)
    np.testing.assert_allclose(out[..., half:], z.imag, atol=1e-12)


def test_rope_known_values_and_invariants(oracle):
    # d = 2: theta_0 = 1, so [1, 0] at pos p becomes [cos p, sin p]
    out = oracle.rope(np.array([[[1.0, 0.0]]]), np.array([3], np.int32), 10000.0)
    np.testing.assert_allclose(out[0, 0], [math.cos(3), math.sin(3)], atol=1e-15)
    r = rng(33)
    k = r.standard_normal((4, 3, 64))
    # position 0 is the identity
    np.testing.assert_allclose(oracle.rope(k, np.zeros(4, np.int32), 500000.0), k, atol=0)
    # per-pair norms preserved
    out = oracle.rope(k, np.array([5, 100, 1000, 30000], np.int32), 500000.0)
    n0 = k[..., :32] ** 2 + k[..., 32:] ** 2
    n1 = out[..., :32] ** 2 + out[..., 32:] ** 2
    np.testing.assert_allclose(n1, n0, rtol=1e-12)
    # relative-position property: <R(a, m), R(b, n)> depends on m - n only
    a = r.standard_normal((1, 1, 64)); b = r.standard_normal((1, 1, 64))
    def dot(m, n):
        return float((oracle.rope(a, np.array([m], np.int32), 500000.0) *
                      oracle.rope(b, np.array([n], np.int32), 500000.0)).sum())
    assert abs(dot(10, 3) - dot(1010, 1003)) < 1e-10
    assert abs(dot(10, 3) - dot(3, 10)) > 1e-6   # not symmetric in general


def test_memory_update_k_rotated_v_not(oracle):
    r = rng(34)
    hkv, d, D = 2, 8, 16
    x = r.standard_normal((3, D)); w = r.standard_normal((2 * hkv * d, D)) * 0.02
    pos = np.array([16, 32, 48], np.int32)
    k, v = oracle.memory_update(x, w, pos, hkv, d, 10000.0)
    y = x @ w.T
    np.testing.assert_allclose(v, y[:, hkv * d:].reshape(3, hkv, d), atol=1e-14)
    kk = y[:, : hkv * d].reshape(3, hkv, d)
    np.testing.assert_allclose(k, oracle.rope(kk, pos, 10000.0), atol=1e-14)
    # a slot and the raw token after it share a position id: with the same
    # projection and hidden state both get the same key (copy-init invariant)
    k_raw, _ = oracle.memory_update(x[:1], w, np.array([16], np.int32), hkv, d, 10000.0)
    np.testing.assert_allclose(k_raw[0], k[0], atol=0)


# --------------------------------------------------------------------------
# argmax and greedy accept
# --------------------------------------------------------------------------

def test_argmax_matches_numpy_including_ties_and_nan(oracle):
    r = rng(41)
    x = r.standard_normal((6, 1000)).astype(np.float32)
    x[1, 10] = x[1, 500] = 50.0            # tie -> lowest index
    x[2, 7] = np.nan; x[2, 3] = np.nan     # NaN ranks highest, first NaN wins
    x[3, :] = 0.0; x[3, 999] = -0.0        # all equal -> 0
    x[4, 998] = np.inf; x[4, 999] = np.inf
    np.testing.assert_array_equal(oracle.argmax(x), np.argmax(x, axis=1))
    assert oracle.argmax(x)[1] == 10 and oracle.argmax(x)[2] == 3


def test_accept_greedy_cases(oracle):
    r = rng(42)
    B, T, V = 4, 5, 300
    logits = r.standard_normal((B, T, V)).astype(np.float32)
    am = np.argmax(logits, axis=2)
    draft = am[:, : T - 1].copy()
    draft[1, 0] = (am[1, 0] + 1) % V        # reject at 0
    draft[2, 2] = (am[2, 2] + 1) % V        # reject at 2 (and later garbage)
    draft[2, 3] = (am[2, 3] + 5) % V
    draft[3, 3] = (am[3, 3] + 1) % V        # reject at the last drafted token
    na, nx = oracle.accept_greedy(logits, draft)
    np.testing.assert_array_equal(na, [4, 0, 2, 3])
    np.testing.assert_array_equal(nx, [am[0, 4], am[1, 0], am[2, 2], am[3, 3]])
    # T = 1 (nothing drafted): emit the target's argmax
    na, nx = oracle.accept_greedy(logits[:, :1], np.zeros((B, 0), np.int32))
    np.testing.assert_array_equal(na, 0)
    np.testing.assert_array_equal(nx, am[:, 0])
