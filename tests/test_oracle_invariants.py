"""The oracle's invariants named by the method itself, and a randomized brute
force for its arithmetic routines.

* A memory that holds every evicted raw token uncompressed turns the compact
  view into full causal attention (Sec. 3.1: the working memory replaces the
  raw tokens that left the window).  Checked for the paper's sets (sinks +
  evicted tokens + the local window of raw query p) and for the [memory | ring
  | new token] key list the C ABI receives (rows placed by the host layout),
  against float64 causal SDPA over the whole sequence.
* With no slots (slot interval longer than the prefix) the compact view is the
  sinks plus a sliding window of W tokens: the SWA draft of the experimental
  setup, checked against SDPA under a sinks + sliding-window mask.
* Pure-Python brute force (math.fsum) on random tiny inputs (d <= 4, at most 8
  keys) for attend, verify, project and rope; rope by applying the one-step
  rotation `pos` times instead of evaluating the angle pos * theta.
"""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle.masw_sets import MaswSets
from paper_2608_30252_amd.state import MemoryLayout

pytestmark = pytest.mark.filterwarnings("ignore::UserWarning")


def _causal_sdpa(q, k, v, scale, mask):
    """float64 SDPA: q [Hq, L, d], k/v [Hkv, L, d], mask [L, L] bool (True = visible)."""
    tq, tk, tv = (torch.from_numpy(np.ascontiguousarray(a))[None] for a in (q, k, v))
    out = F.scaled_dot_product_attention(tq, tk, tv, attn_mask=torch.from_numpy(mask)[None, None], scale=scale,
                                         enable_gqa=True)
    return out[0].numpy()


def _sequence(seed, L, Hq, Hkv, d):
    r = np.random.default_rng(seed)
    return (r.standard_normal((Hq, L, d)), r.standard_normal((Hkv, L, d)), r.standard_normal((Hkv, L, d)))


# ---------------------------------------------------------------- invariants --

@pytest.mark.parametrize("S,W,r,L", [(0, 8, 4, 40), (4, 8, 4, 40), (3, 5, 2, 31), (0, 1, 3, 17), (2, 16, 16, 24)])
def test_uncompressed_memory_of_evicted_tokens_is_full_attention_sets(oracle, S, W, r, L):
    """Raw query p attends its sinks and window (paper sets); a memory holding the
    evicted raw tokens [S, window start) in place of the slots completes it to
    the whole causal prefix [0, p]."""
    Hq, Hkv, d = 4, 2, 8
    G = Hq // Hkv
    q, k, v = _sequence(100 + S + W + r, L, Hq, Hkv, d)
    sets = MaswSets(S, W, r)
    full = _causal_sdpa(q, k, v, 0.3, np.tril(np.ones((L, L), bool)))
    for p in range(L):
        view = sets.raw_view(p)
        w_lo = view.window[0] if view.window else p + 1
        evicted = list(range(S, w_lo)) if p >= S else []
        keys = view.sink + evicted + view.window
        assert sorted(keys) == list(range(p + 1))     # no gap, no duplicate at the window edge
        for c in range(Hkv):
            o, lse = oracle.attend(q[c * G:(c + 1) * G, p], k[c, keys], v[c, keys], 0.3)
            np.testing.assert_allclose(o, full[c * G:(c + 1) * G, p], rtol=0, atol=1e-12)


@pytest.mark.parametrize("S,W,ring_extra", [(0, 8, 0), (4, 8, 5), (2, 5, 3), (0, 1, 2)])
def test_uncompressed_memory_of_evicted_tokens_is_full_attention_abi_keys(oracle, S, W, ring_extra):
    """The same invariant on the key list the decode entry point assembles:
    memory rows [0, mem_len) (sinks, then every evicted raw token in order), the
    ring rows start .. start+len-1 (mod cap) of the host layout, then the new
    token -- attended by the batched oracle as one list per (sequence, KV head)."""
    Hq, Hkv, d, L = 8, 2, 16, 45
    q, k, v = _sequence(7 + S + W, L, Hq, Hkv, d)
    ring_cap = W + ring_extra
    lay = MemoryLayout(S, W, r=L + 1, ring_cap=ring_cap, mem_cap=L)
    full = _causal_sdpa(q, k, v, 0.25, np.tril(np.ones((L, L), bool)))
    ring_k = np.full((Hkv, ring_cap, d), np.nan)
    ring_v = np.full((Hkv, ring_cap, d), np.nan)
    for p in range(S, L):
        view = lay.decode_view(p)
        n_evicted = p - S - view.win_len
        mem_rows = list(range(S)) + list(range(S, S + n_evicted))   # sinks, evicted raw tokens
        kl = [k[:, x] for x in mem_rows]
        vl = [v[:, x] for x in mem_rows]
        for i in range(view.win_len):
            row = (view.win_start + i) % ring_cap
            kl.append(ring_k[:, row])
            vl.append(ring_v[:, row])
        kl.append(k[:, p])
        vl.append(v[:, p])
        K = np.stack(kl, 1)[None]
        V = np.stack(vl, 1)[None]
        o, lse = oracle.attend_batched(q[:, p][None], K, V, np.array([K.shape[2]]), 0.25)
        np.testing.assert_allclose(o[0], full[:, p], rtol=0, atol=1e-12)
        # the decode call appends the current token at ring row (start + len) % cap
        row = (view.win_start + view.win_len) % ring_cap
        assert row == lay.ring_row(p)
        ring_k[:, row], ring_v[:, row] = k[:, p], v[:, p]


@pytest.mark.parametrize("S,W", [(0, 6), (4, 6), (2, 1), (3, 12)])
def test_zero_slots_is_sinks_plus_sliding_window(oracle, S, W):
    """Slot interval longer than the prefix: no slot exists, and every raw query
    attends exactly sinks [0, min(S, p+1)) and its last W non-sink tokens --
    the sliding-window draft with attention sinks."""
    Hq, Hkv, d, L = 4, 1, 8, 30
    q, k, v = _sequence(55 + S + W, L, Hq, Hkv, d)
    sets = MaswSets(S, W, r=L + 1)
    mask = np.zeros((L, L), bool)
    for p in range(L):
        for j in range(p + 1):
            mask[p, j] = j < S or j > p - W
    ref = _causal_sdpa(q, k, v, 0.35, mask)
    for p in range(L):
        view = sets.raw_view(p)
        assert view.slots == [] and sets.slots_after(p + 1) == 0
        keys = view.sink + view.window
        o, _ = oracle.attend(q[:, p], k[0, keys], v[0, keys], 0.35)
        np.testing.assert_allclose(o, ref[:, p], rtol=0, atol=1e-12)
    # the host layout agrees: no memory rows beyond the sinks
    lay = MemoryLayout(S, W, r=L + 1, ring_cap=W + 4, mem_cap=S)
    assert all(lay.decode_view(p).mem_len == S for p in range(S, L))


# -------------------------------------------------------------- brute force --

def _bf_attend(q, k, v, scale):
    """One query row: scores, max, weights, normaliser and output by math.fsum."""
    s = [scale * math.fsum(qi * ki for qi, ki in zip(q, kj)) for kj in k]
    m = max(s)
    w = [math.exp(x - m) for x in s]
    z = math.fsum(w)
    o = [math.fsum(wj * vj[i] for wj, vj in zip(w, v)) / z for i in range(len(q))]
    return o, m + math.log(z)


@pytest.mark.parametrize("seed", range(12))
def test_attend_random_brute_force(oracle, seed):
    r = np.random.default_rng(seed)
    G, d, n = int(r.integers(1, 4)), int(r.integers(1, 5)), int(r.integers(1, 9))
    scale = float(r.uniform(0.2, 2.0))
    q = r.standard_normal((G, d)) * 2
    k = r.standard_normal((n, d))
    v = r.standard_normal((n, d))
    o, lse = oracle.attend(q, k, v, scale)
    for g in range(G):
        bo, bl = _bf_attend(q[g].tolist(), k.tolist(), v.tolist(), scale)
        np.testing.assert_allclose(o[g], bo, rtol=0, atol=1e-13)
        assert abs(lse[g] - bl) <= 1e-13


@pytest.mark.parametrize("seed", range(8))
def test_verify_random_brute_force(oracle, seed):
    """Query t of sequence b sees rows 0 .. len[b]-T+t of its KV head h // G."""
    r = np.random.default_rng(50 + seed)
    B, T, Hkv, G, d = int(r.integers(1, 3)), int(r.integers(1, 4)), int(r.integers(1, 3)), int(r.integers(1, 3)), \
        int(r.integers(1, 5))
    Hq, cap = Hkv * G, 8
    length = r.integers(T, cap + 1, size=B)
    q = r.standard_normal((B, T, Hq, d))
    k = r.standard_normal((B, Hkv, cap, d))
    v = r.standard_normal((B, Hkv, cap, d))
    o, lse = oracle.verify(q, k, v, length, 0.7)
    for b in range(B):
        for t in range(T):
            n = int(length[b]) - T + t + 1
            for h in range(Hq):
                c = h // G
                bo, bl = _bf_attend(q[b, t, h].tolist(), k[b, c, :n].tolist(), v[b, c, :n].tolist(), 0.7)
                np.testing.assert_allclose(o[b, t, h], bo, rtol=0, atol=1e-13)
                assert abs(lse[b, t, h] - bl) <= 1e-13


@pytest.mark.parametrize("seed", range(6))
def test_project_random_brute_force(oracle, seed):
    r = np.random.default_rng(90 + seed)
    R, D, N = int(r.integers(1, 4)), int(r.integers(1, 5)), int(r.integers(1, 6))
    x = r.standard_normal((R, D))
    w = r.standard_normal((N, D))
    y = oracle.project(x, w)
    for i in range(R):
        for j in range(N):
            assert abs(y[i, j] - math.fsum(x[i, c] * w[j, c] for c in range(D))) <= 1e-14


@pytest.mark.parametrize("seed", range(6))
def test_rope_random_brute_force_by_repeated_rotation(oracle, seed):
    """RoPE at position pos = the one-step rotation by theta_i applied pos times
    to each pair (i, i + d/2), theta_i = base^(-2i/d)."""
    r = np.random.default_rng(120 + seed)
    d = 2 * int(r.integers(1, 3))          # 2 or 4
    base = float(r.uniform(5.0, 1e4))
    pos = r.integers(0, 9, size=3)
    k = r.standard_normal((3, 1, d))
    got = oracle.rope(k, pos, base)
    for row in range(3):
        for i in range(d // 2):
            th = base ** (-2.0 * i / d)
            c, s = math.cos(th), math.sin(th)
            a, b = k[row, 0, i], k[row, 0, i + d // 2]
            for _ in range(int(pos[row])):
                a, b = math.fsum([a * c, -b * s]), math.fsum([b * c, a * s])
            assert abs(got[row, 0, i] - a) <= 1e-13 and abs(got[row, 0, i + d // 2] - b) <= 1e-13
