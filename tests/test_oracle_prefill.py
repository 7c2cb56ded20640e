"""Pins of the oracle's memory-prefill attention (Sec. 3.3 prefill; the
appendix on memory prefill).

The oracle builds each query's key list from the visible-set simulator.  The
pins below build the prefill pass the way the appendix describes it instead:
one sequence in pass order -- every raw token followed by the slot tokens
materialised in its pass -- and one dense attention mask over it, from the
appendix's rules (sinks globally visible; a slot sees the earlier slots, itself
and the raw tokens of its unit, i.e. the W before its position id; a raw token
sees the sinks, the slots already materialised before it and its bounded local
window), evaluated with torch's scaled_dot_product_attention in float64.
Special cases reduce to textbook forms: with no slots and a window covering
the prefix the pass is causal attention; with W = 1 and no sinks or slots each
raw token attends only to itself.
"""
import numpy as np
import pytest
import torch

import oracle
from oracle.masw_sets import MaswSets


def _pass_order(P, S, r, u):
    """[('raw', x) | ('slot', m)] in the order the prefill pass processes them."""
    seq, m = [], 0
    for x in range(P):
        seq.append(("raw", x))
        if x + 1 > S and (x + 1 - S) % (r * u) == 0:   # the last raw token of a block of u units
            for _ in range(u):
                m += 1
                seq.append(("slot", m))
    return seq


def _dense_reference(q_raw, q_slot, mem_k, mem_v, raw_k, raw_v, P, S, W, r, u, scale):
    seq = _pass_order(P, S, r, u)
    n = len(seq)
    Hq, d = q_raw.shape[1], q_raw.shape[2]
    Hkv = mem_k.shape[0]
    Q = np.zeros((Hq, n, d))
    K = np.zeros((Hkv, n, d))
    V = np.zeros((Hkv, n, d))
    for i, (kind, idx) in enumerate(seq):
        if kind == "raw":
            Q[:, i], K[:, i], V[:, i] = q_raw[idx], raw_k[:, idx], raw_v[:, idx]
        else:
            Q[:, i], K[:, i], V[:, i] = q_slot[idx - 1], mem_k[:, S + idx - 1], mem_v[:, S + idx - 1]
    mask = np.zeros((n, n), dtype=bool)
    for i, (qk, qi) in enumerate(seq):
        for j, (kk, kj) in enumerate(seq):
            if qk == "raw":
                if kk == "raw":
                    mask[i, j] = kj <= qi and (kj < S or kj >= qi - W + 1)
                else:
                    mask[i, j] = j < i                       # already materialised
            else:
                b = S + qi * r                                # the slot's position id
                if kk == "raw":
                    mask[i, j] = kj < S or (b - W <= kj <= b - 1)
                else:
                    mask[i, j] = kj <= qi
    G = Hq // Hkv
    Kr = torch.from_numpy(K).repeat_interleave(G, dim=0)
    Vr = torch.from_numpy(V).repeat_interleave(G, dim=0)
    o = torch.nn.functional.scaled_dot_product_attention(torch.from_numpy(Q), Kr, Vr,
                                                         attn_mask=torch.from_numpy(mask), scale=scale).numpy()
    return seq, o   # o [Hq, n, d]


def _inputs(P, S, W, r, u, Hq=4, Hkv=2, d=8, seed=0):
    rng = np.random.default_rng(seed)
    M = MaswSets(S, W, r, u).slots_after(P)
    q_raw = rng.standard_normal((P, Hq, d))
    q_slot = rng.standard_normal((max(M, 1), Hq, d))
    raw_k = rng.standard_normal((Hkv, P, d))
    raw_v = rng.standard_normal((Hkv, P, d))
    mem_k = rng.standard_normal((Hkv, S + max(M, 1), d))
    mem_v = rng.standard_normal((Hkv, S + max(M, 1), d))
    s = min(S, P)
    mem_k[:, :s], mem_v[:, :s] = raw_k[:, :s], raw_v[:, :s]   # the sinks are raw tokens 0..S-1
    return q_raw, q_slot, mem_k, mem_v, raw_k, raw_v, M


@pytest.mark.parametrize("P,S,W,r,u", [
    (97, 0, 16, 4, 1),     # per-boundary schedule, no sinks
    (120, 3, 10, 4, 2),    # batched schedule, sinks
    (61, 5, 7, 3, 1),      # window shorter than a slot unit pair
    (4, 6, 5, 2, 1),       # a prefix shorter than the sinks
    (130, 4, 4, 8, 3),     # window shorter than the slot interval
])
def test_oracle_matches_the_pass_order_mask(P, S, W, r, u):
    scale = 0.37
    q_raw, q_slot, mem_k, mem_v, raw_k, raw_v, M = _inputs(P, S, W, r, u, seed=P + S)
    raw_out, slot_out = oracle.memory_prefill(q_raw, q_slot if M else None, mem_k, mem_v, raw_k, raw_v,
                                              P, S, W, r, u, scale)
    seq, o = _dense_reference(q_raw, q_slot, mem_k, mem_v, raw_k, raw_v, P, S, W, r, u, scale)
    assert len(raw_out) == P and len(slot_out) == M
    for i, (kind, idx) in enumerate(seq):
        got = raw_out[idx][0] if kind == "raw" else slot_out[idx][0]
        np.testing.assert_allclose(got, o[:, i], rtol=0, atol=1e-12, err_msg=f"{kind} {idx}")


def test_no_slots_and_a_covering_window_is_causal_attention():
    P, scale = 50, 0.5
    q_raw, _, mem_k, mem_v, raw_k, raw_v, M = _inputs(P, 0, P, P + 1, 1, seed=3)
    assert M == 0
    raw_out, _ = oracle.memory_prefill(q_raw, None, mem_k, mem_v, raw_k, raw_v, P, 0, P, P + 1, 1, scale)
    G = 2
    o = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q_raw.transpose(1, 0, 2).copy()), torch.from_numpy(raw_k).repeat_interleave(G, 0),
        torch.from_numpy(raw_v).repeat_interleave(G, 0), is_causal=True, scale=scale).numpy()
    for p in range(P):
        np.testing.assert_allclose(raw_out[p][0], o[:, p], rtol=0, atol=1e-12)


def test_unit_window_without_sinks_or_slots_attends_to_itself():
    P = 20
    q_raw, _, mem_k, mem_v, raw_k, raw_v, _ = _inputs(P, 0, 1, 1000, 1, seed=4)
    raw_out, _ = oracle.memory_prefill(q_raw, None, mem_k, mem_v, raw_k, raw_v, P, 0, 1, 1000, 1, 1.0)
    for p in range(P):
        o, lse = raw_out[p]
        np.testing.assert_array_equal(o, np.repeat(raw_v[:, p], 2, axis=0))
        want = np.array([q_raw[p, h] @ raw_k[h // 2, p] for h in range(4)])
        np.testing.assert_allclose(lse, want, rtol=0, atol=1e-12)


def test_slot_count_of_the_prefix():
    # 32K prefix, r = 16, four slots per update: 2048 slots; the paper's own
    # setting S = 128, r = 4: floor((t - S) / r)
    assert MaswSets(0, 1024, 16, 4).slots_after(32768) == 2048
    assert MaswSets(128, 128, 4, 1).slots_after(1000) == (1000 - 128) // 4
    assert sum(1 for k, _ in _pass_order(32768, 0, 16, 4) if k == "slot") == 2048
