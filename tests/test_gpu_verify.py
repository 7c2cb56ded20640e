"""GPU parity of the verify attention against the fp64 oracle.

mad_verify_attn reads the verifier's cache as it is, K and V in rows of d
([B][Hkv][cap][d]); mad_verify_attn_vt reads a V cache stored key-contiguous
per feature ([B][Hkv][d][cap]).  The oracle reads the same values in natural
layout.  Query t of the T new tokens sees rows 0 .. len-T+t.  Tolerances: see
parity.py.
"""
import numpy as np
import pytest
import torch

from parity import abs_score_verify, check_lse, check_out, to_np

pytestmark = pytest.mark.gpu

LAYOUTS = ("natural", "transposed_v")


def _inputs(B, T, Hq, Hkv, d, cap, seed):
    from paper_2608_30252_amd import synth
    s = 1000 * seed
    q = synth.normal((B, T, Hq, d), s + 1)
    k = synth.normal((B, Hkv, cap, d), s + 2)
    v = synth.normal((B, Hkv, cap, d), s + 3)
    return q, k, v


def _run(q, k, v, length, layout="natural"):
    import paper_2608_30252_amd as mad
    dev = torch.device("cuda")
    if layout == "natural":
        out, lse = mad.verify_attn(q.to(dev), mad.KV(k.to(dev), v.to(dev), list(length)))
    else:
        vt = v.transpose(-1, -2).contiguous()
        out, lse = mad.verify_attn_vt(q.to(dev), k.to(dev), vt.to(dev), length)
    torch.cuda.synchronize()
    return out.cpu(), lse.cpu()


def _check(q, k, v, length, out, lse, targets=None):
    """Every sequence against the oracle; with targets (b, t, h) -> key row, also the
    target key's softmax weight (>= 0.9 for a peaky query)."""
    import oracle
    B, T, Hq, d = q.shape
    for b in range(B):
        qb, kb = q[b:b + 1].double().numpy(), k[b:b + 1].double().numpy()
        o_ref, lse_ref = oracle.verify(qb, kb, v[b:b + 1].double().numpy(), np.array([length[b]]), d ** -0.5)
        if targets:
            for (bb, t, h), j in targets.items():
                if bb == b:
                    w = np.exp(d ** -0.5 * float(qb[0, t, h] @ kb[0, h // (Hq // k.shape[1]), j]) - lse_ref[0, t, h])
                    assert w >= 0.9, f"peaky query ({b}, {t}, {h}): target weight {w:.3f}"
        check_out(to_np(out[b:b + 1]), o_ref, out.dtype == torch.bfloat16, f"out b{b}")
        check_lse(to_np(lse[b:b + 1]), lse_ref, abs_score_verify(qb, kb, [length[b]], d ** -0.5), d, f"lse b{b}")


def _make_peaky(q, k, length, c):
    """q[b, t, h] = c * a key row that query t sees (rows 0 .. len-T+t of KV head h // G)."""
    B, T, Hq, d = q.shape
    G = Hq // k.shape[1]
    targets = {}
    for b in range(B):
        for t in range(T):
            n = length[b] - T + t + 1
            for h in range(Hq):
                j = (h * 131 + t * 17 + b * 7) % n
                q[b, t, h] = (c * k[b, h // G, j].float()).to(q.dtype)
                targets[(b, t, h)] = j
    return targets


@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("Hq,Hkv,d,T", [(32, 8, 128, 5), (64, 8, 128, 5), (32, 8, 64, 6), (16, 1, 128, 4),
                                        (8, 8, 128, 1), (16, 16, 64, 2), (64, 4, 64, 4), (32, 2, 128, 4)])
def test_small_shapes(Hq, Hkv, d, T, layout):
    B, cap = 2, 520
    q, k, v = _inputs(B, T, Hq, Hkv, d, cap, seed=Hq + d + T)
    length = [517, 300]
    out, lse = _run(q, k, v, length, layout)
    _check(q, k, v, length, out, lse)


@pytest.mark.parametrize("layout", LAYOUTS)
def test_edge_lengths(layout):
    B, T, Hq, Hkv, d, cap = 3, 5, 32, 8, 128, 64
    q, k, v = _inputs(B, T, Hq, Hkv, d, cap, seed=40)
    length = [5, 64, 37]          # only the new tokens; full capacity; ragged
    out, lse = _run(q, k, v, length, layout)
    _check(q, k, v, length, out, lse)


@pytest.mark.parametrize("layout", LAYOUTS)
def test_maximum_batch(layout):
    # the largest batch the ABI takes: 64 sequences (128 units, one split each), ragged lengths
    B, T, Hq, Hkv, d, cap = 64, 5, 8, 2, 64, 320
    q, k, v = _inputs(B, T, Hq, Hkv, d, cap, seed=47)
    rng = np.random.default_rng(47)
    length = rng.integers(T, cap + 1, B).tolist()
    length[0], length[1] = T, cap
    out, lse = _run(q, k, v, length, layout)
    _check(q, k, v, length, out, lse)


@pytest.mark.parametrize("B,T,Hq,Hkv,d,cap", [(3, 5, 8, 2, 64, 300), (2, 4, 16, 1, 128, 133), (1, 1, 4, 4, 64, 40)])
def test_fp32_natural_layout(B, T, Hq, Hkv, d, cap):
    # fp32 verify (vector ALUs): every sequence against the oracle at the fp32 bar
    from paper_2608_30252_amd import synth
    s = 1000 * (48 + d + T)
    q = synth.normal((B, T, Hq, d), s + 1, dtype=torch.float32)
    k = synth.normal((B, Hkv, cap, d), s + 2, dtype=torch.float32)
    v = synth.normal((B, Hkv, cap, d), s + 3, dtype=torch.float32)
    length = [cap - 7 * b for b in range(B)]
    length[-1] = max(T, length[-1] // 2)
    out, lse = _run(q, k, v, length, "natural")
    assert out.dtype == torch.float32
    _check(q, k, v, length, out, lse)


def test_natural_layout_any_capacity():
    # the natural layout takes any cache capacity (here not a multiple of 8) and odd lengths
    B, T, Hq, Hkv, d, cap = 2, 5, 32, 8, 64, 301
    q, k, v = _inputs(B, T, Hq, Hkv, d, cap, seed=46)
    length = [301, 77]
    out, lse = _run(q, k, v, length, "natural")
    _check(q, k, v, length, out, lse)


@pytest.mark.parametrize("layout", LAYOUTS)
def test_stale_values_past_len_do_not_leak(layout):
    """Rows past len in the cache may hold anything (here: inf/NaN bit
    patterns); the output must not depend on them."""
    B, T, Hq, Hkv, d, cap = 1, 5, 32, 8, 128, 136
    q, k, v = _inputs(B, T, Hq, Hkv, d, cap, seed=41)
    length = [101]
    k2, v2 = k.clone(), v.clone()
    k2[:, :, 101:] = float("nan")
    v2[:, :, 101:] = float("inf")
    out, lse = _run(q, k2, v2, length, layout)
    _check(q, k, v, length, out, lse)


def test_future_new_tokens_do_not_affect_earlier_queries():
    B, T, Hq, Hkv, d, cap = 1, 5, 32, 8, 128, 1024
    q, k, v = _inputs(B, T, Hq, Hkv, d, cap, seed=42)
    length = [1000]
    out_a, _ = _run(q, k, v, length)
    k2, v2 = k.clone(), v.clone()
    k2[:, :, 998:1000] += 3.0     # new tokens 3 and 4
    v2[:, :, 998:1000] -= 2.0
    out_b, _ = _run(q, k2, v2, length)
    assert torch.equal(out_a[:, :3].view(torch.int16), out_b[:, :3].view(torch.int16))
    assert not torch.equal(out_a[:, 3:].view(torch.int16), out_b[:, 3:].view(torch.int16))


@pytest.mark.parametrize("layout", LAYOUTS)
def test_70b_shaped_layer_full_size(layout):
    # 64 query / 8 KV heads, d 128, batch 1, 32768-token prefix + 5 new tokens
    B, T, Hq, Hkv, d = 1, 5, 64, 8, 128
    length = [32768 + T]
    cap = 32776
    q, k, v = _inputs(B, T, Hq, Hkv, d, cap, seed=43)
    out, lse = _run(q, k, v, length, layout)
    _check(q, k, v, length, out, lse)


@pytest.mark.parametrize("layout", LAYOUTS)
def test_8b_shaped_layer_full_size(layout):
    # 32 query / 8 KV heads, d 128, batch 4, 32768-token prefix + 5 new tokens; every sequence checked
    B, T, Hq, Hkv, d = 4, 5, 32, 8, 128
    length = [32768 + T] * B
    cap = 32776
    q, k, v = _inputs(B, T, Hq, Hkv, d, cap, seed=44)
    out, lse = _run(q, k, v, length, layout)
    _check(q, k, v, length, out, lse)


@pytest.mark.parametrize("B,Hq,c", [(4, 32, 2.0), (1, 64, 2.0), (1, 64, 3.0)])
def test_peaky_queries_full_size(B, Hq, c):
    # both target shapes at the 32K prefix with q = c k_j (j visible to the query): the target key holds
    # at least 0.9 of the softmax weight (asserted), o is close to its value row, lse ~ 11 c
    T, Hkv, d = 5, 8, 128
    length = [32768 + T] * B
    q, k, v = _inputs(B, T, Hq, Hkv, d, 32776, seed=45 + Hq)
    targets = _make_peaky(q, k, length, c)
    out, lse = _run(q, k, v, length)
    _check(q, k, v, length, out, lse, targets)
