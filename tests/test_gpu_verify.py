"""GPU parity of mad_verify_attn against the fp64 oracle.

K is stored [B][Hkv][cap][d]; V is stored key-contiguous per feature,
[B][Hkv][d][cap] (the verifier's cache layout).  The oracle reads the same
values in natural layout.  Query t of the T new tokens sees rows
0 .. len-T+t.  Tolerances: see parity.py.
"""
import numpy as np
import pytest
import torch

from parity import check, check_out, to_np, F32_ATOL

pytestmark = pytest.mark.gpu


def _inputs(B, T, Hq, Hkv, d, cap, seed):
    from paper_2608_30252_amd import synth
    s = 1000 * seed
    q = synth.normal((B, T, Hq, d), s + 1)
    k = synth.normal((B, Hkv, cap, d), s + 2)
    v = synth.normal((B, Hkv, cap, d), s + 3)
    return q, k, v


def _run(q, k, v, length):
    import paper_2608_30252_amd as mad
    dev = torch.device("cuda")
    vt = v.transpose(-1, -2).contiguous()
    out, lse = mad.verify_attn(q.to(dev), k.to(dev), vt.to(dev), length)
    torch.cuda.synchronize()
    return out.cpu(), lse.cpu()


def _check(q, k, v, length, out, lse, bs=None):
    import oracle
    B, T, Hq, d = q.shape
    bs = range(B) if bs is None else bs
    for b in bs:
        o_ref, lse_ref = oracle.verify(q[b:b + 1].double().numpy(), k[b:b + 1].double().numpy(),
                                       v[b:b + 1].double().numpy(), np.array([length[b]]), d ** -0.5)
        check_out(to_np(out[b:b + 1]), o_ref, True, f"out b{b}")
        check(to_np(lse[b:b + 1]), lse_ref, F32_ATOL, None, f"lse b{b}")


@pytest.mark.parametrize("Hq,Hkv,d,T", [(32, 8, 128, 5), (64, 8, 128, 5), (32, 8, 64, 6), (16, 1, 128, 4),
                                        (8, 8, 128, 1), (16, 16, 64, 2), (64, 4, 64, 4), (32, 2, 128, 4)])
def test_small_shapes(Hq, Hkv, d, T):
    B, cap = 2, 520
    q, k, v = _inputs(B, T, Hq, Hkv, d, cap, seed=Hq + d + T)
    length = [517, 300]
    out, lse = _run(q, k, v, length)
    _check(q, k, v, length, out, lse)


def test_edge_lengths():
    B, T, Hq, Hkv, d, cap = 3, 5, 32, 8, 128, 64
    q, k, v = _inputs(B, T, Hq, Hkv, d, cap, seed=40)
    length = [5, 64, 37]          # only the new tokens; full capacity; ragged
    out, lse = _run(q, k, v, length)
    _check(q, k, v, length, out, lse)


def test_stale_values_past_len_do_not_leak():
    """Rows past len in the cache may hold anything (here: inf/NaN bit
    patterns); the output must not depend on them."""
    B, T, Hq, Hkv, d, cap = 1, 5, 32, 8, 128, 136
    q, k, v = _inputs(B, T, Hq, Hkv, d, cap, seed=41)
    length = [101]
    k2, v2 = k.clone(), v.clone()
    k2[:, :, 101:] = float("nan")
    v2[:, :, 101:] = float("inf")
    out, lse = _run(q, k2, v2, length)
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


def test_70b_shaped_layer_full_size():
    # 64 query / 8 KV heads, d 128, batch 1, 32768-token prefix + 5 new tokens
    B, T, Hq, Hkv, d = 1, 5, 64, 8, 128
    length = [32768 + T]
    cap = 32776
    q, k, v = _inputs(B, T, Hq, Hkv, d, cap, seed=43)
    out, lse = _run(q, k, v, length)
    _check(q, k, v, length, out, lse)


def test_8b_shaped_layer_full_size_sampled():
    # 32 query / 8 KV heads, d 128, batch 4, 32768-token prefix + 5 new tokens;
    # the oracle checks two of the four sequences
    B, T, Hq, Hkv, d = 4, 5, 32, 8, 128
    length = [32768 + T] * B
    cap = 32776
    q, k, v = _inputs(B, T, Hq, Hkv, d, cap, seed=44)
    out, lse = _run(q, k, v, length)
    _check(q, k, v, length, out, lse, bs=[1, 3])
