"""GPU parity of mad_draft_decode_attn against the fp64 oracle.

Each case fills the memory segment, the window ring and the new token with
seeded values, runs the kernel through the C ABI, and compares with the
oracle's attention over the key list the ABI defines:
    mem rows [0, mlen) ++ ring rows (start + i) % cap, i < wlen ++ new token.
The same bf16 (or fp32) values feed both sides.  Every buffer the kernel
writes is surrounded by sentinel bands checked after the call.  Tolerances:
see parity.py.
"""
import numpy as np
import pytest
import torch

from parity import abs_score_batched, check_lse, check_out, to_np

pytestmark = pytest.mark.gpu


def _case(dtype, B, Hq, Hkv, d, mlen, wlen, wcap, wstart, new=True, seed=0, mcap=None, peaky=0.0,
          mem=True):
    import paper_2608_30252_amd as mad
    from paper_2608_30252_amd import synth
    dev = torch.device("cuda")
    mlen = list(mlen) if hasattr(mlen, "__len__") else [mlen] * B
    wlen = list(wlen) if hasattr(wlen, "__len__") else [wlen] * B
    wstart = list(wstart) if hasattr(wstart, "__len__") else [wstart] * B
    mcap = mcap or max(max(mlen), 1)
    s = 1000 * seed
    q = synth.normal((B, Hq, d), s + 1, dtype=dtype)
    mk = synth.normal((B, Hkv, mcap, d), s + 2, dtype=dtype)
    mv = synth.normal((B, Hkv, mcap, d), s + 3, dtype=dtype)
    wk = synth.normal((B, Hkv, wcap, d), s + 4, dtype=dtype)
    wv = synth.normal((B, Hkv, wcap, d), s + 5, dtype=dtype)
    kn = synth.normal((B, Hkv, d), s + 6, dtype=dtype)
    vn = synth.normal((B, Hkv, d), s + 7, dtype=dtype)
    G = Hq // Hkv
    targets = {}
    if peaky:
        # each query is peaky * one visible key: with peaky >= 2 the softmax is close to one-hot
        # (the target key's weight is checked below) and o is close to that key's value row
        for b in range(B):
            for h in range(Hq):
                c = h // G
                if wlen[b] > 0:
                    kt = wk[b, c, (wstart[b] + (h * 7) % wlen[b]) % wcap]
                elif mlen[b] > 0:
                    kt = mk[b, c, (h * 5) % mlen[b]]
                else:
                    continue
                q[b, h] = (peaky * kt.float()).to(dtype)
                targets[(b, h)] = kt.double().numpy()
    g = {n: t.to(dev) for n, t in dict(q=q, mk=mk, mv=mv, kn=kn, vn=vn).items()}
    # every buffer the kernel writes (output, lse, the ring it appends to) sits
    # between two 4 KiB sentinel bands that must come back untouched
    guards = []

    def guarded(t, fill):
        pad = 4096 // t.element_size()
        buf = torch.full((t.numel() + 2 * pad,), fill, dtype=t.dtype, device=dev)
        view = buf[pad:pad + t.numel()].view(t.shape)
        view.copy_(t)
        guards.append((buf, pad, t.numel(), buf.clone()))
        return view

    g["wk"], g["wv"] = guarded(wk.to(dev), -77.0), guarded(wv.to(dev), -77.0)
    wk_before, wv_before = g["wk"].clone(), g["wv"].clone()
    memkv = mad.KV(g["mk"], g["mv"], mlen) if mem else None
    win = mad.KV(g["wk"], g["wv"], wlen, wstart)
    out = guarded(torch.full_like(g["q"], 3.0), 3.0)
    lse = guarded(torch.full((B, Hq), 5.0, device=dev), 5.0)
    mad.draft_decode_attn(g["q"], memkv, win, g["kn"] if new else None, g["vn"] if new else None, out, lse)
    torch.cuda.synchronize()
    for buf, pad, n_, before in guards:
        for band in (slice(0, pad), slice(pad + n_, 2 * pad + n_)):
            a_, b_ = buf[band], before[band]
            assert torch.equal(a_.view(torch.int16) if a_.element_size() == 2 else a_.view(torch.int32),
                               b_.view(torch.int16) if b_.element_size() == 2 else b_.view(torch.int32)), "guard band"

    # oracle key lists per sequence
    import oracle
    n = [mlen[b] * (1 if mem else 0) + wlen[b] + (1 if new else 0) for b in range(B)]
    nmax = max(max(n), 1)
    K = np.zeros((B, Hkv, nmax, d)); V = np.zeros((B, Hkv, nmax, d))
    mk64, mv64, wk64, wv64 = (t.double().numpy() for t in (mk, mv, wk, wv))
    kn64, vn64 = kn.double().numpy(), vn.double().numpy()
    for b in range(B):
        rows_k, rows_v = [], []
        if mem and mlen[b]:
            rows_k.append(mk64[b, :, : mlen[b]]); rows_v.append(mv64[b, :, : mlen[b]])
        if wlen[b]:
            idx = (wstart[b] + np.arange(wlen[b])) % wcap
            rows_k.append(wk64[b][:, idx]); rows_v.append(wv64[b][:, idx])
        if new:
            rows_k.append(kn64[b][:, None]); rows_v.append(vn64[b][:, None])
        if rows_k:
            K[b, :, : n[b]] = np.concatenate(rows_k, axis=1)
            V[b, :, : n[b]] = np.concatenate(rows_v, axis=1)
    o_ref, lse_ref = oracle.attend_batched(q.double().numpy(), K, V, np.array(n), d ** -0.5)
    bf = dtype == torch.bfloat16
    q64 = q.double().numpy()
    for (b, h), kt in targets.items():
        w = np.exp(d ** -0.5 * float(q64[b, h] @ kt) - lse_ref[b, h])
        assert w >= 0.9 if peaky >= 2 else w > 0, f"peaky query ({b}, {h}): target weight {w:.3f}"
    check_out(to_np(out), o_ref, bf)
    check_lse(to_np(lse), lse_ref, abs_score_batched(q64, K, n, d ** -0.5), d)

    # the new token's K and V rows were appended at ring row (start + len) % cap; no other bit moved
    for before, new_rows, name in ((wk_before, kn, "wk"), (wv_before, vn, "wv")):
        after = g[name].cpu()
        expect = before.cpu().clone()
        if new:
            for b in range(B):
                expect[b, :, (wstart[b] + wlen[b]) % wcap] = new_rows[b]
        assert torch.equal(after.view(torch.int16) if bf else after.view(torch.int32),
                           expect.view(torch.int16) if bf else expect.view(torch.int32)), f"{name} ring bits"
    return out, lse


def test_tiny_fp32_shape():
    # 4 query heads / 1 KV head, d 64: 64 slots + 127 window rows + the new token
    _case(torch.float32, 1, 4, 1, 64, 64, 127, 144, 5, seed=1)


def test_tiny_fp32_ring_wrap_and_peaky():
    _case(torch.float32, 1, 4, 1, 64, 64, 127, 144, 140, seed=2, peaky=2.0)


def test_draft_8k_layer_bf16():
    _case(torch.bfloat16, 1, 32, 8, 64, 512, 511, 512 + 32, 17, seed=3)


def test_draft_32k_compressed_layer_bf16():
    _case(torch.bfloat16, 1, 32, 8, 64, 2048, 1023, 1024 + 32, 1000, seed=4)


def test_draft_32k_full_kv_layer_bf16():
    # the uncompressed comparison: no memory, the whole 32768-token prefix in the window
    _case(torch.bfloat16, 1, 32, 8, 64, 0, 32768, 32768 + 64, 0, seed=5, mem=False)


@pytest.mark.parametrize("r,mlen", [(4, 8288), (8, 4208)])
def test_paper_shaped_memory_32k_bf16(r, mlen):
    # 32K prefix, 128 sinks + (32768 - 128) / r slots (materialised 4 at a time), a 128-token window:
    # 8416 keys at r = 4, 4336 at r = 8 (the ring wraps: 127 rows from row 200 of a 256-row ring)
    _case(torch.bfloat16, 1, 32, 8, 64, mlen, 127, 256, 200, seed=13 + r)


@pytest.mark.parametrize("c", [3.0, 4.0])
def test_peaky_queries_bf16(c):
    # the 32K compact layer (2048 slots + 1023 window + new token) with q = c k_j: the target key holds
    # at least 0.9 of the softmax weight (asserted; at c = 2 a short key among 3072 can hold only ~0.8),
    # lse ~ 8 c
    _case(torch.bfloat16, 1, 32, 8, 64, 2048, 1023, 1056, 50, seed=6, peaky=c)


def test_peaky_queries_on_memory_rows_bf16():
    # no window: every query points at a memory row
    _case(torch.bfloat16, 2, 32, 8, 64, 2048, 0, 16, 0, seed=14, peaky=3.0, new=False)


def test_ragged_batch_bf16():
    B = 16
    rng = np.random.default_rng(7)
    mlen = rng.integers(0, 1025, B).tolist()
    wlen = rng.integers(0, 512, B).tolist()
    wlen[3] = 0
    mlen[5] = 0
    start = rng.integers(0, 544, B).tolist()
    _case(torch.bfloat16, B, 32, 8, 64, mlen, wlen, 544, start, seed=8, mcap=1024)


def test_maximum_batch_ragged_bf16():
    # the largest batch the ABI takes (64 sequences, 512 units), ragged memories and windows,
    # some sequences with an empty memory or window
    B = 64
    rng = np.random.default_rng(64)
    mlen = rng.integers(0, 201, B).tolist()
    wlen = rng.integers(0, 121, B).tolist()
    mlen[0], wlen[1], mlen[2], wlen[2] = 0, 0, 0, 0
    start = rng.integers(0, 160, B).tolist()
    _case(torch.bfloat16, B, 32, 8, 64, mlen, wlen, 160, start, seed=64, mcap=200)


def test_long_full_kv_reaches_the_split_cap_bf16():
    # 131072 keys in one sequence of 4 KV heads: the plan aims at 128 splits a
    # unit and is held to the merge buffer's cap (65 splits of 4 heads x d 64)
    n = 131071
    _case(torch.bfloat16, 1, 16, 4, 64, 0, n, n + 65, 40, seed=65, mem=False)


def test_folded_last_split_with_a_ragged_batch_bf16():
    # 2 rows x 8 KV heads: 32 splits of 256 keys; row 0 (8192 + new = 8193 keys)
    # folds its new token into the last split, row 1 (4999 + new) leaves its
    # last splits empty
    _case(torch.bfloat16, 2, 32, 8, 64, 0, [8192, 4999], 8192 + 64, [11, 3000], seed=70, mem=False)


@pytest.mark.parametrize("n", [8192, 32768])
def test_full_kv_leftover_key_folded_into_the_last_split_bf16(n):
    # n window keys + the new token: 64 splits of n / 64 keys would leave the
    # token for a 65th split whose workgroups would not all be resident at
    # once, so the last split takes it (the token is also appended)
    _case(torch.bfloat16, 1, 32, 8, 64, 0, n, n + 64, 17, seed=66 + n // 8192, mem=False)


@pytest.mark.parametrize("n", [768, 1280, 1792])
def test_twelve_twenty_and_twenty_eight_splits_bf16(n):
    # n keys per row (slots + 511 window rows + the new token) cut into 12 / 20 / 28 splits of 64:
    # the merge's lanes then take 3 / 5 / 7 splits each
    _case(torch.bfloat16, 1, 32, 8, 64, n - 512, 511, 576, 33, seed=80 + n // 256)


def test_batched_sixteen_sequences_bench_configuration():
    # the benchmark's batched launch: 16 sequences x (1024 slots + 511 window + new), 8-wave workgroups
    _case(torch.bfloat16, 16, 32, 8, 64, 1024, 511, 576, [(37 * i) % 64 for i in range(16)], seed=12, mcap=1024)


def test_no_new_token_and_no_memory():
    _case(torch.bfloat16, 2, 32, 8, 64, 300, 200, 256, 100, new=False, seed=9)
    _case(torch.bfloat16, 2, 32, 8, 64, 0, 200, 256, 100, new=True, seed=10, mem=False)


def test_empty_key_set_gives_zero_and_minus_inf():
    out, lse = _case(torch.bfloat16, 2, 8, 2, 64, [0, 5], [0, 3], 16, [0, 2], new=False, seed=11)
    assert torch.all(out[0].float() == 0) and torch.all(torch.isneginf(lse[0]))


def test_empty_row_beside_a_long_one_merges_to_zero_and_minus_inf():
    # row 0 holds no key at all while row 1's 3071 keys give every unit 24 splits:
    # row 0's units merge 24 empty partials
    out, lse = _case(torch.bfloat16, 2, 32, 8, 64, [0, 2048], [0, 1023], 1056, [0, 7], new=False, seed=15)
    assert torch.all(out[0].float() == 0) and torch.all(torch.isneginf(lse[0]))


@pytest.mark.parametrize("Hq,Hkv,d", [(8, 8, 64), (16, 8, 64), (64, 8, 128), (32, 2, 128), (16, 1, 64)])
def test_group_sizes_and_head_dims(Hq, Hkv, d):
    _case(torch.bfloat16, 2, Hq, Hkv, d, 333, 120, 160, 90, seed=20 + Hq + d)


def test_fp32_head_dim_128_group_8():
    _case(torch.float32, 2, 16, 2, 128, 100, 90, 128, 60, seed=30)


def test_deterministic():
    a = _case(torch.bfloat16, 1, 32, 8, 64, 2048, 1023, 1056, 3, seed=12)
    b = _case(torch.bfloat16, 1, 32, 8, 64, 2048, 1023, 1056, 3, seed=12)
    assert torch.equal(a[0].view(torch.int16), b[0].view(torch.int16))
    assert torch.equal(a[1], b[1])


def test_one_workspace_serves_calls_of_different_shapes():
    """Calls of different shapes share one workspace: counters must never sit
    where another shape's call wrote split partials."""
    import paper_2608_30252_amd as mad
    shapes = [(2, 16, 1, 64), (8, 64, 8, 128), (2, 16, 1, 64), (4, 16, 2, 128), (1, 32, 8, 64)]
    nbytes = max(mad.workspace_bytes(mad.MAD_OP_DECODE, *s) for s in shapes)
    ws = torch.zeros(nbytes, dtype=torch.uint8, device="cuda")
    for i, (B, Hq, Hkv, d) in enumerate(shapes * 2):
        _case_ws(ws, B, Hq, Hkv, d, seed=100 + i)


def _case_ws(ws, B, Hq, Hkv, d, seed):
    import oracle
    import paper_2608_30252_amd as mad
    from paper_2608_30252_amd import synth
    n = 700
    q = synth.normal((B, Hq, d), seed * 10 + 1)
    k = synth.normal((B, Hkv, n, d), seed * 10 + 2)
    v = synth.normal((B, Hkv, n, d), seed * 10 + 3)
    out, lse = mad.draft_decode_attn(q.cuda(), mad.KV(k.cuda(), v.cuda(), [n] * B), None, ws=ws)
    o_ref, lse_ref = oracle.attend_batched(q.double().numpy(), k.double().numpy(), v.double().numpy(),
                                           np.full(B, n), d ** -0.5)
    check_out(to_np(out), o_ref, True, f"out B{B} Hq{Hq} Hkv{Hkv} d{d}")
    check_lse(to_np(lse), lse_ref, abs_score_batched(q.double().numpy(), k.double().numpy(), [n] * B, d ** -0.5), d)
