"""GPU parity of mad_accept_greedy against the oracle: bit-exact.

Draft tokens are planted so that each sequence accepts a chosen prefix: the
drafted token equals the target argmax up to position k_b and differs there.
Edge rows carry ties, NaN, signed zeros and infinities.
"""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu


def _planted(logits, seed):
    B, T, V = logits.shape
    rng = np.random.default_rng(seed)
    am = np.argmax(logits, axis=2)
    draft = am[:, : T - 1].copy()
    ks = rng.integers(0, T, B)       # accepted prefix length per sequence (T-1 = all)
    for b, k in enumerate(ks):
        if k < T - 1:
            draft[b, k] = (am[b, k] + 1 + rng.integers(0, V - 1)) % V
            if draft[b, k] == am[b, k]:
                draft[b, k] = (am[b, k] + 1) % V
    return draft.astype(np.int32), ks


def _run(logits_t, draft):
    import paper_2608_30252_amd as mad
    dev = torch.device("cuda")
    d = torch.from_numpy(draft).to(dev) if draft is not None and draft.size else None
    na, nx = mad.accept_greedy(logits_t.to(dev), d)
    torch.cuda.synchronize()
    return na.cpu().numpy(), nx.cpu().numpy()


@pytest.mark.parametrize("B,T,V", [(4, 5, 128256), (1, 5, 128256), (16, 6, 128256), (3, 1, 128256),
                                   (2, 256, 1001), (64, 3, 4099)])
def test_planted_acceptance_fp32(B, T, V):
    # the last two: the largest T (256 rows of a sequence) and the largest batch, unaligned vocabularies
    import oracle
    from paper_2608_30252_amd import synth
    logits = synth.normal((B, T, V), 500 + B * 10 + T + V, dtype=torch.float32)
    x = logits.numpy()
    draft, ks = _planted(x, seed=B + T) if T > 1 else (np.zeros((B, 0), np.int32), np.zeros(B, int))
    na, nx = _run(logits, draft)
    na_ref, nx_ref = oracle.accept_greedy(x, draft)
    np.testing.assert_array_equal(na, na_ref)
    np.testing.assert_array_equal(nx, nx_ref)
    if T > 1:
        np.testing.assert_array_equal(na, ks)


def test_bf16_logits():
    import oracle
    from paper_2608_30252_amd import synth
    B, T, V = 4, 5, 128256
    logits = synth.normal((B, T, V), 77, dtype=torch.bfloat16)   # many exact ties in bf16
    x = logits.float().numpy()
    draft, ks = _planted(x, seed=3)
    na, nx = _run(logits, draft)
    na_ref, nx_ref = oracle.accept_greedy(x, draft)
    np.testing.assert_array_equal(na, na_ref)
    np.testing.assert_array_equal(nx, nx_ref)


def test_ties_nan_signed_zero_infinities():
    import oracle
    B, T, V = 2, 5, 20000
    x = np.random.default_rng(5).standard_normal((B, T, V)).astype(np.float32)
    x[0, 0, 17] = x[0, 0, 19000] = 9.0          # tie: lowest index
    x[0, 1, 12000] = np.nan                     # NaN ranks highest
    x[0, 1, 3] = np.nan                         # first NaN wins
    x[0, 2, :] = -0.0
    x[0, 2, 5] = 0.0                            # all equal -> index 0
    x[0, 3, 9999] = np.inf
    x[0, 3, 10000] = np.inf                     # tie at +inf
    x[1, :, :] = -np.inf
    x[1, 2, 8191] = -1e30                       # chunk boundary
    x[1, 3, 8192] = np.float32(3.4e38)
    am = np.argmax(x, axis=2)
    draft = am[:, :4].astype(np.int32)
    na, nx = _run(torch.from_numpy(x), draft)
    na_ref, nx_ref = oracle.accept_greedy(x, draft)
    np.testing.assert_array_equal(na, na_ref)
    np.testing.assert_array_equal(nx, nx_ref)
    np.testing.assert_array_equal(na, [4, 4])
    assert am[0, 0] == 17 and am[0, 1] == 3 and am[0, 2] == 0 and am[0, 3] == 9999


def test_small_vocab_and_repeated_calls_share_workspace():
    import oracle
    for i, V in enumerate([1, 7, 8192, 8193, 50000]):
        B, T = 2, 3
        x = np.random.default_rng(i).standard_normal((B, T, V)).astype(np.float32)
        am = np.argmax(x, axis=2)
        draft = am[:, :2].astype(np.int32)
        draft[1, 1] = (draft[1, 1] + 1) % V if V > 1 else draft[1, 1]
        na, nx = _run(torch.from_numpy(x), draft)
        na_ref, nx_ref = oracle.accept_greedy(x, draft)
        np.testing.assert_array_equal(na, na_ref)
        np.testing.assert_array_equal(nx, nx_ref)


def test_workspace_shared_with_decode_and_garbage_past_the_counters():
    """The row keys live in the counter region, which every call leaves at
    zero; whatever other calls left in the rest of a shared workspace (here: a
    decode's split partials, then 0xFF bytes) must not leak into the argmax."""
    import oracle
    import paper_2608_30252_amd as mad
    from paper_2608_30252_amd import synth
    dev = torch.device("cuda")
    ws = torch.zeros(4 << 20, dtype=torch.uint8, device=dev)
    # a decode with many splits writes partials after the counter region
    q = synth.normal((1, 32, 64), 901).to(dev)
    kv = synth.normal((1, 8, 4096, 64), 902).to(dev)
    mad.draft_decode_attn(q, None, mad.KV(kv, kv, [4096], [0]), ws=ws)
    B, T, V = 3, 5, 30000
    x = np.random.default_rng(9).standard_normal((B, T, V)).astype(np.float32)
    draft, _ = _planted(x, seed=9)
    for fill in (None, 0xFF):
        if fill is not None:
            ws[1 << 20:] = fill
        na, nx = mad.accept_greedy(torch.from_numpy(x).to(dev), torch.from_numpy(draft).to(dev), ws=ws)
        torch.cuda.synchronize()
        na_ref, nx_ref = oracle.accept_greedy(x, draft)
        np.testing.assert_array_equal(na.cpu().numpy(), na_ref)
        np.testing.assert_array_equal(nx.cpu().numpy(), nx_ref)
    assert int(ws[: 1 << 20].count_nonzero()) == 0   # counters and row keys left at zero
