"""GPU parity of mad_accept_stochastic against the fp64 oracle.

Both sides take the same float32 probabilities, drafted tokens and uniforms.
The accept decisions are exact in double precision on both sides, so
n_accept must match bit for bit.  The emitted token is an inverse-CDF draw
whose running sums the GPU forms in a different order than the oracle's
sequential scan; it must match unless u * Z lies within 1e-9 * Z of the
oracle's bin edge (checked, not assumed, for every mismatch).
"""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu


def _dist(rng, shape, temp=1.0):
    x = rng.standard_normal(shape) / temp
    e = np.exp(x - x.max(-1, keepdims=True))
    return (e / e.sum(-1, keepdims=True)).astype(np.float32)


def _edge_distance(p_row, q_row, resid, t):
    """Distance from t to the nearest bin edge of the oracle's sequential running sum."""
    r = p_row.astype(np.float64) - (q_row.astype(np.float64) if resid else 0.0)
    r = np.where(r > 0, r, 0.0)
    c = np.cumsum(r)
    return float(np.min(np.abs(c - t))), float(c[-1])


def _run(B, T, V, seed, accept_bias=0.0, oob=False, tail=0):
    import oracle
    import paper_2608_30252_amd as mad
    rng = np.random.default_rng(seed)
    p = _dist(rng, (B, T, V), 0.5)
    if tail:   # most of p's mass on the last `tail` entries, so the draw lands there
        p[..., V - tail:] += 10.0
        p = (p / p.sum(-1, keepdims=True)).astype(np.float32)
    q = _dist(rng, (B, T - 1, V), 0.5) if T > 1 else np.zeros((B, 0, V), np.float32)
    if T > 1 and accept_bias:
        q = (accept_bias * p[:, :T - 1] + (1 - accept_bias) * q).astype(np.float32)
    draft = np.zeros((B, T - 1), np.int64)
    for b in range(B):
        for i in range(T - 1):
            c = np.cumsum(q[b, i].astype(np.float64))
            draft[b, i] = min(int(np.searchsorted(c, rng.random() * c[-1], side="right")), V - 1)
    if oob and T > 1:
        draft[0, 0] = V + 3
    u = rng.random((B, T)).astype(np.float32)
    na_ref, nx_ref = oracle.accept_stochastic(p, q, draft, u)

    dev = torch.device("cuda")
    tp = torch.from_numpy(p).to(dev)
    tq = torch.from_numpy(q).to(dev) if T > 1 else None
    td = torch.from_numpy(draft.astype(np.int32)).to(dev) if T > 1 else None
    tu = torch.from_numpy(u).to(dev)
    na, nx = mad.accept_stochastic(tp, tq, td, tu)
    torch.cuda.synchronize()
    na, nx = na.cpu().numpy(), nx.cpu().numpy()
    assert np.array_equal(na, na_ref), (na, na_ref)
    for b in range(B):
        if nx[b] == nx_ref[b]:
            continue
        a = int(na_ref[b])
        resid = a < T - 1
        _, Z = _edge_distance(p[b, a], q[b, a] if resid else None, resid, 0.0)
        dist, _ = _edge_distance(p[b, a], q[b, a] if resid else None, resid, float(u[b, T - 1]) * Z)
        assert dist <= 1e-9 * Z, f"seq {b}: gpu {nx[b]} vs oracle {nx_ref[b]}, edge distance {dist:.3e}"
    return na, nx


@pytest.mark.parametrize("B,T", [(4, 5), (1, 5), (16, 6), (3, 1), (2, 2)])
def test_target_vocabulary(B, T):
    _run(B, T, 128256, seed=100 * B + T)


def test_high_acceptance_and_bonus_tokens():
    na, _ = _run(8, 5, 128256, seed=7, accept_bias=0.97)
    assert (na == 4).any()   # some sequences accept everything and draw the bonus token


def test_small_and_unaligned_vocabularies():
    for i, V in enumerate([1, 3, 7, 8191, 8192, 8193, 50001]):
        _run(3, 4, V, seed=200 + i)


@pytest.mark.parametrize("V", [8196, 8228, 16420, 128256])
def test_draw_in_a_ragged_last_chunk_of_an_aligned_vocabulary(V):
    # V % 4 == 0 takes the float4 path; its last 8192-entry chunk is ragged and
    # the draw lands in it, where runs reach past the chunk's end
    tail = V % 8192
    for T in (3, 1):   # a residual draw, then a draw from p alone
        _, nx = _run(4, T, V, seed=V + T, tail=tail)
        assert (nx >= V - tail).all(), nx


def test_out_of_range_drafted_token_is_rejected():
    na, _ = _run(2, 5, 4096, seed=9, oob=True)
    assert na[0] == 0


def test_threshold_equality_rejects():
    import oracle
    import paper_2608_30252_amd as mad
    dev = torch.device("cuda")
    p = np.array([[[0.1, 0.2, 0.3, 0.4], [0.25, 0.25, 0.25, 0.25]]], np.float32)
    q = np.array([[[0.1, 0.4, 0.3, 0.2]]], np.float32)
    for u0, want in ((0.5, 0), (0.49, 1)):
        u = np.array([[u0, 0.3]], np.float32)
        d = np.array([[1]])
        na_ref, nx_ref = oracle.accept_stochastic(p, q, d, u)
        na, nx = mad.accept_stochastic(torch.from_numpy(p).to(dev), torch.from_numpy(q).to(dev),
                                       torch.from_numpy(d.astype(np.int32)).to(dev), torch.from_numpy(u).to(dev))
        torch.cuda.synchronize()
        assert int(na.item()) == int(na_ref[0]) == want
        assert int(nx.item()) == int(nx_ref[0])
